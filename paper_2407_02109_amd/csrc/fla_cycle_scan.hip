// Cycle-scan (HRSAM Sec. 3.5), fp32, gfx950: the selective state-space scan of every
// channel over the token sequence laid out `repeats` times, the output summed over the copies.
//
// Per channel and state (diagonal A, zero-order hold of the SSM equations of Sec. 3.5):
//   h_t = Abar_t h_{t-1} + Bbar_t x_t,  y_t = sum_n C_t[n] h_t[n],
//   Abar_t = exp(Delta_t a),  Bbar_t = (exp(Delta_t a) - 1) / a * B_t.
// The copies are never laid out.  The scan is linear in its initial state, so the state at
// token t of copy k + 1 is h1_t + P_t S_k, with h1 the scan of one copy from zero, P_t the
// decay from the sequence start to t and S_k the state at the end of copy k
// (S_k = (1 + P_L + ... + P_L^{k-1}) S_1).  Summed over the r copies:
//   sum_k h_t^(k) = r h1_t + P_t G,   G = sum_{j=0}^{r-2} (r-1-j) P_L^j S_1,
// which is the scan of r x started from G instead of zero.  Over chunks of T tokens:
//   pass A  (cycle_scan_chunks): every chunk scanned from zero; its output y1_t = C_t . h1_t
//           goes to y, its end state and its sum of Delta to the workspace;
//   pass B  (cycle_scan_carries): per (batch entry, channel, state), the chunks' carries in
//           order: the state entering chunk c, H_{c-1}, the state S_1 after the sequence, and
//           E_c = r H_{c-1} + P(start -> chunk c) G, the state from which chunk c of the summed
//           scan starts;
//   pass C  (cycle_scan_outputs): within chunk c the summed scan's state is r h1_t + P_t E_c
//           (P_t: the decay from the chunk's start to t), so y_t = r y1_t +
//           sum_n C_t[n] exp(a_n cum_t) E_c[n], cum_t the sum of Delta from the chunk's start
//           to t; no recurrence, y overwritten in place.
// Two passes of exponentials over the data, where scanning the laid-out copies takes r.
//
// A wave takes 64 channels of one chunk: a lane holds one channel's N states in registers;
// x (pass C: y1) and Delta of a token are one coalesced 256-byte read per wave, and B_t, C_t,
// the same for every channel, are wave-uniform reads.  Bound by the vector ALU (one
// exponential per token, channel and state in each of passes A and C).
#include "fla_cycle_scan.h"
#include "fla_swin_device.h"

namespace fla {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kBatch = 32;   // chunk values per load batch of the carry pass
constexpr int kTokens = 4;   // tokens whose x and Delta the scan passes load together

// The N entries of a row of B or C.  The row is the same for the whole wave and read-only
// for the kernel's life: read through the constant address space, so that it comes in by
// scalar loads into scalar registers.
typedef __attribute__((address_space(4))) const float const_float;
template <int N>
__device__ __forceinline__ void load_row(const float* p, float (&w)[N]) {
    const const_float* q = (const const_float*)p;
#pragma unroll
    for (int n = 0; n < N; ++n) w[n] = q[n];
}

template <int N>
__global__ __launch_bounds__(64) void cycle_scan_chunks(CycleArgs c) {
    const int cg = blockIdx.x % c.cgroups;
    const int rest = blockIdx.x / c.cgroups;
    const int chunk = rest % c.nch;
    const int b = rest / c.nch;
    const int ch = cg * 64 + (int)threadIdx.x;
    const bool ok = ch < c.d;
    const int chs = ok ? ch : c.d - 1;
    // the state scaled by a, g = a h, takes one product less per step:
    // g <- dA g + (dA - 1) u b; the output C . h = sum_n (C[n] / a[n]) g[n]
    float a2[N], ia[N], g[N];
#pragma unroll
    for (int n = 0; n < N; ++n) {
        const float a = c.A[(size_t)chs * N + n];
        a2[n] = a * kLog2e;
        ia[n] = 1.f / a;
        g[n] = 0.f;
    }
    const int t0 = chunk * c.T;
    const int t1 = min(t0 + c.T, c.L);
    const float* xp = c.x + (size_t)b * c.L * c.d + chs;
    const float* dp = c.delta + (size_t)b * c.L * c.d + chs;
    const size_t rb = (size_t)b * c.L;
    float sd = 0.f;
    auto step = [&](int t, float u, float dl) {
        const size_t row = rb + t;
        float w[N], cv[N];
        load_row<N>(c.Bm + row * N, w);
        load_row<N>(c.Cm + row * N, cv);
        float acc[2] = {0.f, 0.f};   // two sums, two dependency chains
#pragma unroll
        for (int n = 0; n < N; ++n) {
            const float dA = __builtin_amdgcn_exp2f(dl * a2[n]);
            const float z = u * w[n];
            g[n] = __builtin_fmaf(dA, g[n] + z, -z);   // dA g + (dA - 1) z
            acc[n & 1] = __builtin_fmaf(cv[n] * ia[n], g[n], acc[n & 1]);
        }
        sd += dl;
        // lanes past the last channel compute channel d - 1 from the same inputs: the value
        // they store there is the same
        c.y[row * c.d + chs] = acc[0] + acc[1];
    };
    // whole groups of kTokens tokens: their x and Delta loaded together, one wait per group
    const int tfull = t0 + (t1 - t0) / kTokens * kTokens;
    for (int tg = t0; tg < tfull; tg += kTokens) {
        float uu[kTokens], dd[kTokens];
#pragma unroll
        for (int j = 0; j < kTokens; ++j) {
            uu[j] = xp[(size_t)(tg + j) * c.d];
            dd[j] = dp[(size_t)(tg + j) * c.d];
        }
#pragma unroll
        for (int j = 0; j < kTokens; ++j) step(tg + j, uu[j], dd[j]);
    }
    for (int t = tfull; t < t1; ++t) step(t, xp[(size_t)t * c.d], dp[(size_t)t * c.d]);
    if (ok) {
        // A is read in full before any store (a store to the workspace could alias it, so
        // interleaved, every load would wait for the store before it)
        float a[N];
#pragma unroll
        for (int n = 0; n < N; ++n) a[n] = c.A[(size_t)ch * N + n];
        float* hw = c.ws_h + (((size_t)b * c.nch + chunk) * c.d + ch) * N;
#pragma unroll
        for (int n = 0; n < N; ++n) hw[n] = g[n] / a[n];
        c.ws_s[((size_t)b * c.nch + chunk) * c.d + ch] = sd;
    }
}

// One thread per (batch entry, channel, state): the chunks' carries, in chunk order.
// One workgroup holds every segment of cpw = 256 / seg (channel, state) pairs of one batch
// entry: thread (segment s, pair j).  The chunks of a pair are split into seg consecutive
// segments; each thread scans its segment from zero (its chunks' values come in batches of
// kBatch loads issued before the recurrence, so one memory round trip per batch), the
// segments' end states and Delta sums meet in LDS, every thread combines those before its own
// (its carry in) and all of them (the state after one copy), and then runs over its segment
// again writing E_c = r H_{c-1} + P(start -> chunk c) G.  A segment of one batch keeps its
// values in registers for the second run.
__global__ __launch_bounds__(256) void cycle_scan_carries(CycleArgs c) {
    __shared__ float seg_h[256], seg_s[256];
    const int S = c.seg;
    const int cpw = 256 / S;
    const int tid = (int)threadIdx.x;
    const int j = tid % cpw, seg = tid / cpw;
    const long long per_b = (long long)c.d * c.N;
    const long long wg_per_b = (per_b + cpw - 1) / cpw;
    const int b = (int)(blockIdx.x / wg_per_b);
    const long long cn_ll = (long long)(blockIdx.x - b * wg_per_b) * cpw + j;
    const bool live = cn_ll < per_b;
    const int cn = live ? (int)cn_ll : (int)(per_b - 1);   // ch * N + n (past the end: a copy, not stored)
    const int ch = cn / c.N;
    const float a2 = c.A[cn] * kLog2e;
    const size_t hbase = (size_t)b * c.nch * per_b + cn;              // + chunk * d * N
    const size_t sbase = (size_t)b * c.nch * c.d + ch;                // + chunk * d
    const int cps = (c.nch + S - 1) / S;
    const int k_begin = min(seg * cps, c.nch), k_end = min(k_begin + cps, c.nch);
    const bool one_batch = k_end - k_begin <= kBatch;
    float sv[kBatch], hv[kBatch];
    auto load_batch = [&](int k0) {
#pragma unroll
        for (int i = 0; i < kBatch; ++i) {
            const int k = min(k0 + i, k_end - 1);
            sv[i] = c.ws_s[sbase + (size_t)k * c.d];
            hv[i] = c.ws_h[hbase + (size_t)k * per_b];
        }
    };
    // the segment from zero: its end state and the decay over it (as a sum of Delta)
    float H = 0.f, cum = 0.f;
    for (int k0 = k_begin; k0 < k_end; k0 += kBatch) {
        load_batch(k0);
#pragma unroll
        for (int i = 0; i < kBatch; ++i)
            if (k0 + i < k_end) {
                H = __builtin_fmaf(__builtin_amdgcn_exp2f(a2 * sv[i]), H, hv[i]);
                cum += sv[i];
            }
    }
    seg_h[tid] = H;
    seg_s[tid] = cum;
    __syncthreads();
    // the state entering this segment, and after the whole sequence (S_1) with its decay
    float Hin = 0.f, cin = 0.f, Htot = 0.f, ctot = 0.f;
    for (int s = 0; s < S; ++s) {
        if (s == seg) {
            Hin = Htot;
            cin = ctot;
        }
        const float cs = seg_s[s * cpw + j];
        Htot = __builtin_fmaf(__builtin_amdgcn_exp2f(a2 * cs), Htot, seg_h[s * cpw + j]);
        ctot += cs;
    }
    const float PL = __builtin_amdgcn_exp2f(a2 * ctot);
    float g = 0.f;   // sum_{i=0}^{r-2} (r-1-i) PL^i, Horner from the top power
    for (int i = c.repeats - 2; i >= 0; --i) g = __builtin_fmaf(g, PL, (float)(c.repeats - 1 - i));
    const float G = g * Htot;
    // E_c = r H_{c-1} + P(start -> chunk c) G over the segment's chunks
    H = Hin;
    cum = cin;
    const float r = (float)c.repeats;
    for (int k0 = k_begin; k0 < k_end; k0 += kBatch) {
        if (!one_batch) load_batch(k0);
#pragma unroll
        for (int i = 0; i < kBatch; ++i)
            if (k0 + i < k_end) {
                if (live)
                    c.ws_h[hbase + (size_t)(k0 + i) * per_b] = __builtin_fmaf(__builtin_amdgcn_exp2f(a2 * cum), G, r * H);
                H = __builtin_fmaf(__builtin_amdgcn_exp2f(a2 * sv[i]), H, hv[i]);
                cum += sv[i];
            }
    }
}

template <int N>
__global__ __launch_bounds__(64) void cycle_scan_outputs(CycleArgs c) {
    const int cg = blockIdx.x % c.cgroups;
    const int rest = blockIdx.x / c.cgroups;
    const int chunk = rest % c.nch;
    const int b = rest / c.nch;
    const int ch = cg * 64 + (int)threadIdx.x;
    const bool ok = ch < c.d;
    const int chs = ok ? ch : c.d - 1;
    const float* hw = c.ws_h + (((size_t)b * c.nch + chunk) * c.d + chs) * N;
    float a2[N], e[N];
#pragma unroll
    for (int n = 0; n < N; ++n) {
        a2[n] = c.A[(size_t)chs * N + n] * kLog2e;
        e[n] = hw[n];   // E_c
    }
    const float r = (float)c.repeats;
    const int t0 = chunk * c.T;
    const int t1 = min(t0 + c.T, c.L);
    const size_t rb = (size_t)b * c.L;
    float* yp = c.y + rb * c.d + chs;
    const float* dp = c.delta + rb * c.d + chs;
    float cum = 0.f;   // sum of Delta from the chunk's start to t
    auto step = [&](int t, float y1, float dl) {
        const size_t row = rb + t;
        float cv[N];
        load_row<N>(c.Cm + row * N, cv);
        cum += dl;
        float acc[2] = {r * y1, 0.f};
#pragma unroll
        for (int n = 0; n < N; ++n) {
            const float p = __builtin_amdgcn_exp2f(a2[n] * cum);   // decay from the chunk's start
            acc[n & 1] = __builtin_fmaf(cv[n], p * e[n], acc[n & 1]);
        }
        // each lane reads y1 and then writes y at its own address; lanes past the last
        // channel, which repeat channel d - 1, must not write there (the lane of channel d - 1
        // may already have replaced the y1 they read)
        if (ok) yp[(size_t)t * c.d] = acc[0] + acc[1];
    };
    const int tfull = t0 + (t1 - t0) / kTokens * kTokens;
    for (int tg = t0; tg < tfull; tg += kTokens) {
        float yy[kTokens], dd[kTokens];
#pragma unroll
        for (int j = 0; j < kTokens; ++j) {
            yy[j] = yp[(size_t)(tg + j) * c.d];
            dd[j] = dp[(size_t)(tg + j) * c.d];
        }
#pragma unroll
        for (int j = 0; j < kTokens; ++j) step(tg + j, yy[j], dd[j]);
    }
    for (int t = tfull; t < t1; ++t) step(t, yp[(size_t)t * c.d], dp[(size_t)t * c.d]);
}

template <int N>
hipError_t launch_n(const CycleArgs& a, hipStream_t stream) {
    CycleArgs args = a;
    // carry pass: up to 8 segments of at least kBatch chunks per (channel, state)
    args.seg = 1;
    while (args.seg < 8 && (long long)args.seg * kBatch < a.nch) args.seg *= 2;
    void* params[] = {&args};
    const long long scan_groups = (long long)a.B * a.nch * a.cgroups;
    hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(&cycle_scan_chunks<N>), dim3((unsigned)scan_groups),
                                   dim3(64), params, 0, stream);
    if (e != hipSuccess) return e;
    const long long per_wg = 256 / args.seg;
    const long long carry_groups = (long long)a.B * (((long long)a.d * a.N + per_wg - 1) / per_wg);
    e = hipLaunchKernel(reinterpret_cast<const void*>(&cycle_scan_carries), dim3((unsigned)carry_groups), dim3(256),
                        params, 0, stream);
    if (e != hipSuccess) return e;
    return hipLaunchKernel(reinterpret_cast<const void*>(&cycle_scan_outputs<N>), dim3((unsigned)scan_groups),
                           dim3(64), params, 0, stream);
}

}  // namespace

bool cycle_states_supported(int N) { return N == 1 || N == 2 || N == 4 || N == 8 || N == 16 || N == 32; }

hipError_t launch_cycle_scan(const CycleArgs& a, hipStream_t stream) {
    switch (a.N) {
        case 1: return launch_n<1>(a, stream);
        case 2: return launch_n<2>(a, stream);
        case 4: return launch_n<4>(a, stream);
        case 8: return launch_n<8>(a, stream);
        case 16: return launch_n<16>(a, stream);
        case 32: return launch_n<32>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace fla
