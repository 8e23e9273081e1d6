// Flash Swin attention forward, bf16 storage, gfx950 (CDNA4) matrix cores.
//
// One workgroup = one (batch entry, window, block of up to 256 queries, head).  The
// window's rectangle comes from integer arithmetic on the shifted-window geometry
// (HRSAM Sec. 3.3 / App. A): no index table, no reordered copy.  Its real tokens are
// taken in row-major order inside the rectangle (Eq. nonshift), so the key set is dense:
// n = rows * cols keys, no masked slots except the MFMA tail of the last key tile.
//
// Per workgroup:
//   1. K rows of the window -> LDS row-major (row stride 144 B);
//      V rows -> LDS transposed (V^T, one row per channel), so that P.V can take V as the
//      A operand with keys along the reduction dimension.
//   2. Each of the 4 waves owns 64 queries.  Q stays in registers as the B operand.
//      For every tile of 64 keys:  S^T = K . Q^T  (v_mfma_f32_16x16x32_bf16, fp32 acc),
//      scale into the exp2 domain, mask the key tail, online softmax per query column
//      (cross-lane max over the 4 lane groups), P^T rounded to bf16 stays in registers in
//      exactly the layout the next MFMA reads as its B operand, O^T += V^T . P^T.
//   3. Epilogue: O^T / l, round to bf16 (RNE), store each query row at its own token.
//
// KV-only padding (Sec. 3.4, App. B): the pad token (row L of k, v) is loaded as key n of
// the window and its logit is raised by log2(n_pad), so it carries the weight of the
// n_pad = window^2 - n virtual slots it stands for.
#include "fla_swin_internal.h"

namespace fla {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int D = kHeadDim;     // 64 channels per head
constexpr int THREADS = 256;    // 4 waves of 64
constexpr int KC = 256;         // keys staged in LDS at a time
constexpr int KT = 64;          // keys per inner tile
constexpr int KS = D + 8;       // K row stride in LDS, bf16 elements (144 B)
constexpr int VS = KC + 8;      // V^T row stride in LDS, bf16 elements (528 B)

__device__ __forceinline__ uint4 ld_global16(const uint16_t* p) {
    return *reinterpret_cast<const uint4*>(p);
}

__device__ __forceinline__ float wave_max_groups(float x) {
    // max over the 4 lanes {l, l^16, l^32, l^48}: same query column, different key rows
    x = fmaxf(x, __shfl_xor(x, 16));
    x = fmaxf(x, __shfl_xor(x, 32));
    return x;
}

__device__ __forceinline__ float wave_sum_groups(float x) {
    x += __shfl_xor(x, 16);
    x += __shfl_xor(x, 32);
    return x;
}

// 2 waves per SIMD: the register budget (256) matches what the 70 KB of LDS allows (2 workgroups per CU).
__global__ __launch_bounds__(THREADS) __attribute__((amdgpu_waves_per_eu(2, 2)))
void swin_fwd_bf16_kernel(SwinArgs a) {
    __shared__ __attribute__((aligned(16))) uint16_t Ks[KC * KS];
    __shared__ __attribute__((aligned(16))) uint16_t Vt[D * VS];

    // ---- workgroup -> (b, window, query block, head); heads vary fastest so that the
    //      12 workgroups of one window read adjacent 128-byte pieces of the same rows
    long long id = blockIdx.x;
    const int head = (int)(id % a.heads);
    id /= a.heads;
    const int qblk = (int)(id % a.nqb);
    id /= a.nqb;
    const int nwin = a.nwy * a.nwx;
    const int win = (int)(id % nwin);
    const int b = (int)(id / nwin);

    const WindowRect wr = window_rect(a, win);
    const int n = wr.rows * wr.cols;
    const int q_begin = qblk * kQueryBlock;
    if (q_begin >= n) return;   // whole workgroup: this window has fewer query blocks

    const long long n_pad = (long long)a.window * a.window - n;
    const bool has_pad = a.pad_mode == 1 && n_pad > 0;
    const int nk = n + (has_pad ? 1 : 0);
    const float pad_bias = has_pad ? log2f((float)n_pad) : 0.f;

    const uint16_t* qg = static_cast<const uint16_t*>(a.q) + (long long)b * a.q_batch_stride + head * D;
    const uint16_t* kg = static_cast<const uint16_t*>(a.k) + (long long)b * a.kv_batch_stride + head * D;
    const uint16_t* vg = static_cast<const uint16_t*>(a.v) + (long long)b * a.kv_batch_stride + head * D;
    uint16_t* og = static_cast<uint16_t*>(a.out) + (long long)b * a.q_batch_stride + head * D;
    const long long L = (long long)a.H * a.W;

    // token row (in elements, relative to the per-(b, head) base) of window-local index t
    auto token_off = [&](int t) -> long long {
        if (t >= n) return L * a.tok_stride;          // the pad token (KV-token mode only)
        const int r = t / wr.cols;
        const int c = t - r * wr.cols;
        return ((long long)(wr.y0 + r) * a.W + (wr.x0 + c)) * a.tok_stride;
    };

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int g = lane >> 4;        // lane group: MFMA reduction slice / output row quad
    const int li = lane & 15;       // MFMA row (A) / column (B, output)

    const int wq0 = q_begin + wave * 64;
    const int nq = min(64, n - wq0);   // queries of this wave (<= 0: wave only loads)

    // ---- Q in registers, B-operand layout: lane holds q[query 16*j + li][32*c + 8*g .. +8]
    bf16x8 qop[4][2];
    if (nq > 0) {
        for (int j = 0; j < 4; ++j) {
            const int t = min(wq0 + 16 * j + li, n - 1);
            const uint16_t* row = qg + token_off(t);
            for (int c = 0; c < 2; ++c)
                qop[j][c] = __builtin_bit_cast(bf16x8, ld_global16(row + 32 * c + 8 * g));
        }
    }

    float m_run[4], l_run[4];
    floatx4 o[4][4];   // O^T: [channel block][query block]
    for (int j = 0; j < 4; ++j) {
        m_run[j] = -INFINITY;
        l_run[j] = 0.f;
        for (int db = 0; db < 4; ++db) o[db][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    }

    for (int kc0 = 0; kc0 < nk; kc0 += KC) {
        const int ck = min(KC, nk - kc0);
        const int ck_pad = (ck + KT - 1) / KT * KT;
        if (kc0 > 0) __syncthreads();   // previous chunk fully consumed

        // ---- K chunk -> LDS (row-major).  8 threads per 128-byte row: coalesced.
        for (int i = tid; i < ck_pad * 8; i += THREADS) {
            const int key = i >> 3, part = i & 7;
            uint4 val = make_uint4(0u, 0u, 0u, 0u);
            if (key < ck) val = ld_global16(kg + token_off(kc0 + key) + part * 8);
            *reinterpret_cast<uint4*>(&Ks[key * KS + part * 8]) = val;
        }
        // ---- V chunk -> LDS transposed.  A thread takes 4 keys x 8 channels, swaps
        //      16-bit halves in registers and writes 8 rows of V^T, 4 keys each.
        const int n_quads = ck_pad / 4;
        for (int i = tid; i < n_quads * 8; i += THREADS) {
            const int quad = (i & 7) + ((i >> 6) << 3);
            const int part = (i >> 3) & 7;
            uint4 r[4];
            for (int u = 0; u < 4; ++u) {
                const int key = quad * 4 + u;
                r[u] = make_uint4(0u, 0u, 0u, 0u);
                if (key < ck) r[u] = ld_global16(vg + token_off(kc0 + key) + part * 8);
            }
            const uint32_t* w0 = reinterpret_cast<const uint32_t*>(&r[0]);
            const uint32_t* w1 = reinterpret_cast<const uint32_t*>(&r[1]);
            const uint32_t* w2 = reinterpret_cast<const uint32_t*>(&r[2]);
            const uint32_t* w3 = reinterpret_cast<const uint32_t*>(&r[3]);
            for (int m = 0; m < 4; ++m) {
                uint2 lo, hi;   // channel 2m and 2m+1 of keys quad*4 .. +3
                lo.x = (w0[m] & 0xffffu) | (w1[m] << 16);
                lo.y = (w2[m] & 0xffffu) | (w3[m] << 16);
                hi.x = (w0[m] >> 16) | (w1[m] & 0xffff0000u);
                hi.y = (w2[m] >> 16) | (w3[m] & 0xffff0000u);
                const int ch = part * 8 + 2 * m;
                *reinterpret_cast<uint2*>(&Vt[ch * VS + quad * 4]) = lo;
                *reinterpret_cast<uint2*>(&Vt[(ch + 1) * VS + quad * 4]) = hi;
            }
        }
        __syncthreads();

        if (nq > 0) {
            for (int t0 = 0; t0 < ck; t0 += KT) {
                // ---- S^T tile: 64 keys x 64 queries, lane holds keys 16*kb + 4*g + r
                floatx4 s[4][4];
                for (int kb = 0; kb < 4; ++kb) {
                    const uint16_t* krow = &Ks[(t0 + 16 * kb + li) * KS + 8 * g];
                    const bf16x8 ka0 = *reinterpret_cast<const bf16x8*>(krow);
                    const bf16x8 ka1 = *reinterpret_cast<const bf16x8*>(krow + 32);
                    for (int j = 0; j < 4; ++j) {
                        floatx4 acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            ka0, qop[j][0], floatx4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                        s[kb][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka1, qop[j][1], acc, 0, 0, 0);
                    }
                }
                // ---- scale to the exp2 domain, mask keys past the window, pad-token weight
                const int key_base = kc0 + t0 + 4 * g;
                for (int kb = 0; kb < 4; ++kb) {
                    for (int r = 0; r < 4; ++r) {
                        const int key = key_base + 16 * kb + r;
                        const bool valid = key < nk;
                        const float bias = (has_pad && key == n) ? pad_bias : 0.f;
                        for (int j = 0; j < 4; ++j) {
                            const float x = s[kb][j][r] * a.scale_log2 + bias;
                            s[kb][j][r] = valid ? x : -INFINITY;
                        }
                    }
                }
                // ---- online softmax per query column
                bf16x8 pb[4][2];
                for (int j = 0; j < 4; ++j) {
                    float mx = -INFINITY;
                    for (int kb = 0; kb < 4; ++kb)
                        for (int r = 0; r < 4; ++r) mx = fmaxf(mx, s[kb][j][r]);
                    mx = wave_max_groups(mx);
                    const float m_new = fmaxf(m_run[j], mx);   // finite: key 0 of a tile is valid
                    const float alpha = __builtin_amdgcn_exp2f(m_run[j] - m_new);
                    m_run[j] = m_new;
                    l_run[j] *= alpha;
                    for (int db = 0; db < 4; ++db) o[db][j] *= alpha;
                    float p[4][4];
                    float lsum = 0.f;
                    for (int kb = 0; kb < 4; ++kb)
                        for (int r = 0; r < 4; ++r) {
                            p[kb][r] = __builtin_amdgcn_exp2f(s[kb][j][r] - m_new);
                            lsum += p[kb][r];
                        }
                    l_run[j] += lsum;
                    // B operand of P.V: slots 0..3 = key block 2c, slots 4..7 = key block 2c+1
                    for (int c = 0; c < 2; ++c) {
                        bf16x8 v8;
                        for (int r = 0; r < 4; ++r) {
                            v8[r] = (__bf16)p[2 * c][r];
                            v8[4 + r] = (__bf16)p[2 * c + 1][r];
                        }
                        pb[j][c] = v8;
                    }
                }
                // ---- O^T += V^T . P^T; A operand: channel 16*db + li, the same 8 keys
                for (int c = 0; c < 2; ++c) {
                    for (int db = 0; db < 4; ++db) {
                        const uint16_t* vrow = &Vt[(16 * db + li) * VS + t0 + 32 * c + 4 * g];
                        const bf16x4 va = *reinterpret_cast<const bf16x4*>(vrow);
                        const bf16x4 vb = *reinterpret_cast<const bf16x4*>(vrow + 16);
                        const bf16x8 vA = {va[0], va[1], va[2], va[3], vb[0], vb[1], vb[2], vb[3]};
                        for (int j = 0; j < 4; ++j)
                            o[db][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vA, pb[j][c], o[db][j], 0, 0, 0);
                    }
                }
            }
        }
    }

    // ---- epilogue: normalise, round to bf16 (RNE), store at the query's own token
    if (nq > 0) {
        for (int j = 0; j < 4; ++j) {
            const float l_tot = wave_sum_groups(l_run[j]);
            const float inv = 1.f / l_tot;
            const int qi = 16 * j + li;
            if (qi < nq) {
                uint16_t* row = og + token_off(wq0 + qi);
                for (int db = 0; db < 4; ++db) {
                    bf16x4 r4;
                    for (int r = 0; r < 4; ++r) r4[r] = (__bf16)(o[db][j][r] * inv);
                    *reinterpret_cast<bf16x4*>(row + 16 * db + 4 * g) = r4;
                }
            }
        }
    }
}

}  // namespace

hipError_t launch_swin_fwd_bf16(const SwinArgs& a, hipStream_t stream) {
    SwinArgs args = a;
    void* params[] = {&args};
    return hipLaunchKernel(reinterpret_cast<const void*>(&swin_fwd_bf16_kernel),
                           dim3((unsigned)a.n_groups), dim3(THREADS), params, 0, stream);
}

}  // namespace fla
