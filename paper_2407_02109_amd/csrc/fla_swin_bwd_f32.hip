// Flash Swin attention backward, fp32 storage and arithmetic (vector ALU), and the
// reduction of the pad token's gradient shared with the bf16 path.
//
// The gradients of Eq. 1 inside each window (the paper trains through Flash Swin, App. D),
// with c = 1/sqrt(d), LSE_i stored by the training forward and D_i = <dO_i, O_i>:
//   P_ij = w_j exp(c <q_i, k_j> - LSE_i),  dS_ij = P_ij (<dO_i, v_j> - D_i)
//   dq_i = c sum_j dS_ij k_j,   dk_j = c sum_i dS_ij q_i,   dv_j = sum_i P_ij dO_i
// Nothing of size n^2 is stored: every kernel recomputes P from q, k and LSE.
//
// Three kernels over the forward's decomposition (one workgroup per batch entry, window,
// block of 256 tokens and head):
//   dq:  one query per thread; keys stream through LDS 64 at a time.  In KV-token mode the
//        pad token (Sec. 3.4, App. B) is one more key of weight n_pad, and the block also
//        writes its share of the pad token's own gradient to the workspace.
//   dv, dk:  one key per thread; queries (q, dO, LSE, D) stream through LDS.
// The pad reduce kernel then sums the workspace shares in a fixed order into row L of dk
// and dv, so the result does not depend on scheduling.
#include "fla_swin_device.h"

namespace fla {
namespace {

constexpr int D = kHeadDim;
constexpr int THREADS = kQueryBlock;   // one token per thread
constexpr int CH = 64;                 // tokens per LDS chunk
constexpr float kLog2e = 1.4426950408889634f;

struct Block {
    int head, blk, win, b;
};

__device__ __forceinline__ Block decode(const SwinArgs& a) {
    long long id = blockIdx.x;
    Block r;
    r.head = (int)(id % a.heads);
    id /= a.heads;
    r.blk = (int)(id % a.nqb);
    id /= a.nqb;
    r.win = (int)(id % a.n_windows);
    r.b = (int)(id / a.n_windows);
    return r;
}

// element offset of window-local token t (t < n) from the start of a batch entry's head
__device__ __forceinline__ long long token_elems(const SwinArgs& a, const WindowRect& wr, int t) {
    const int r = t / wr.cols;
    return (wr.tok0 + (long long)r * wr.W + (t - r * wr.cols)) * a.tok_stride;
}

__device__ __forceinline__ long long token_index(const WindowRect& wr, int t) {
    const int r = t / wr.cols;
    return wr.tok0 + (long long)r * wr.W + (t - r * wr.cols);
}

__global__ __launch_bounds__(THREADS) void swin_bwd_f32_dq_kernel(SwinBwdArgs ba) {
    const SwinArgs& a = ba.f;
    __shared__ __attribute__((aligned(16))) float Kf[CH * D];
    __shared__ __attribute__((aligned(16))) float Vf[CH * D];
    __shared__ float Pp[THREADS], Sp[THREADS];

    const Block blk = decode(a);
    const WindowRect wr = window_rect<true>(a, blk.win);
    const int n = wr.rows * wr.cols;
    const int q_begin = blk.blk * kQueryBlock;
    const long long n_pad = (long long)a.window * a.window - n;
    const bool has_pad = a.pad_mode == 1 && n_pad > 0;
    // KV-token mode: every block writes its share of the pad token's gradient (zero when the
    // window has no virtual slots or the block no queries), so the reduction reads a dense array
    float* ws_entry = a.pad_mode == 1
        ? ba.ws + (((long long)blk.b * a.heads + blk.head) * a.n_windows + blk.win) * a.nqb * kPadPartial +
              (long long)blk.blk * kPadPartial
        : nullptr;
    if (ws_entry != nullptr && !(has_pad && q_begin < n) && threadIdx.x < kPadPartial) ws_entry[threadIdx.x] = 0.f;
    if (q_begin >= n) return;
    const int nq = min(kQueryBlock, n - q_begin);

    const long long qoff = (long long)blk.b * a.q_batch_stride + blk.head * D;
    const long long kvoff = (long long)blk.b * a.kv_batch_stride + blk.head * D;
    const float* qg = static_cast<const float*>(a.q) + qoff;
    const float* og = static_cast<const float*>(ba.out) + qoff;
    const float* dog = static_cast<const float*>(ba.dout) + qoff;
    float* dqg = static_cast<float*>(ba.dq) + qoff;
    const float* kg = static_cast<const float*>(a.k) + kvoff;
    const float* vg = static_cast<const float*>(a.v) + kvoff;
    const long long lse0 = ((long long)blk.b * a.heads + blk.head) * a.L;

    const int tid = threadIdx.x;
    const int t = q_begin + tid;
    const bool active = t < n;
    const int tq = active ? t : n - 1;

    float qv[D], dov[D], dq[D];
    float Dv = 0.f;
    {
        const float* qr = qg + token_elems(a, wr, tq);
        const float* orow = og + token_elems(a, wr, tq);
        const float* dr = dog + token_elems(a, wr, tq);
        for (int i = 0; i < D; ++i) {
            qv[i] = qr[i] * a.scale_log2;   // logits in the exp2 domain
            dov[i] = dr[i];
            Dv = fmaf(dr[i], orow[i], Dv);
            dq[i] = 0.f;
        }
    }
    const float lse2 = ba.lse[lse0 + token_index(wr, tq)] * kLog2e;

    for (int kc0 = 0; kc0 < n; kc0 += CH) {
        const int ck = min(CH, n - kc0);
        __syncthreads();
        for (int i = tid; i < CH * (D / 4); i += THREADS) {
            const int key = i / (D / 4), part = i % (D / 4);
            float4 kx = make_float4(0.f, 0.f, 0.f, 0.f), vx = kx;
            if (key < ck) {
                const long long off = token_elems(a, wr, kc0 + key) + part * 4;
                kx = *reinterpret_cast<const float4*>(kg + off);
                vx = *reinterpret_cast<const float4*>(vg + off);
            }
            *reinterpret_cast<float4*>(&Kf[key * D + part * 4]) = kx;
            *reinterpret_cast<float4*>(&Vf[key * D + part * 4]) = vx;
        }
        __syncthreads();
        for (int j = 0; j < ck; ++j) {
            const float* kr = &Kf[j * D];
            const float* vr = &Vf[j * D];
            float s = 0.f, dp = 0.f;
            for (int i = 0; i < D; ++i) {
                s = fmaf(qv[i], kr[i], s);
                dp = fmaf(dov[i], vr[i], dp);
            }
            const float ds = exp2f(s - lse2) * (dp - Dv);
            for (int i = 0; i < D; ++i) dq[i] = fmaf(ds, kr[i], dq[i]);
        }
    }

    float p_pad = 0.f, ds_pad = 0.f;
    if (has_pad) {
        const long long prow = (long long)blk.b * a.kv_batch_stride + a.L * a.tok_stride + blk.head * D;
        const float* kp = static_cast<const float*>(a.k) + prow;
        const float* vp = static_cast<const float*>(a.v) + prow;
        float s = 0.f, dp = 0.f;
        for (int i = 0; i < D; ++i) {
            s = fmaf(qv[i], kp[i], s);
            dp = fmaf(dov[i], vp[i], dp);
        }
        p_pad = exp2f(s + log2f((float)n_pad) - lse2);
        ds_pad = p_pad * (dp - Dv);
        for (int i = 0; i < D; ++i) dq[i] = fmaf(ds_pad, kp[i], dq[i]);
    }

    if (active) {
        float* row = dqg + token_elems(a, wr, t);
        for (int i = 0; i < D; i += 4)
            *reinterpret_cast<float4*>(row + i) =
                make_float4(dq[i] * ba.scale, dq[i + 1] * ba.scale, dq[i + 2] * ba.scale, dq[i + 3] * ba.scale);
    }

    if (has_pad) {
        // this block's share of the pad token's gradient:
        //   dk_pad += c sum_i dS_ip q_i,  dv_pad += sum_i P_ip dO_i   (over the block's queries)
        Pp[tid] = active ? p_pad : 0.f;
        Sp[tid] = active ? ds_pad : 0.f;
        __syncthreads();
        if (tid < kPadPartial) {
            const bool is_k = tid < D;
            const int ch = is_k ? tid : tid - D;
            const float* src = is_k ? qg : dog;
            const float* wgt = is_k ? Sp : Pp;
            float acc = 0.f;
            for (int i = 0; i < nq; ++i) acc = fmaf(wgt[i], src[token_elems(a, wr, q_begin + i) + ch], acc);
            ws_entry[tid] = is_k ? acc * ba.scale : acc;
        }
    }
}

// KIND 0: dv_j = sum_i P_ij dO_i;  KIND 1: dk_j = c sum_i dS_ij q_i
template <int KIND>
__global__ __launch_bounds__(THREADS) void swin_bwd_f32_dkv_kernel(SwinBwdArgs ba) {
    const SwinArgs& a = ba.f;
    __shared__ __attribute__((aligned(16))) float Qf[CH * D];
    __shared__ __attribute__((aligned(16))) float Gf[CH * D];   // dO rows
    __shared__ float Lf[CH], Df[CH];

    const Block blk = decode(a);
    const WindowRect wr = window_rect<true>(a, blk.win);
    const int n = wr.rows * wr.cols;
    const int k_begin = blk.blk * kQueryBlock;
    if (k_begin >= n) return;

    const long long qoff = (long long)blk.b * a.q_batch_stride + blk.head * D;
    const long long kvoff = (long long)blk.b * a.kv_batch_stride + blk.head * D;
    const float* qg = static_cast<const float*>(a.q) + qoff;
    const float* og = static_cast<const float*>(ba.out) + qoff;
    const float* dog = static_cast<const float*>(ba.dout) + qoff;
    const float* kg = static_cast<const float*>(a.k) + kvoff;
    const float* vg = static_cast<const float*>(a.v) + kvoff;
    float* outg = static_cast<float*>(KIND == 0 ? ba.dv : ba.dk) + kvoff;
    const long long lse0 = ((long long)blk.b * a.heads + blk.head) * a.L;

    const int tid = threadIdx.x;
    const int t = k_begin + tid;
    const bool active = t < n;
    const int tk = active ? t : n - 1;

    float kv[D], vv[KIND == 1 ? D : 1], acc[D];
    {
        const float* kr = kg + token_elems(a, wr, tk);
        for (int i = 0; i < D; ++i) {
            kv[i] = kr[i] * a.scale_log2;
            acc[i] = 0.f;
        }
        if constexpr (KIND == 1) {
            const float* vr = vg + token_elems(a, wr, tk);
            for (int i = 0; i < D; ++i) vv[i] = vr[i];
        }
    }

    for (int qc0 = 0; qc0 < n; qc0 += CH) {
        const int cq = min(CH, n - qc0);
        __syncthreads();
        for (int i = tid; i < CH * (D / 4); i += THREADS) {
            const int qi = i / (D / 4), part = i % (D / 4);
            float4 qx = make_float4(0.f, 0.f, 0.f, 0.f), gx = qx;
            if (qi < cq) {
                const long long off = token_elems(a, wr, qc0 + qi) + part * 4;
                qx = *reinterpret_cast<const float4*>(qg + off);
                gx = *reinterpret_cast<const float4*>(dog + off);
            }
            *reinterpret_cast<float4*>(&Qf[qi * D + part * 4]) = qx;
            *reinterpret_cast<float4*>(&Gf[qi * D + part * 4]) = gx;
        }
        if (tid < CH) {
            float lse2 = 0.f, dd = 0.f;
            if (tid < cq) {
                lse2 = ba.lse[lse0 + token_index(wr, qc0 + tid)] * kLog2e;
                if constexpr (KIND == 1) {
                    const long long off = token_elems(a, wr, qc0 + tid);
                    for (int i = 0; i < D; ++i) dd = fmaf(dog[off + i], og[off + i], dd);
                }
            }
            Lf[tid] = lse2;
            Df[tid] = dd;
        }
        __syncthreads();
        for (int i = 0; i < cq; ++i) {
            const float* qr = &Qf[i * D];
            const float* gr = &Gf[i * D];
            float s = 0.f;
            for (int e = 0; e < D; ++e) s = fmaf(kv[e], qr[e], s);
            const float p = exp2f(s - Lf[i]);
            if constexpr (KIND == 0) {
                for (int e = 0; e < D; ++e) acc[e] = fmaf(p, gr[e], acc[e]);
            } else {
                float dp = 0.f;
                for (int e = 0; e < D; ++e) dp = fmaf(vv[e], gr[e], dp);
                const float ds = p * (dp - Df[i]);
                for (int e = 0; e < D; ++e) acc[e] = fmaf(ds, qr[e], acc[e]);
            }
        }
    }

    if (active) {
        const float sc = KIND == 1 ? ba.scale : 1.f;
        float* row = outg + token_elems(a, wr, t);
        for (int i = 0; i < D; i += 4)
            *reinterpret_cast<float4*>(row + i) =
                make_float4(acc[i] * sc, acc[i + 1] * sc, acc[i + 2] * sc, acc[i + 3] * sc);
    }
}

// One workgroup per (batch entry, head): row L of dk and dv = the sum of the partials of
// every (window, query block).  1024 threads = 8 slices x 128 columns; slice s adds entries
// s, s + 8, ... in their order, fetching 32 of them at a time (one memory round trip per 32
// instead of one per few), and the eight slice sums are added in order.
constexpr int kRedSlices = 8;
constexpr int kRedBatch = 32;
template <typename T>
__global__ __launch_bounds__(kRedSlices * kPadPartial) void swin_bwd_pad_reduce_kernel(SwinBwdArgs ba) {
    const SwinArgs& a = ba.f;
    __shared__ float part[kRedSlices][kPadPartial];
    const int bh = blockIdx.x;
    const int col = threadIdx.x % kPadPartial;
    const int slice = threadIdx.x / kPadPartial;
    const long long nent = (long long)a.n_windows * ba.pad_blocks;
    const float* src = ba.ws + (long long)bh * nent * kPadPartial + col;
    float acc = 0.f;
    for (long long e0 = slice; e0 < nent; e0 += (long long)kRedBatch * kRedSlices) {
        float v[kRedBatch];
#pragma unroll
        for (int u = 0; u < kRedBatch; ++u) {
            const long long e = e0 + (long long)u * kRedSlices;
            v[u] = e < nent ? src[e * kPadPartial] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < kRedBatch; ++u) acc += v[u];
    }
    part[slice][col] = acc;
    __syncthreads();
    if (slice == 0) {
        float s = part[0][col];
        for (int i = 1; i < kRedSlices; ++i) s += part[i][col];
        const int b = bh / a.heads, head = bh - b * a.heads;
        const long long row = (long long)b * a.kv_batch_stride + a.L * a.tok_stride + head * D;
        T* dst = static_cast<T*>(col < D ? ba.dk : ba.dv) + row + (col % D);
        if constexpr (sizeof(T) == 2) {
            const __bf16 r = (__bf16)s;
            *dst = __builtin_bit_cast(uint16_t, r);
        } else {
            *dst = s;
        }
    }
}

}  // namespace

hipError_t launch_swin_bwd_f32(const SwinBwdArgs& a, hipStream_t stream) {
    SwinBwdArgs args = a;
    void* params[] = {&args};
    const dim3 grid((unsigned)a.f.n_groups), block(THREADS);
    hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(&swin_bwd_f32_dq_kernel), grid, block,
                                   params, 0, stream);
    if (e != hipSuccess) return e;
    e = hipLaunchKernel(reinterpret_cast<const void*>(&swin_bwd_f32_dkv_kernel<0>), grid, block, params, 0,
                        stream);
    if (e != hipSuccess) return e;
    return hipLaunchKernel(reinterpret_cast<const void*>(&swin_bwd_f32_dkv_kernel<1>), grid, block, params,
                           0, stream);
}

hipError_t launch_swin_bwd_pad_reduce(const SwinBwdArgs& a, int elem_bytes, hipStream_t stream) {
    SwinBwdArgs args = a;
    void* params[] = {&args};
    const void* fn = elem_bytes == 2 ? reinterpret_cast<const void*>(&swin_bwd_pad_reduce_kernel<uint16_t>)
                                     : reinterpret_cast<const void*>(&swin_bwd_pad_reduce_kernel<float>);
    return hipLaunchKernel(fn, dim3((unsigned)(a.f.B * a.f.heads)), dim3(kRedSlices * kPadPartial), params, 0,
                           stream);
}

}  // namespace fla
