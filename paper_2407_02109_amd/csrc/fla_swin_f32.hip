// Flash Swin attention forward, fp32 storage and arithmetic (vector ALU).
//
// Same workgroup decomposition and window geometry as the bf16 kernel (HRSAM Sec. 3.3,
// App. A): one workgroup per (batch entry, window, block of 256 queries, head).  Each
// thread owns one query: its q row and output accumulator live in registers; the
// window's keys stream through LDS 64 at a time and every thread reads the same key
// row (an LDS broadcast).  The online softmax takes 16 keys per rescale step.
// KV-only padding (Sec. 3.4, App. B): the pad token is key n with logit + log2(n_pad).
#include "fla_swin_internal.h"

namespace fla {
namespace {

constexpr int THREADS = kQueryBlock;   // one query per thread
constexpr int KC = 64;                 // keys per LDS chunk
constexpr int KG = 16;                 // keys per rescale step

// D: head_dim (64; the plain forward also has instances for 32 and 128)
template <int D>
__global__ __launch_bounds__(THREADS) void swin_fwd_f32_kernel(SwinArgs a) {
    __shared__ __attribute__((aligned(16))) float Kf[KC * D];
    __shared__ __attribute__((aligned(16))) float Vf[KC * D];

    long long id = blockIdx.x;
    const int head = (int)(id % a.heads);
    id /= a.heads;
    const int qblk = (int)(id % a.nqb);
    id /= a.nqb;
    const int nwin = a.n_windows;
    const int win = (int)(id % nwin);
    const int b = (int)(id / nwin);

    const WindowRect wr = window_rect<true>(a, win);
    const int n = wr.rows * wr.cols;
    const int q_begin = qblk * kQueryBlock;
    if (q_begin >= n) return;

    const long long n_pad = (long long)a.window * a.window - n;
    const bool has_pad = a.pad_mode == 1 && n_pad > 0;
    const int nk = n + (has_pad ? 1 : 0);
    const float pad_bias = has_pad ? log2f((float)n_pad) : 0.f;

    const float* qg = static_cast<const float*>(a.q) + (long long)b * a.q_batch_stride + head * D;
    const float* kg = static_cast<const float*>(a.k) + (long long)b * a.kv_batch_stride + head * D;
    const float* vg = static_cast<const float*>(a.v) + (long long)b * a.kv_batch_stride + head * D;
    float* og = static_cast<float*>(a.out) + (long long)b * a.q_batch_stride + head * D;
    const long long L = a.L;
    auto token_off = [&](int t) -> long long {
        if (t >= n) return L * a.tok_stride;
        const int r = t / wr.cols;
        const int c = t - r * wr.cols;
        return (wr.tok0 + (long long)r * wr.W + c) * a.tok_stride;
    };

    const int tid = threadIdx.x;
    const int t = q_begin + tid;
    const bool active = t < n;

    // 2-D RoPE (when asked): rotate the pairs of 4 channels starting at channel c0 of token t
    // (angles in double: the fp32 path is the tight-tolerance reference)
    auto rope4 = [&](float4& x, int tt, int c0) {
        const int r = tt / wr.cols;
        const double pos = (double)(c0 < D / 2 ? wr.y0 + r : wr.x0 + (tt - r * wr.cols)) * (double)a.rope_scale;
        const int j = (c0 % (D / 2)) / 2;
        double s0, c0s, s1, c1s;
        sincos(pos * a.rope_freq[j], &s0, &c0s);
        sincos(pos * a.rope_freq[j + 1], &s1, &c1s);
        x = make_float4((float)(x.x * c0s - x.y * s0), (float)(x.y * c0s + x.x * s0),
                        (float)(x.z * c1s - x.w * s1), (float)(x.w * c1s + x.z * s1));
    };

    float qv[D], o[D];
    {
        const int tq = active ? t : n - 1;
        const float4* row = reinterpret_cast<const float4*>(qg + token_off(tq));
        for (int i = 0; i < D / 4; ++i) {
            float4 x = row[i];
            if (a.rope) rope4(x, tq, 4 * i);
            qv[4 * i] = x.x * a.scale_log2;
            qv[4 * i + 1] = x.y * a.scale_log2;
            qv[4 * i + 2] = x.z * a.scale_log2;
            qv[4 * i + 3] = x.w * a.scale_log2;
        }
    }
    for (int i = 0; i < D; ++i) o[i] = 0.f;
    float m_run = -INFINITY, l_run = 0.f;

    for (int kc0 = 0; kc0 < nk; kc0 += KC) {
        const int ck = min(KC, nk - kc0);
        __syncthreads();
        // 16 threads per 256-byte key row
        for (int i = tid; i < KC * (D / 4); i += THREADS) {
            const int key = i / (D / 4), part = i % (D / 4);
            float4 kx = make_float4(0.f, 0.f, 0.f, 0.f), vx = kx;
            if (key < ck) {
                const long long off = token_off(kc0 + key) + part * 4;
                kx = *reinterpret_cast<const float4*>(kg + off);
                vx = *reinterpret_cast<const float4*>(vg + off);
                if (a.rope && kc0 + key < n) rope4(kx, kc0 + key, part * 4);   // not the pad token
            }
            *reinterpret_cast<float4*>(&Kf[key * D + part * 4]) = kx;
            *reinterpret_cast<float4*>(&Vf[key * D + part * 4]) = vx;
        }
        __syncthreads();

        for (int j0 = 0; j0 < ck; j0 += KG) {
            float sc[KG];
            float mx = -INFINITY;
            for (int u = 0; u < KG; ++u) {
                const int key = j0 + u;
                const float* kr = &Kf[key * D];
                float acc = 0.f;
                for (int i = 0; i < D; ++i) acc = fmaf(qv[i], kr[i], acc);
                if (has_pad && kc0 + key == n) acc += pad_bias;
                sc[u] = key < ck ? acc : -INFINITY;
                mx = fmaxf(mx, sc[u]);
            }
            const float m_new = fmaxf(m_run, mx);   // finite: key j0 is valid
            const float alpha = exp2f(m_run - m_new);
            m_run = m_new;
            l_run *= alpha;
            for (int i = 0; i < D; ++i) o[i] *= alpha;
            for (int u = 0; u < KG; ++u) {
                const float p = exp2f(sc[u] - m_new);
                l_run += p;
                const float* vr = &Vf[(j0 + u) * D];
                for (int i = 0; i < D; ++i) o[i] = fmaf(p, vr[i], o[i]);
            }
        }
    }

    if (active) {
        if (a.lse != nullptr) {
            const int r = t / wr.cols;
            const long long tok = wr.tok0 + (long long)r * wr.W + (t - r * wr.cols);
            a.lse[((long long)b * a.heads + head) * L + tok] = (m_run + log2f(l_run)) * 0.693147180559945309f;
        }
        const float inv = 1.f / l_run;
        float4* row = reinterpret_cast<float4*>(og + token_off(t));
        for (int i = 0; i < D / 4; ++i)
            row[i] = make_float4(o[4 * i] * inv, o[4 * i + 1] * inv, o[4 * i + 2] * inv, o[4 * i + 3] * inv);
    }
}

}  // namespace

hipError_t launch_swin_fwd_f32(const SwinArgs& a, hipStream_t stream) {
    SwinArgs args = a;
    void* params[] = {&args};
    const void* fn = a.head_dim == 32    ? reinterpret_cast<const void*>(&swin_fwd_f32_kernel<32>)
                     : a.head_dim == 128 ? reinterpret_cast<const void*>(&swin_fwd_f32_kernel<128>)
                                         : reinterpret_cast<const void*>(&swin_fwd_f32_kernel<kHeadDim>);
    return hipLaunchKernel(fn, dim3((unsigned)a.n_groups), dim3(THREADS), params, 0, stream);
}

}  // namespace fla
