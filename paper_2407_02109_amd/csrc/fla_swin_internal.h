// Internal interface between the C-ABI host code and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fla {

__host__ __device__ inline unsigned mulhi_u32(unsigned a, unsigned b) {
    return (unsigned)(((unsigned long long)a * b) >> 32);
}

// Unsigned division by a divisor fixed at launch, exact for every n < 2^31.  Powers of two
// shift; otherwise q = mulhi(n, m) >> s with s = floor(log2 d) and m = ceil(2^(32+s) / d)
// (Granlund & Montgomery, 1994): m = 2^(32+s)/d + e with 0 <= e < 1, and the error term
// n*e / 2^(32+s) stays below 1/d while n < 2^(32+s)/d, which exceeds 2^31.
struct FastDiv {
    unsigned m, s;
    __host__ __device__ unsigned div(unsigned n) const { return (m ? mulhi_u32(n, m) : n) >> s; }
    static __host__ FastDiv make(unsigned d) {
        FastDiv f;
        unsigned s = 0;
        while ((2ull << s) <= d) ++s;   // s = floor(log2 d)
        f.s = s;
        f.m = (d & (d - 1)) == 0 ? 0u : (unsigned)((((unsigned long long)1 << (32 + s)) + d - 1) / d);
        return f;
    }
};

constexpr int kHeadDim = 64;    // head_dim supported by the kernels
constexpr int kQueryBlock = 256; // queries of one window handled by one workgroup

// Everything a kernel needs, computed once on the host per call.
struct SwinArgs {
    const void* q;
    const void* k;
    const void* v;
    void* out;
    int B, heads, H, W;
    int window, shift;
    int origin;                 // (window - shift) % window: virtual tokens in front of each axis
    int nwy, nwx;               // windows per axis: ceil((H + origin) / window), same for W
    int nqb;                    // query blocks per window: ceil(max window size / kQueryBlock)
    int pad_mode;               // 0 = mask virtual keys, 1 = pad token at row L
    int64_t tok_stride;         // elements between consecutive tokens: heads * head_dim
    int64_t q_batch_stride;     // elements between batch entries of q / out: L * tok_stride
    int64_t kv_batch_stride;    // same for k / v (L or L + 1 rows)
    float scale_log2;           // log2(e) / sqrt(head_dim): logits go straight to exp2
    int64_t n_groups;           // workgroups: B * heads * windows * query blocks
    int n_cus;                  // compute units of the device
    FastDiv div_heads, div_nqb, div_nwin, div_nwx;   // workgroup index decode
};

hipError_t launch_swin_fwd_bf16(const SwinArgs& a, hipStream_t stream);
hipError_t launch_swin_fwd_f32(const SwinArgs& a, hipStream_t stream);

// Window of workgroup `win` (raster order over nwy x nwx), clipped to the grid.
struct WindowRect {
    int y0, x0, rows, cols;
};

__device__ __forceinline__ WindowRect window_rect(const SwinArgs& a, int win) {
    const int wy = (int)a.div_nwx.div((unsigned)win);
    const int wx = win - wy * a.nwx;
    const long long ys = (long long)wy * a.window - a.origin;
    const long long xs = (long long)wx * a.window - a.origin;
    const long long ye = ys + a.window < a.H ? ys + a.window : a.H;
    const long long xe = xs + a.window < a.W ? xs + a.window : a.W;
    WindowRect r;
    r.y0 = ys > 0 ? (int)ys : 0;
    r.x0 = xs > 0 ? (int)xs : 0;
    r.rows = (int)(ye - r.y0);
    r.cols = (int)(xe - r.x0);
    return r;
}

}  // namespace fla
