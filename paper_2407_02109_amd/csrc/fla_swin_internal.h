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
// n*e / 2^(32+s) stays below 1/d while n < 2^(32+s)/d, which exceeds 2^31.  Both cases are
// one branch-free expression, (mulhi(n, m) + (n & one)) >> s, with m = 0 and one = ~0 for
// powers of two and one = 0 otherwise, so the workgroup decode has no branch to wait on.
struct FastDiv {
    unsigned m, s, one;
    __host__ __device__ unsigned div(unsigned n) const { return (mulhi_u32(n, m) + (n & one)) >> s; }
    static __host__ FastDiv make(unsigned d) {
        FastDiv f;
        unsigned s = 0;
        while ((2ull << s) <= d) ++s;   // s = floor(log2 d)
        f.s = s;
        const bool pow2 = (d & (d - 1)) == 0;
        f.m = pow2 ? 0u : (unsigned)((((unsigned long long)1 << (32 + s)) + d - 1) / d);
        f.one = pow2 ? ~0u : 0u;
        return f;
    }
};

constexpr int kHeadDim = 64;    // head_dim of every kernel (the training, RoPE and backward paths)
// head_dim values of the plain forward kernels (bf16 and fp32): 64, and the instances 32 and 128
__host__ __device__ constexpr bool fwd_head_dim_ok(int d) { return d == 32 || d == 64 || d == 128; }
constexpr int kQueryBlock = 256; // queries of one window handled by one workgroup

constexpr int kMaxGrids = 8;    // token grids of one multi-scale sequence

// One token grid of the sequence (a single grid, or the image grid and the anchor-map grid
// of multi-scale attention).  Its windows are numbered after those of the grids before it.
struct GridDesc {
    int H, W;                   // rows and columns of tokens
    int nwx;                    // windows per row: ceil((W + origin) / window)
    int win_begin;              // index of its first window among all windows
    int64_t tok_off;            // index of its first token within a batch entry
    FastDiv div_nwx;
};

// Everything a kernel needs, computed once on the host per call.
struct SwinArgs {
    const void* q;
    const void* k;
    const void* v;
    void* out;
    float* lse;                 // optional [B, heads, L] log-sum-exp output (NULL: not kept)
    int B, heads;
    int window, shift;
    int origin;                 // (window - shift) % window: virtual tokens in front of each axis
    int nqb;                    // query blocks per window: ceil(max window size / kQueryBlock)
    int pad_mode;               // 0 = mask virtual keys, 1 = pad token at row L
    int64_t L;                  // tokens per batch entry, all grids (the pad token's row)
    int64_t tok_stride;         // elements between consecutive tokens: heads * head_dim
    int64_t q_batch_stride;     // elements between batch entries of q / out: L * tok_stride
    int64_t kv_batch_stride;    // same for k / v (L or L + 1 rows)
    float scale_log2;           // log2(e) / sqrt(head_dim): logits go straight to exp2
    int64_t n_groups;           // workgroups: B * heads * windows * query blocks
    int64_t n_units;            // B * heads * windows
    int xcd_group;              // forward: the query blocks of a unit share an XCD (nqb > 1)
    int n_cus;                  // compute units of the device
    int n_grids, n_windows;     // grids, and windows over all grids
    GridDesc grid[kMaxGrids];
    FastDiv div_heads, div_nqb, div_nwin;   // workgroup index decode
    // 2-D rotary position embedding of q and k (0: none): channel pair (2j, 2j+1) of the
    // first half of a head turns by (row * rope_scale) * f_j, of the second half by
    // (column * rope_scale) * f_j, f_j = theta^(-2j / (head_dim / 2)).  rope_rev[j] is f_j in
    // revolutions per position unit (f_j / 2 pi, for the hardware sine of the bf16 kernel);
    // rope_freq[j] is f_j in double for the fp32 kernel.
    int rope;
    float rope_scale;
    float rope_rev[kHeadDim / 4];
    double rope_freq[kHeadDim / 4];
    int head_dim;               // channels per head (the forward kernels' instance)
};


// Workgroups of a bf16 forward launch: one per unit in groups of 8 (the last one padded), or
// with xcd_group the nqb query blocks of each unit on one XCD, in groups of 8 units.
__host__ __device__ inline int64_t fwd_bf16_groups(const SwinArgs& a) {
    return a.xcd_group ? 8 * (int64_t)a.nqb * ((a.n_units + 7) / 8) : 8 * ((a.n_groups + 7) / 8);
}

// Workgroup id -> unit for launches of one workgroup per unit (b, window, head), heads
// fastest.  The dispatcher deals ids to the 8 XCDs in turn, so with ids in unit order XCD x
// would only ever see the units u = x (mod 8): with 12 heads, the heads of one residue class
// mod 4.  Loads of some heads run measurably slower than others' (their 128-byte rows sit at
// a different offset in every token's record), and the XCDs holding those heads then
// finish last.  Ids 8 g .. 8 g + 7 take the units 8 g .. 8 g + 7 rotated by g >> s: every XCD
// passes through every class, 2^s groups at a time (mixing the classes on an XCD at a finer
// grain measured slower).  Ids of the last group may fall past the last unit.
__device__ __forceinline__ unsigned xcd_rotate(unsigned id, unsigned s) {
    const unsigned g = id >> 3;
    return (g << 3) + ((id + (g >> s)) & 7u);
}

hipError_t launch_swin_fwd_bf16(const SwinArgs& a, hipStream_t stream);
hipError_t launch_swin_fwd_f32(const SwinArgs& a, hipStream_t stream);

constexpr int kBwdBlock = 128;    // tokens of one bf16 backward block (and of one streamed chunk)
constexpr int kPadPartial = 2 * kHeadDim;   // floats per pad-gradient partial: dk then dv

// Backward pass: the forward's geometry plus the gradient tensors.  Inputs q, k, v (in f),
// out, dout and lse; outputs dq, dk, dv.  ws holds one pad-gradient partial per (b, head,
// window, block) in KV-token mode: ws[((b * heads + head) * n_windows + win) * pad_blocks
// + blk][0:64] = dk part, [64:128] = dv part.  Every block writes its entry (zero when its
// window has no virtual slots), and the pad reduce kernel sums them.  The bf16 kernel's
// blocks are kBwdBlock tokens (pad_blocks = nbb), the fp32 kernels' kQueryBlock tokens
// (pad_blocks = f.nqb).
struct SwinBwdArgs {
    SwinArgs f;
    const void* out;
    const void* dout;
    const float* lse;
    void* dq;
    void* dk;
    void* dv;
    float* ws;
    int pad_blocks;             // blocks per window in the layout of ws
    int nbb;                    // bf16: kBwdBlock-token blocks of the largest window
    FastDiv div_2nbb;           // bf16 workgroup decode: division by 2 * nbb
    int64_t n_units;            // bf16: B * heads * windows
    float scale;                // 1 / sqrt(head_dim)
    int store_nt;               // bf16: gradient rows stored non-temporally (see store_row)
};

// Workgroups of one bf16 backward launch: both roles of every block of every unit, in
// groups of 8 units (one per XCD).
__host__ __device__ inline int64_t bwd_bf16_groups(int64_t n_units, int nbb) {
    return 16 * (int64_t)nbb * ((n_units + 7) / 8);
}

// bf16: one workgroup per window for launches whose windows all hold at most 256 tokens
// (pad_blocks = 1); key-role and query-role workgroups per kBwdBlock-token block otherwise
// (pad_blocks = nbb)
hipError_t launch_swin_bwd_bf16_window(const SwinBwdArgs& a, hipStream_t stream);
hipError_t launch_swin_bwd_bf16_blocks(const SwinBwdArgs& a, hipStream_t stream);
hipError_t launch_swin_bwd_f32(const SwinBwdArgs& a, hipStream_t stream);

// Static device scratch of the allocation-free backward: its size, and its device address
// on the current device (taken with hipGetSymbolAddress on the first call per device).
constexpr int64_t kScratchBytes = int64_t(16) << 20;
hipError_t scratch_address(void** ptr);
// sums the partials of ws into row L of dk and dv (elem_bytes 2: bf16, 4: fp32)
hipError_t launch_swin_bwd_pad_reduce(const SwinBwdArgs& a, int elem_bytes, hipStream_t stream);

// Window `win` (numbered over all grids, raster order within a grid), clipped to its grid.
struct WindowRect {
    int y0, x0, rows, cols;
    int W;                      // tokens per row of its grid
    int64_t tok0;               // index of its first token (y0, x0) within a batch entry
};

// MULTI = false: the launch has one grid, and the scan over the grid list (dependent
// kernel-argument loads) is skipped.
template <bool MULTI>
__device__ __forceinline__ WindowRect window_rect(const SwinArgs& a, int win) {
    int g = 0;
    if constexpr (MULTI)
        for (int i = 1; i < kMaxGrids; ++i)
            if (i < a.n_grids && win >= a.grid[i].win_begin) g = i;
    const GridDesc& G = a.grid[g];
    const int lw = win - G.win_begin;
    const int wy = (int)G.div_nwx.div((unsigned)lw);
    const int wx = lw - wy * G.nwx;
    const long long ys = (long long)wy * a.window - a.origin;
    const long long xs = (long long)wx * a.window - a.origin;
    const long long ye = ys + a.window < G.H ? ys + a.window : G.H;
    const long long xe = xs + a.window < G.W ? xs + a.window : G.W;
    WindowRect r;
    r.y0 = ys > 0 ? (int)ys : 0;
    r.x0 = xs > 0 ? (int)xs : 0;
    r.rows = (int)(ye - r.y0);
    r.cols = (int)(xe - r.x0);
    r.W = G.W;
    r.tok0 = G.tok_off + (int64_t)r.y0 * G.W + r.x0;
    return r;
}

}  // namespace fla
