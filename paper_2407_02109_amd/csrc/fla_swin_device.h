// Device-side helpers shared by the gfx950 kernels: vector types, buffer-resource
// addressing and the window-local token decode.
#pragma once

#include "fla_swin_internal.h"

namespace fla {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef int v2i __attribute__((ext_vector_type(2)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// max / sum over lanes l and l ^ 32 (the two halves holding the same query column)
__device__ __forceinline__ float xhalf_max(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xhalf_sum(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// ---- global memory through buffer resources: 32-bit byte offsets from the window's first
//      token, and hardware range checks (a load outside the resource returns 0, a store
//      outside it is dropped), so no access can leave the tensor it belongs to.
constexpr unsigned kOutside = 0x80000000u;   // offset that is always out of range
constexpr int kMaxRecords = 0x7fffffff;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, long long bytes) {
    const int n = bytes < kMaxRecords ? (int)bytes : kMaxRecords;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}

// A 16-byte row piece of a result, with the non-temporal cache policy (NT) or the ordinary one.
// The backward stores its gradients non-temporally when the call's bytes fit the last-level
// cache: the next call then finds its inputs still there (at 64x64 tokens 11% faster); beyond
// that cache ordinary stores measured ~2% faster.  The caller picks NT once per workgroup
// (with_store_policy), so the store loop has no branch.
template <bool NT>
__device__ __forceinline__ void store_row(u32x4 v, __amdgpu_buffer_rsrc_t r, unsigned off) {
    __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, NT ? 2 : 0);
}
template <typename F>
__device__ __forceinline__ void with_store_policy(bool nt, F&& f) {
    if (nt)
        f(std::integral_constant<bool, true>{});
    else
        f(std::integral_constant<bool, false>{});
}

__device__ __forceinline__ uint4 bload16(__amdgpu_buffer_rsrc_t r, unsigned off) {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

// Byte offset of window-local index t (t = row * cols + col, row-major in the window's
// rectangle) from the window's first token.  row = t / cols is a multiply-high by
// ceil(2^32 / cols), exact for t * cols < 2^32 (the host guarantees n * cols <= 2^32);
// cols == 1 uses magic 0 and adds t through one_mask.
struct WindowAddr {
    unsigned row_bytes;   // bytes between grid rows: W * heads * head_dim * 2
    unsigned tok_bytes;   // bytes between adjacent tokens of a row: heads * head_dim * 2
    unsigned magic, one_mask, cols;

    __host__ __device__ __forceinline__ void init(int c, unsigned rowb, unsigned tokb) {
        cols = (unsigned)c;
        magic = c > 1 ? 0xffffffffu / (unsigned)c + 1u : 0u;   // ceil(2^32 / c), a 32-bit division
        one_mask = c > 1 ? 0u : 0xffffffffu;
        row_bytes = rowb;
        tok_bytes = tokb;
    }
    __host__ __device__ __forceinline__ unsigned operator()(int t) const {
        const unsigned r = mulhi_u32((unsigned)t, magic) + ((unsigned)t & one_mask);
        const unsigned c = (unsigned)t - r * cols;
        return r * row_bytes + c * tok_bytes;
    }
    // tokens from the window's first token to window-local index t, for a grid W wide
    __host__ __device__ __forceinline__ unsigned token(int t, unsigned W) const {
        const unsigned r = mulhi_u32((unsigned)t, magic) + ((unsigned)t & one_mask);
        return r * W + ((unsigned)t - r * cols);
    }
};

// ---- rotary position embedding (RoPE) on bf16 channel pairs, for kernels without a
//      per-window cos / sin table.  cos and sin of the angle pos * rev revolutions come from
//      v_cos_f32 / v_sin_f32 after reducing it to [-1/2, 1/2] revolution.
__device__ __forceinline__ float2 rope_cs(float pos, float rev) {
    float t = pos * rev;
    t -= __builtin_rintf(t);
    return make_float2(__builtin_amdgcn_cosf(t), __builtin_amdgcn_sinf(t));
}

// Rotate the 4 channel pairs of 8 consecutive bf16 channels by pos * rev[i] (in fp32,
// rounded back to bf16).
__device__ __forceinline__ bf16x8 rope_rotate_bf16x8(bf16x8 x, float pos, const float* rev) {
    bf16x8 r;
    for (int i = 0; i < 4; ++i) {
        const float2 cs = rope_cs(pos, rev[i]);
        const float a = (float)x[2 * i], b = (float)x[2 * i + 1];
        r[2 * i] = (__bf16)(a * cs.x - b * cs.y);
        r[2 * i + 1] = (__bf16)(b * cs.x + a * cs.y);
    }
    return r;
}

// The transpose of that rotation on one fp32 channel pair (a, b) (used on gradients).
__device__ __forceinline__ void rope_unrotate_pair(float& a, float& b, float pos, float rev) {
    const float2 cs = rope_cs(pos, rev);
    const float ra = a * cs.x + b * cs.y, rb = b * cs.x - a * cs.y;
    a = ra;
    b = rb;
}

}  // namespace fla
