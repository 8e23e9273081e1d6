// Flash Swin attention backward, bf16 storage, gfx950 (CDNA4) matrix cores.
//
// Gradients of Eq. 1 inside each shifted window (the paper trains HRSAM through Flash
// Swin, App. D).  With c = 1/sqrt(d), the log-sum-exp LSE_i kept by the training forward
// and D_i = <dO_i, O_i>:
//   P = exp(c Q K^T - LSE),  dP = dO V^T,  dS = P o (dP - D)
//   dV = P^T dO,  dK = c dS^T Q,  dQ = c dS K
// P is recomputed, never stored.
//
// One launch, two kinds of workgroup (256 threads = 4 waves) per (batch entry, window,
// block of 128 tokens, head):
//   * key role: owns 128 keys of the window.  Wave w keeps the K and V rows of keys
//     32w .. 32w + 31 in registers (MFMA B operands) and accumulates their dK^T and dV^T
//     in registers, while the window's queries stream through LDS in chunks of 128 (Q and
//     dO rows, -D and LSE log2(e) per query).  Per 32-query tile:
//        S = Q K_w^T, dP - D = dO V_w^T - D        (C operand -D)
//        P = exp2(S c log2(e) - LSE log2(e)), dS = P (dP - D), both rounded to bf16
//        dV_w^T += dO^T P, dK_w^T += Q^T dS       (dO^T, Q^T by the transposing LDS read)
//   * query role: owns 128 queries.  Wave w keeps the Q and dO rows of queries 32w .. + 31
//     in registers (B operands), their LSE and D in one register each (a lane holds one
//     query), and accumulates their dQ^T in registers, while the window's keys stream
//     through LDS in chunks of 128 (K and V rows).  Per 32-key tile:
//        S^T = K Q_w^T, dP^T - D = V dO_w^T - D
//        dS^T = P^T o (dP^T - D) in fp32, rounded to bf16
//        dQ_w^T += K^T dS^T                        (K^T by the transposing LDS read)
// No accumulator is shared between waves, so the tile loops run without barriers, and a
// workgroup needs 39 KB of LDS and at most 168 VGPRs: three workgroups (three waves per
// SIMD) share a compute unit, and one's loads run under the others' products.  All the
// workgroups of one (batch entry, window, head) -- both roles of every block -- get ids
// that are equal mod 8, which the dispatcher sends to one XCD one after the other, so the
// window's rows come from HBM once and the other readers find them in that XCD's L2.
//
// Keys past the window's end are zero rows in LDS (query role): their dS multiplies a zero
// K row, and the one partial key tile of a chunk clears their P as well, so no infinity can
// reach the products.  Rows past a window's end are never stored.
//
// RoPE (Sec. 3.1; the training form of the forward's prologue fusion): q and k are rotated
// as they are loaded, and dq, dk are rotated back (the transpose) before rounding; the pad
// token is never rotated.
//
// KV-only padding (Sec. 3.4, App. B): the pad token is one more key of weight n_pad per
// query.  Its terms are rank one per query: the query role adds dS_p k_p to dQ, and key
// block 0's key role sums the pad token's own gradient over the window's queries (P_p and
// dS_p per query in LDS, then one column sum per channel) into the workspace, which a small
// kernel sums over the windows in a fixed order.
#include "fla_swin_device.h"

namespace fla {
namespace {

constexpr int D = kHeadDim;            // 64 channels
constexpr int THREADS = 256;
constexpr int NW = 4;                  // waves
constexpr int TL = 32;                 // keys (key role) or queries (query role) per wave
constexpr int NMAX = kBwdBlock;        // 128 = NW * TL tokens per block and per chunk
constexpr int RPP = THREADS / 8;       // rows staged per pass, 8 threads per 128-byte row
constexpr int RS = D + 8;              // bf16 stride of staged rows (144 B)
static_assert(NW * TL == NMAX && NMAX % RPP == 0, "block geometry");
constexpr float kLog2e = 1.4426950408889634f;

// LDS carve-up, bytes.  Key role: A = Q rows, B = dO rows of the query chunk, L and ND per
// query; pad token: its k and v rows (PADKV), PP and DSP (its P and dS per query of the
// chunk) and PADW (two half sums per channel of its gradient).  Query role: A = K rows, B = V rows of the key chunk,
// the pad token's key row in PADW; A stages the dQ rows at the end.
constexpr int OFF_A = 0;                              // [128][RS] bf16
constexpr int OFF_B = OFF_A + NMAX * RS * 2;          // [128][RS] bf16
constexpr int OFF_L = OFF_B + NMAX * RS * 2;          // LSE * log2(e) [128] fp32
constexpr int OFF_ND = OFF_L + NMAX * 4;              // -D [128] fp32
constexpr int OFF_PP = OFF_ND + NMAX * 4;             // [128] fp32
constexpr int OFF_DSP = OFF_PP + NMAX * 4;            // [128] fp32
constexpr int OFF_PADW = OFF_DSP + NMAX * 4;          // [2][128] fp32
constexpr int OFF_PADKV = OFF_PADW + 2 * kPadPartial * 4;   // pad token's k then v row, [128] bf16
constexpr int LDS_BYTES = OFF_PADKV + kPadPartial * 2;
static_assert(3 * LDS_BYTES <= 160 * 1024, "three workgroups per compute unit");
static_assert(THREADS == 2 * kPadPartial, "two threads per pad-gradient channel");

typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) shortx4 lds_shortx4;

// Transposing LDS read of a 32 x 16 operand: lane l receives column `col0 + (l & 31)` of
// rows row0 + 4 * (l >> 5) + {0..3} and row0 + 8 + 4 * (l >> 5) + {0..3} of a row-major
// bf16 array with row stride `stride`.  Within each 16-lane group, ds_read_b64_tr_b16 has
// lane i name a 4-element piece (row i / 4, elements 4 * (i % 4) .. + 3) of a 4 x 16 block
// and returns to lane i the block's column i.  The row order matches the rows a lane holds
// in the accumulator of a 32 x 32 product, so that accumulator, rounded, is the other
// operand of a product summed over those rows.
__device__ __forceinline__ bf16x8 tr_operand(const uint16_t* base, int stride, int row0, int col0, int lane) {
    const int e = (lane & 15) >> 2, q = lane & 3, g1 = (lane >> 4) & 1, h = lane >> 5;
    const uint16_t* p = base + (row0 + 4 * h + e) * stride + col0 + 16 * g1 + 4 * q;
    const shortx4 va = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_shortx4*)(const_cast<uint16_t*>(p)));
    const shortx4 vb = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_shortx4*)(const_cast<uint16_t*>(p + 8 * stride)));
    const bf16x4 a4 = __builtin_bit_cast(bf16x4, va), b4 = __builtin_bit_cast(bf16x4, vb);
    return bf16x8{a4[0], a4[1], a4[2], a4[3], b4[0], b4[1], b4[2], b4[3]};
}

__device__ __forceinline__ float dot8(const uint4& x, const uint4& y) {
    const bf16x8 a = __builtin_bit_cast(bf16x8, x), b = __builtin_bit_cast(bf16x8, y);
    float s = 0.f;
    for (int e = 0; e < 8; e += 2)
        s = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{a[e], a[e + 1]}, bf16x2{b[e], b[e + 1]}, s, false);
    return s;
}

__device__ __forceinline__ float dot8(const bf16x8& a, const bf16x8& b, float s) {
    for (int e = 0; e < 8; e += 2)
        s = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{a[e], a[e + 1]}, bf16x2{b[e], b[e + 1]}, s, false);
    return s;
}

// sum over the 8 lanes l, l ^ 1, ..., l ^ 7
__device__ __forceinline__ float sum8(float x) {
    x += __shfl_xor(x, 1);
    x += __shfl_xor(x, 2);
    x += __shfl_xor(x, 4);
    return x;
}

// Key role, one tile: the 32 queries whose rows start at q0 (Q, dO rows, -D and LSE*log2(e)
// in LDS) against the wave's 32 keys (kreg, vreg).  dK^T and dV^T add up in registers.
__device__ __forceinline__ void key_tile(const uint16_t* Qs, const uint16_t* dOs, const float* ND, const float* Ls,
                                         const bf16x8 (&kreg)[4], const bf16x8 (&vreg)[4], floatx16 (&dkT)[2],
                                         floatx16 (&dvT)[2], int q0, float c2, int lane) {
    const int li = lane & 31, h = lane >> 5;
    // dP - D in one go: the C operand holds -D of each entry's query
    floatx16 sacc = {}, pacc;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float4 d4 = *reinterpret_cast<const float4*>(ND + q0 + 8 * i + 4 * h);
        pacc[4 * i] = d4.x;
        pacc[4 * i + 1] = d4.y;
        pacc[4 * i + 2] = d4.z;
        pacc[4 * i + 3] = d4.w;
    }
    const uint16_t* qrow = Qs + (q0 + li) * RS + 8 * h;
    const uint16_t* grow = dOs + (q0 + li) * RS + 8 * h;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8*>(qrow + 16 * s), kreg[s],
                                                      sacc, 0, 0, 0);
        pacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8*>(grow + 16 * s), vreg[s],
                                                      pacc, 0, 0, 0);
    }
    // entry r: query q0 + 8 (r / 4) + 4 h + r % 4, the wave's key li
    bf16x8 pb[2], sb[2];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float4 l4 = *reinterpret_cast<const float4*>(Ls + q0 + 8 * i + 4 * h);
        const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = 4 * i + j;
            const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[r], c2, -lv[j]));
            pb[i >> 1][4 * (i & 1) + j] = (__bf16)p;
            sb[i >> 1][4 * (i & 1) + j] = (__bf16)(p * pacc[r]);
        }
    }
#pragma unroll
    for (int sg = 0; sg < 2; ++sg)
#pragma unroll
        for (int dh = 0; dh < 2; ++dh) {
            const bf16x8 ga = tr_operand(dOs, RS, q0 + 16 * sg, 32 * dh, lane);
            const bf16x8 qa = tr_operand(Qs, RS, q0 + 16 * sg, 32 * dh, lane);
            dvT[dh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ga, pb[sg], dvT[dh], 0, 0, 0);
            dkT[dh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa, sb[sg], dkT[dh], 0, 0, 0);
        }
}

// Query role, one tile: the 32 keys whose rows start at k0 (K, V rows in LDS) against the
// wave's 32 queries (qreg, greg; one query per lane column with its -D and LSE*log2(e)).
// dQ^T adds up in registers.  MASKED: keys k0 + j with j >= nvalid get P = 0.
template <bool MASKED>
__device__ __forceinline__ void query_tile(const uint16_t* Ks, const uint16_t* Vs, const bf16x8 (&qreg)[4],
                                           const bf16x8 (&greg)[4], float nd, float l2, floatx16 (&dqT)[2],
                                           int k0, int nvalid, float c2, int lane) {
    const int li = lane & 31, h = lane >> 5;
    floatx16 sacc = {}, pacc;
#pragma unroll
    for (int r = 0; r < 16; ++r) pacc[r] = nd;
    const uint16_t* krow = Ks + (k0 + li) * RS + 8 * h;
    const uint16_t* vrow = Vs + (k0 + li) * RS + 8 * h;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8*>(krow + 16 * s), qreg[s],
                                                      sacc, 0, 0, 0);
        pacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8*>(vrow + 16 * s), greg[s],
                                                      pacc, 0, 0, 0);
    }
    // entry r: key k0 + 8 (r / 4) + 4 h + r % 4, the lane's query li
    bf16x8 sb[2];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[r], c2, -l2));
        if (MASKED && 8 * (r >> 2) + 4 * h + (r & 3) >= nvalid) p = 0.f;
        sb[r >> 3][r & 7] = (__bf16)(p * pacc[r]);
    }
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
        for (int dh = 0; dh < 2; ++dh)
            dqT[dh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_operand(Ks, RS, k0 + 16 * s2, 32 * dh, lane), sb[s2],
                                                             dqT[dh], 0, 0, 0);
}

// What both roles know about their block.
struct Block {
    int b, win, blk, head;
    WindowRect wr;
    int n;                      // tokens of the window
    long long n_pad;            // virtual key slots of its canvas square (KV-token mode)
    WindowAddr addr;
    __amdgpu_buffer_rsrc_t qr, orr, dor, kr, vr, lr;
};

// (row, col) grid coordinates of window-local index t
__device__ __forceinline__ void coords(const Block& k, int t, float& y, float& x) {
    const unsigned r = __umulhi((unsigned)t, k.addr.magic) + ((unsigned)t & k.addr.one_mask);
    y = (float)(k.wr.y0 + (int)r);
    x = (float)(k.wr.x0 + (int)((unsigned)t - r * k.addr.cols));
}

// Key role: a query chunk's rows (rows r0 + RPP u of the 8-thread row groups, zero past the
// chunk's nq rows) -> LDS: Q and dO rows, -D and LSE log2(e) per query.  Every load is issued
// before the first LDS write.  With RoPE each thread then rotates its own pieces of the Q rows
// in place (its LDS writes and reads stay in order), once the loaded registers are free.
template <bool ROPE>
__device__ __forceinline__ void key_stage(const SwinArgs& a, const Block& k, unsigned char* smem, int qbase, int nq) {
    uint16_t* Qs = reinterpret_cast<uint16_t*>(smem + OFF_A);
    uint16_t* dOs = reinterpret_cast<uint16_t*>(smem + OFF_B);
    float* Ls = reinterpret_cast<float*>(smem + OFF_L);
    float* ND = reinterpret_cast<float*>(smem + OFF_ND);
    const int part = threadIdx.x & 7, r0 = threadIdx.x >> 3;
    constexpr int NU = NMAX / RPP;
    uint4 qv[NU], gv[NU], ov[NU];
    float lse_raw[NU];
#pragma unroll
    for (int u = 0; u < NU; ++u) {
        const int r = r0 + RPP * u;
        const unsigned off = r < nq ? k.addr(qbase + r) + 16 * part : kOutside;
        qv[u] = bload16(k.qr, off);
        gv[u] = bload16(k.dor, off);
        ov[u] = bload16(k.orr, off);
        lse_raw[u] = __builtin_bit_cast(
            float, __builtin_amdgcn_raw_buffer_load_b32(
                       k.lr, r < nq ? 4 * k.addr.token(qbase + r, (unsigned)k.wr.W) : kOutside, 0, 0));
    }
#pragma unroll
    for (int u = 0; u < NU; ++u) {
        const int r = r0 + RPP * u;
        *reinterpret_cast<uint4*>(Qs + r * RS + 8 * part) = qv[u];
        *reinterpret_cast<uint4*>(dOs + r * RS + 8 * part) = gv[u];
        const float dd = sum8(dot8(gv[u], ov[u]));
        if (part == 0) {
            ND[r] = -dd;
            Ls[r] = lse_raw[u] * kLog2e;
        }
    }
    if constexpr (ROPE) {
#pragma unroll 1
        for (int u = 0; u < NU; ++u) {
            const int r = r0 + RPP * u;
            float y, x;
            coords(k, min(qbase + r, k.n - 1), y, x);
            uint4* piece = reinterpret_cast<uint4*>(Qs + r * RS + 8 * part);
            *piece = __builtin_bit_cast(uint4, rope_rotate_bf16x8(__builtin_bit_cast(bf16x8, *piece),
                                                                  (part < 4 ? y : x) * a.rope_scale,
                                                                  a.rope_rev + 4 * (part & 3)));
        }
    }
}

// Key role, KV-token mode, after a chunk is staged: the pad token's P and dS per query, two
// threads per row (32 channels each) from the staged Q and dO rows.
__device__ __forceinline__ void key_pad_terms(const SwinArgs& a, unsigned char* smem, int nq, float log2_npad) {
    const uint16_t* Qs = reinterpret_cast<const uint16_t*>(smem + OFF_A);
    const uint16_t* dOs = reinterpret_cast<const uint16_t*>(smem + OFF_B);
    const float* Ls = reinterpret_cast<const float*>(smem + OFF_L);
    const float* ND = reinterpret_cast<const float*>(smem + OFF_ND);
    float* PP = reinterpret_cast<float*>(smem + OFF_PP);
    float* DSP = reinterpret_cast<float*>(smem + OFF_DSP);
    const uint16_t* PADKV = reinterpret_cast<const uint16_t*>(smem + OFF_PADKV);
    static_assert(THREADS == 2 * NMAX, "two threads per staged row");
    const int r = threadIdx.x >> 1, half = threadIdx.x & 1;
    float zp = 0.f, dp = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int c = 32 * half + 8 * j;
        zp = dot8(*reinterpret_cast<const bf16x8*>(Qs + r * RS + c), *reinterpret_cast<const bf16x8*>(PADKV + c), zp);
        dp = dot8(*reinterpret_cast<const bf16x8*>(dOs + r * RS + c), *reinterpret_cast<const bf16x8*>(PADKV + D + c),
                  dp);
    }
    zp += __shfl_xor(zp, 1);
    dp += __shfl_xor(dp, 1);
    // P = n_pad exp(c <q, k_pad> - LSE), dS = P (<dO, v_pad> - D)
    const float p = r < nq ? __builtin_amdgcn_exp2f(__builtin_fmaf(zp, a.scale_log2, log2_npad - Ls[r])) : 0.f;
    if (half == 0) {
        PP[r] = p;
        DSP[r] = p * (dp + ND[r]);
    }
}

template <bool KVPAD, bool ROPE>
__device__ __forceinline__ void key_role(const SwinBwdArgs& ba, const Block& k, unsigned char* smem) {
    const SwinArgs& a = ba.f;
    uint16_t* Qs = reinterpret_cast<uint16_t*>(smem + OFF_A);
    uint16_t* dOs = reinterpret_cast<uint16_t*>(smem + OFF_B);
    float* Ls = reinterpret_cast<float*>(smem + OFF_L);
    float* ND = reinterpret_cast<float*>(smem + OFF_ND);
    float* PP = reinterpret_cast<float*>(smem + OFF_PP);
    float* DSP = reinterpret_cast<float*>(smem + OFF_DSP);
    float* PADW = reinterpret_cast<float*>(smem + OFF_PADW);
    const int tid = threadIdx.x, lane = tid & 63, li = lane & 31, h = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const long long e = (((long long)k.b * a.heads + k.head) * a.n_windows + k.win) * ba.nbb + k.blk;
    const int key0 = NMAX * k.blk;
    if (key0 >= k.n) {   // the window has fewer blocks; its pad partial is still read
        if (KVPAD && tid < kPadPartial) ba.ws[e * kPadPartial + tid] = 0.f;
        return;
    }
    const int nkeys = min(NMAX, k.n - key0);
    const int nkt = (nkeys + TL - 1) / TL;
    const bool pad_here = KVPAD && k.n_pad > 0 && k.blk == 0;

    // K_w and V_w rows: lane holds key key0 + 32 wave + li, channels 16 s + 8 h .. + 7
    const int key = TL * wave + li;
    const unsigned krow = key < nkeys ? k.addr(key0 + key) : kOutside;
    bf16x8 kreg[4], vreg[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        kreg[s] = __builtin_bit_cast(bf16x8, bload16(k.kr, krow + 32 * s + 16 * h));
        vreg[s] = __builtin_bit_cast(bf16x8, bload16(k.vr, krow + 32 * s + 16 * h));
    }
    if constexpr (ROPE) {
        float y, x;
        coords(k, min(key0 + key, k.n - 1), y, x);
#pragma unroll
        for (int s = 0; s < 4; ++s)
            kreg[s] = rope_rotate_bf16x8(kreg[s], (s < 2 ? y : x) * a.rope_scale, a.rope_rev + 8 * (s & 1) + 4 * h);
    }
    // pad token's key and value rows: loaded with the first chunk, kept in LDS (PADKV)
    const int part = tid & 7;
    uint4 padrow = {0u, 0u, 0u, 0u};
    if (pad_here && tid < 16) {
        const long long pad_elems = (long long)k.b * a.kv_batch_stride + a.L * a.tok_stride + k.head * D;
        const __amdgpu_buffer_rsrc_t pr = make_rsrc(static_cast<const uint16_t*>(tid < 8 ? a.k : a.v) + pad_elems, D * 2);
        padrow = bload16(pr, 16 * part);
    }
    float pad_sum = 0.f;   // thread (half, channel): its half of the chunk rows, over the chunks
    const float c2 = a.scale_log2;
    const float log2_npad = pad_here ? log2f((float)k.n_pad) : 0.f;
    floatx16 dkT[2] = {floatx16{}, floatx16{}}, dvT[2] = {floatx16{}, floatx16{}};

    const int nqc = (k.n + NMAX - 1) / NMAX;
    for (int qc = 0; qc < nqc; ++qc) {
        const int qbase = NMAX * qc;
        const int nq = min(NMAX, k.n - qbase);
        const int nqt = (nq + TL - 1) / TL;
        if (qc > 0) __syncthreads();   // every wave is done with the previous chunk's rows
        // ---- the chunk's Q, dO rows -> LDS, -D and LSE log2(e) per query
        key_stage<ROPE>(a, k, smem, qbase, nq);
        if (pad_here && qc == 0 && tid < 16)
            *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(smem + OFF_PADKV) + 8 * tid) = padrow;
        __syncthreads();
        if (pad_here) {
            key_pad_terms(a, smem, nq, log2_npad);
            __syncthreads();
            // the pad token's gradient over this chunk's rows: thread (half, c) sums channel c of
            // dS_p q (c < 64) or P_p dO (c >= 64) over rows half * 64 .. + 63, in row order
            // (four interleaved partial sums, added in a fixed order: rows past nq have P = dS = 0)
            const int c = tid & (kPadPartial - 1), half = tid / kPadPartial;
            const float* w = c < D ? DSP : PP;
            const uint16_t* col = (c < D ? Qs : dOs) + (c & (D - 1));
            float acc4[4] = {0.f, 0.f, 0.f, 0.f};
            const int r_begin = NMAX / 2 * half;
#pragma unroll 4
            for (int i = 0; i < NMAX / 2; i += 4)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int r = r_begin + i + j;
                    acc4[j] = __builtin_fmaf(w[r], __uint_as_float((unsigned)col[r * RS] << 16), acc4[j]);
                }
            pad_sum += (acc4[0] + acc4[1]) + (acc4[2] + acc4[3]);
        }
        // ---- tiles: the wave's keys against each query tile of the chunk (starting at a
        //      different tile per wave, to spread the LDS reads)
        if (wave < nkt) {
            int T = wave < nqt ? wave : wave % nqt;
            for (int t = 0; t < nqt; ++t) {
                key_tile(Qs, dOs, ND, Ls, kreg, vreg, dkT, dvT, TL * T, c2, lane);
                T = T + 1 == nqt ? 0 : T + 1;
            }
        }
    }
    if (pad_here) PADW[tid] = pad_sum;
    __syncthreads();   // the rows are free for staging; the pad sums are complete

    if (KVPAD && tid < kPadPartial) {
        // every block writes its share (zero without virtual slots or past block 0), so the
        // reduction reads a dense array
        const float acc = pad_here ? PADW[tid] + PADW[kPadPartial + tid] : 0.f;
        ba.ws[e * kPadPartial + tid] = tid < D ? acc * ba.scale : acc;
    }

    // ---- dK, dV of the wave's keys: stage its 32 rows in the Q and dO rows, store whole
    //      128-byte rows, 8 lanes per row
    if (wave < nkt) {
        const float sc = ba.scale;
        if constexpr (ROPE) {
            // dk = R^T dk': this lane's key, channels 32 dh + 8 i + 4 h + {0..3} = pairs
            // 4 i + 2 h + {0, 1} of half dh
            float y, x;
            coords(k, min(key0 + key, k.n - 1), y, x);
#pragma unroll
            for (int dh = 0; dh < 2; ++dh)
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int pr = 0; pr < 2; ++pr) {
                        float p0 = dkT[dh][4 * i + 2 * pr], p1 = dkT[dh][4 * i + 2 * pr + 1];
                        rope_unrotate_pair(p0, p1, (dh == 0 ? y : x) * a.rope_scale, a.rope_rev[4 * i + 2 * h + pr]);
                        dkT[dh][4 * i + 2 * pr] = p0;
                        dkT[dh][4 * i + 2 * pr + 1] = p1;
                    }
        }
        uint16_t* krow_s = Qs + (TL * wave + li) * RS;
        uint16_t* vrow_s = dOs + (TL * wave + li) * RS;
#pragma unroll
        for (int dh = 0; dh < 2; ++dh)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                bf16x4 k4, v4;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    k4[j] = (__bf16)(dkT[dh][4 * i + j] * sc);
                    v4[j] = (__bf16)dvT[dh][4 * i + j];
                }
                *reinterpret_cast<bf16x4*>(krow_s + 32 * dh + 8 * i + 4 * h) = k4;
                *reinterpret_cast<bf16x4*>(vrow_s + 32 * dh + 8 * i + 4 * h) = v4;
            }
        asm volatile("" ::: "memory");   // staged rows are read back by other lanes of the wave
        const long long kv_base = (long long)k.b * a.kv_batch_stride + k.wr.tok0 * a.tok_stride + k.head * D;
        const long long kv_bytes = ((long long)a.B * a.kv_batch_stride - kv_base) * 2;
        const __amdgpu_buffer_rsrc_t dkr = make_rsrc(static_cast<uint16_t*>(ba.dk) + kv_base, kv_bytes);
        const __amdgpu_buffer_rsrc_t dvr = make_rsrc(static_cast<uint16_t*>(ba.dv) + kv_base, kv_bytes);
        const int sp = lane & 7;
#pragma unroll
        for (int it = 0; it < TL / 8; ++it) {
            const int rl = TL * wave + 8 * it + (lane >> 3);
            const unsigned off = rl < nkeys ? k.addr(key0 + rl) + 16 * sp : kOutside;
            const uint4 kx = *reinterpret_cast<const uint4*>(Qs + rl * RS + 8 * sp);
            const uint4 vx = *reinterpret_cast<const uint4*>(dOs + rl * RS + 8 * sp);
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, kx), dkr, off, 0, 0);
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, vx), dvr, off, 0, 0);
        }
    }
}

template <bool KVPAD, bool ROPE>
__device__ __forceinline__ void query_role(const SwinBwdArgs& ba, const Block& k, unsigned char* smem) {
    const SwinArgs& a = ba.f;
    uint16_t* Ks = reinterpret_cast<uint16_t*>(smem + OFF_A);
    uint16_t* Vs = reinterpret_cast<uint16_t*>(smem + OFF_B);
    float* KP = reinterpret_cast<float*>(smem + OFF_PADW);
    const int tid = threadIdx.x, lane = tid & 63, li = lane & 31, h = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int q0 = NMAX * k.blk;
    if (q0 >= k.n) return;
    const int nq = min(NMAX, k.n - q0);
    const bool has_pad = KVPAD && k.n_pad > 0;

    // Q_w and dO_w (B operands): lane holds query q0 + 32 wave + li, channels 16 s + 8 h .. + 7;
    // O only for D = <dO, O>, and the query's LSE.  The first key chunk's loads go out with
    // them; each later chunk's are issued before the tiles of the one before (kv, vv).
    const int qi = TL * wave + li;
    const bool q_ok = qi < nq;
    const unsigned qrow = q_ok ? k.addr(q0 + qi) : kOutside;
    const int part = tid & 7, r0 = tid >> 3;
    const int nkc = (k.n + NMAX - 1) / NMAX;
    uint4 kv[NMAX / RPP], vv[NMAX / RPP];
    auto load_chunk = [&](int kbase) {
        const int nk = min(NMAX, k.n - kbase);
#pragma unroll
        for (int u = 0; u < NMAX / RPP; ++u) {
            const int r = r0 + RPP * u;
            const unsigned off = r < nk ? k.addr(kbase + r) + 16 * part : kOutside;
            kv[u] = bload16(k.kr, off);
            vv[u] = bload16(k.vr, off);
        }
    };
    bf16x8 qreg[4], greg[4];
    uint4 oreg[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        qreg[s] = __builtin_bit_cast(bf16x8, bload16(k.qr, qrow + 32 * s + 16 * h));
        greg[s] = __builtin_bit_cast(bf16x8, bload16(k.dor, qrow + 32 * s + 16 * h));
        oreg[s] = bload16(k.orr, qrow + 32 * s + 16 * h);
    }
    load_chunk(0);
    float dd = 0.f;
#pragma unroll
    for (int s = 0; s < 4; ++s) dd = dot8(greg[s], __builtin_bit_cast(bf16x8, oreg[s]), dd);
    const float l2 = __builtin_bit_cast(
                         float, __builtin_amdgcn_raw_buffer_load_b32(
                                    k.lr, q_ok ? 4 * k.addr.token(q0 + qi, (unsigned)k.wr.W) : kOutside, 0, 0)) *
                     kLog2e;
    dd = xhalf_sum(dd);
    const float c2 = a.scale_log2;
    [[maybe_unused]] float qy = 0.f, qx = 0.f;
    if constexpr (ROPE) {
        coords(k, min(q0 + qi, k.n - 1), qy, qx);
#pragma unroll
        for (int s = 0; s < 4; ++s)
            qreg[s] = rope_rotate_bf16x8(qreg[s], (s < 2 ? qy : qx) * a.rope_scale, a.rope_rev + 8 * (s & 1) + 4 * h);
    }
    // pad token as key: dS_p = n_pad exp(c <q, k_pad> - LSE) (<dO, v_pad> - D); dq gets dS_p k_pad
    float dsp = 0.f;
    if (has_pad) {
        const long long pad_elems = (long long)k.b * a.kv_batch_stride + a.L * a.tok_stride + k.head * D;
        const __amdgpu_buffer_rsrc_t kpr = make_rsrc(static_cast<const uint16_t*>(a.k) + pad_elems, D * 2);
        const __amdgpu_buffer_rsrc_t vpr = make_rsrc(static_cast<const uint16_t*>(a.v) + pad_elems, D * 2);
        float zp = 0.f, dp = 0.f;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            zp = dot8(qreg[s], __builtin_bit_cast(bf16x8, bload16(kpr, 32 * s + 16 * h)), zp);
            dp = dot8(greg[s], __builtin_bit_cast(bf16x8, bload16(vpr, 32 * s + 16 * h)), dp);
        }
        zp = xhalf_sum(zp);
        dp = xhalf_sum(dp);
        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(zp, c2, log2f((float)k.n_pad) - l2));
        dsp = p * (dp - dd);
        if (tid < 8) {
            const bf16x8 k8 = __builtin_bit_cast(bf16x8, bload16(kpr, 16 * tid));
            for (int j = 0; j < 8; ++j) KP[8 * tid + j] = (float)k8[j];
        }
    }
    const float nd = -dd;

    floatx16 dqT[2] = {floatx16{}, floatx16{}};
    for (int kc = 0; kc < nkc; ++kc) {
        const int kbase = NMAX * kc;
        const int nk = min(NMAX, k.n - kbase);
        const int nkt = (nk + TL - 1) / TL;
        // ---- the chunk's K, V rows (zero past its end) -> LDS, 8 threads per row
        if (kc > 0) __syncthreads();   // every wave is done with the previous chunk's rows
#pragma unroll
        for (int u = 0; u < NMAX / RPP; ++u) {
            const int r = r0 + RPP * u;
            if constexpr (ROPE) {
                float y, x;
                coords(k, min(kbase + r, k.n - 1), y, x);
                kv[u] = __builtin_bit_cast(uint4, rope_rotate_bf16x8(__builtin_bit_cast(bf16x8, kv[u]),
                                                                     (part < 4 ? y : x) * a.rope_scale,
                                                                     a.rope_rev + 4 * (part & 3)));
            }
            *reinterpret_cast<uint4*>(Ks + r * RS + 8 * part) = kv[u];
            *reinterpret_cast<uint4*>(Vs + r * RS + 8 * part) = vv[u];
        }
        if (kc + 1 < nkc) load_chunk(kbase + NMAX);   // in flight during this chunk's tiles
        __syncthreads();
        // ---- tiles: the wave's queries against each key tile of the chunk; only a partial
        //      last tile masks its missing keys
        if (TL * wave < nq) {
            const int full = nk / TL;
            int T = wave < full ? wave : (full > 0 ? wave % full : 0);
            for (int t = 0; t < full; ++t) {
                query_tile<false>(Ks, Vs, qreg, greg, nd, l2, dqT, TL * T, TL, c2, lane);
                T = T + 1 == full ? 0 : T + 1;
            }
            if (full < nkt) query_tile<true>(Ks, Vs, qreg, greg, nd, l2, dqT, TL * full, nk - TL * full, c2, lane);
        }
    }
    __syncthreads();   // the K rows are free for staging

    // ---- dQ of the wave's queries: + dS_p k_pad, rotate back, scale, round; stage the 32 rows
    //      in the K rows and store whole 128-byte rows, 8 lanes per row.  dqT[dh] entry r:
    //      channel 32 dh + 8 (r / 4) + 4 h + r % 4 of the lane's query.
    if (TL * wave < nq) {
        const float sc = ba.scale;
        uint16_t* row_s = Ks + (TL * wave + li) * RS;
#pragma unroll
        for (int dh = 0; dh < 2; ++dh)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int ch = 32 * dh + 8 * i + 4 * h;
                float v4[4] = {dqT[dh][4 * i], dqT[dh][4 * i + 1], dqT[dh][4 * i + 2], dqT[dh][4 * i + 3]};
                if (has_pad)
#pragma unroll
                    for (int j = 0; j < 4; ++j) v4[j] = __builtin_fmaf(dsp, KP[ch + j], v4[j]);
                if constexpr (ROPE) {
                    // dq = R^T dq': pairs (ch % 32) / 2 + {0, 1} of half dh
                    const float pos = (dh == 0 ? qy : qx) * a.rope_scale;
                    rope_unrotate_pair(v4[0], v4[1], pos, a.rope_rev[4 * i + 2 * h]);
                    rope_unrotate_pair(v4[2], v4[3], pos, a.rope_rev[4 * i + 2 * h + 1]);
                }
                bf16x4 o4;
#pragma unroll
                for (int j = 0; j < 4; ++j) o4[j] = (__bf16)(v4[j] * sc);
                *reinterpret_cast<bf16x4*>(row_s + ch) = o4;
            }
        asm volatile("" ::: "memory");   // staged rows are read back by other lanes of the wave
        const long long q_base = (long long)k.b * a.q_batch_stride + k.wr.tok0 * a.tok_stride + k.head * D;
        const __amdgpu_buffer_rsrc_t dqr =
            make_rsrc(static_cast<uint16_t*>(ba.dq) + q_base, ((long long)a.B * a.q_batch_stride - q_base) * 2);
        const int sp = lane & 7;
#pragma unroll
        for (int it = 0; it < TL / 8; ++it) {
            const int rl = TL * wave + 8 * it + (lane >> 3);
            const unsigned off = rl < nq ? k.addr(q0 + rl) + 16 * sp : kOutside;
            const uint4 qx4 = *reinterpret_cast<const uint4*>(Ks + rl * RS + 8 * sp);
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, qx4), dqr, off, 0, 0);
        }
    }
}

// Workgroup id -> (unit, role, block), unit = (batch entry, window, head): the 2 nbb
// workgroups of unit u (both roles of each of its nbb blocks) get ids
// 8 (2 nbb (u / 8) + j) + u % 8, j = 2 block + role, all on XCD u % 8 and dispatched
// one after the other there.  Units are numbered heads fastest, then windows, then batch
// entries.
template <bool MULTI, bool KVPAD, bool ROPE>
__global__ __launch_bounds__(THREADS) __attribute__((amdgpu_waves_per_eu(3, 3)))
void swin_bwd_bf16_kernel(SwinBwdArgs ba) {
    const SwinArgs& a = ba.f;
    __shared__ __attribute__((aligned(16))) unsigned char smem[LDS_BYTES];
    const unsigned id = blockIdx.x;
    const unsigned rest = id >> 3;
    const unsigned g = ba.div_2nbb.div(rest);
    const unsigned j = rest - g * (2u * (unsigned)ba.nbb);
    const unsigned unit = (g << 3) + (id & 7u);
    if (unit >= (unsigned)ba.n_units) return;
    const bool query = j & 1u;

    Block k;
    k.blk = (int)(j >> 1);
    const unsigned i2 = a.div_heads.div(unit);
    k.head = (int)(unit - i2 * (unsigned)a.heads);
    const unsigned i3 = a.div_nwin.div(i2);
    k.win = (int)(i2 - i3 * (unsigned)a.n_windows);
    k.b = (int)i3;
    k.wr = window_rect<MULTI>(a, k.win);
    k.n = k.wr.rows * k.wr.cols;
    k.n_pad = (long long)a.window * a.window - k.n;

    // buffer resources at the window's first token, head `head`
    const long long win_elems = k.wr.tok0 * a.tok_stride + k.head * D;
    const long long q_base = (long long)k.b * a.q_batch_stride + win_elems;
    const long long kv_base = (long long)k.b * a.kv_batch_stride + win_elems;
    const long long q_bytes = ((long long)a.B * a.q_batch_stride - q_base) * 2;
    const long long kv_bytes = ((long long)a.B * a.kv_batch_stride - kv_base) * 2;
    k.qr = make_rsrc(static_cast<const uint16_t*>(a.q) + q_base, q_bytes);
    k.orr = make_rsrc(static_cast<const uint16_t*>(ba.out) + q_base, q_bytes);
    k.dor = make_rsrc(static_cast<const uint16_t*>(ba.dout) + q_base, q_bytes);
    k.kr = make_rsrc(static_cast<const uint16_t*>(a.k) + kv_base, kv_bytes);
    k.vr = make_rsrc(static_cast<const uint16_t*>(a.v) + kv_base, kv_bytes);
    const long long lse_base = ((long long)k.b * a.heads + k.head) * a.L + k.wr.tok0;
    const long long lse_total = (long long)a.B * a.heads * a.L;
    k.lr = make_rsrc(ba.lse + lse_base, (lse_total - lse_base) * 4);
    k.addr.init(k.wr.cols, (unsigned)((long long)k.wr.W * a.tok_stride * 2), (unsigned)(a.tok_stride * 2));

    if (query)
        query_role<KVPAD, ROPE>(ba, k, smem);
    else
        key_role<KVPAD, ROPE>(ba, k, smem);
}

}  // namespace

hipError_t launch_swin_bwd_bf16(const SwinBwdArgs& a, hipStream_t stream) {
    SwinBwdArgs args = a;
    void* params[] = {&args};
    const bool multi = a.f.n_grids > 1, kv = a.f.pad_mode == 1;
    const void* fn;
    if (a.f.rope)   // RoPE: single grid only (the host admits no grid list with it)
        fn = kv ? reinterpret_cast<const void*>(&swin_bwd_bf16_kernel<false, true, true>)
                : reinterpret_cast<const void*>(&swin_bwd_bf16_kernel<false, false, true>);
    else
        fn = multi ? (kv ? reinterpret_cast<const void*>(&swin_bwd_bf16_kernel<true, true, false>)
                         : reinterpret_cast<const void*>(&swin_bwd_bf16_kernel<true, false, false>))
                   : (kv ? reinterpret_cast<const void*>(&swin_bwd_bf16_kernel<false, true, false>)
                         : reinterpret_cast<const void*>(&swin_bwd_bf16_kernel<false, false, false>));
    return hipLaunchKernel(fn, dim3((unsigned)bwd_bf16_groups(a.n_units, a.nbb)), dim3(THREADS), params, 0, stream);
}

}  // namespace fla
