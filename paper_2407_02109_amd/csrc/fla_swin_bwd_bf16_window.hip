// Flash Swin attention backward, bf16 storage, gfx950 (CDNA4) matrix cores: the kernel for
// launches whose windows all hold at most 256 tokens (window <= 16 covers every grid).
//
// Gradients of Eq. 1 inside each shifted window (the paper trains HRSAM through Flash
// Swin, App. D).  With c = 1/sqrt(d), the log-sum-exp LSE_i kept by the training forward
// and D_i = <dO_i, O_i>:
//   P = exp(c Q K^T - LSE),  dP = dO V^T,  dS = P o (dP - D)
//   dV = P^T dO,  dK = c dS^T Q,  dQ = c dS K
// P is recomputed, never stored.  One workgroup takes a whole (batch entry, window, head),
// so no gradient leaves it half done.  Wider windows take the block kernel of
// fla_swin_bwd_bf16_blocks.hip.
//
// Per workgroup (512 threads = 8 waves):
//   1. Q, dO and K rows of the window -> LDS (row-major, 144-byte rows); LSE and D per query
//      -> LDS (D from the dO and O rows as they arrive).  Wave w owns keys [32w, 32w + 32):
//      its K and V rows also stay in registers as MFMA operands.  Wave w owns query tile w
//      as well: it keeps that tile's dQ^T accumulator in registers.
//   2. Steps t = 0 .. nt-1 (nt = ceil(n / 32) query tiles = key tiles): wave w works on
//      query tile (w + t) mod nt, so at every step each tile belongs to exactly one wave.
//        S = Q K_w^T and dP = dO V_w^T      (v_mfma_f32_32x32x16_bf16, fp32 accumulation;
//                                             each lane holds one key and 16 queries)
//        P = exp2(S c log2(e) - LSE log2(e)), dS = P (dP - D) in fp32, rounded to bf16
//        dV_w^T += dO^T P,  dK_w^T += Q^T dS  (dO^T and Q^T come straight from the LDS
//                                             rows by transposing reads)
//      and hands its dS^T tile over through LDS (two buffers, by step parity).  In step t + 1
//      the owner of that query tile adds its share, dQ^T += K^T dS^T, with K^T read from the
//      K rows by the gfx950 transposing read (ds_read_b64_tr_b16).  A hand-off moves 8 KB
//      per step and wave (bf16 dS^T written and read, K^T read), where passing an fp32 dQ^T
//      accumulator between waves would move 16 KB: the steps are bound by LDS traffic.
//      The matrix cores do the bookkeeping adds as well: keys past the window's end get -inf
//      through the C operand of S (so P = 0), and -D enters as the C operand of dP.  One
//      barrier per step orders the hand-offs; every dQ^T sums its key tiles in step order.
//   3. Epilogue: scale, round to bf16 (RNE), stage each wave's 32 rows of dK, dV and dQ in
//      LDS and store whole 128-byte rows at their own tokens.
//
// RoPE (Sec. 3.1; the training form of the forward's prologue fusion): q and K rows are
// rotated as they are loaded, and dq, dk are rotated back (the transpose) before rounding;
// the pad token is never rotated.
//
// KV-only padding (Sec. 3.4, App. B): the pad token is one more key of weight n_pad per
// query.  Its terms are rank one per query, so they are done during staging: its dS joins
// dQ in the epilogue, and the workgroup's share of the pad token's own gradient goes to
// the workspace, which a small kernel sums over the windows in a fixed order.
#include "fla_swin_device.h"

namespace fla {
namespace {

constexpr int D = kHeadDim;            // 64 channels
constexpr int THREADS = 512;
constexpr int NW = 8;                  // waves
constexpr int TL = 32;                 // keys per wave = queries per tile
constexpr int NMAX = 256;              // tokens of the largest window = NW * TL
constexpr int RS = D + 8;              // bf16 stride of Q / dO / staging rows (144 B)
constexpr int SS = TL + 4;             // bf16 stride of the dS^T hand-off rows (72 B)
constexpr float kLog2e = 1.4426950408889634f;

// LDS carve-up, bytes
// (LSE and D first, then Q and dO: every access the steps make to them is within reach of
// the 16-bit immediate offset of an LDS instruction from one base register)
constexpr int OFF_LSE = 0;                             // LSE * log2(e) [256] fp32
constexpr int OFF_DD = OFF_LSE + NMAX * 4;             // D            [256] fp32
constexpr int OFF_Q = OFF_DD + NMAX * 4;               // Q rows       [256][RS] bf16
constexpr int OFF_DO = OFF_Q + NMAX * RS * 2;          // dO rows      [256][RS] bf16
constexpr int OFF_DSP = OFF_DO + NMAX * RS * 2;        // pad-token dS [256] fp32
constexpr int OFF_KP = OFF_DSP + NMAX * 4;             // pad-token key row [64] fp32
constexpr int OFF_DST = OFF_KP + D * 4;                // dS^T hand-off [2][wave][32][SS] bf16
constexpr int OFF_K = OFF_DST + 2 * NW * TL * SS * 2;  // K rows       [256][RS] bf16
constexpr int LDS_BYTES = OFF_K + NMAX * RS * 2;
static_assert(LDS_BYTES <= 160 * 1024, "LDS budget of one workgroup");
static_assert(NW * kPadPartial * 4 <= NW * TL * SS * 2, "pad partials fit in the dS^T hand-off area");

typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) shortx4 lds_shortx4;

// Transposing LDS read of a 32 x 16 operand: lane l receives column `col0 + (l & 31)` of
// rows row0 + 4 * (l >> 5) + {0..3} and row0 + 8 + 4 * (l >> 5) + {0..3} of a row-major
// bf16 array with row stride `stride`.  Within each 16-lane group, ds_read_b64_tr_b16 has
// lane i name a 4-element piece (row i / 4, elements 4 * (i % 4) .. + 3) of a 4 x 16 block
// and returns to lane i the block's column i.
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

// sum over the 8 lanes l, l ^ 1, ..., l ^ 7
__device__ __forceinline__ float sum8(float x) {
    x += __shfl_xor(x, 1);
    x += __shfl_xor(x, 2);
    x += __shfl_xor(x, 4);
    return x;
}

// One step of a wave: the query tile whose rows start at q0 (Q, dO rows, -D and LSE*log2(e)
// in LDS) against the wave's 32 keys (kreg, vreg in registers).  dK^T and dV^T add up in
// registers; the tile's dS^T goes to the wave's hand-off buffer `dst`, from which the wave
// that owns the query tile takes its dQ^T share after the step's barrier.
__device__ __forceinline__ void wave_step(const uint16_t* Qs, const uint16_t* dOs, const float* Ds, const float* Ls,
                                          uint16_t* dst, const bf16x8 (&kreg)[4], const bf16x8 (&vreg)[4],
                                          const floatx16& s_init, floatx16 (&dkT)[2], floatx16 (&dvT)[2], int q0,
                                          float c2, int lane) {
    const int li = lane & 31, h = lane >> 5;
    // dP - D in one go: the MFMA's C operand holds -D of each entry's query
    floatx16 sacc = s_init, pacc;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float4 d4 = *reinterpret_cast<const float4*>(Ds + q0 + 8 * i + 4 * h);
        pacc[4 * i] = d4.x;
        pacc[4 * i + 1] = d4.y;
        pacc[4 * i + 2] = d4.z;
        pacc[4 * i + 3] = d4.w;
    }
    const uint16_t* qrow = Qs + (q0 + li) * RS + 8 * h;
    const uint16_t* grow = dOs + (q0 + li) * RS + 8 * h;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8*>(qrow + 16 * s),
                                                      kreg[s], sacc, 0, 0, 0);
        pacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8*>(grow + 16 * s),
                                                      vreg[s], pacc, 0, 0, 0);
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
            const float ds = p * pacc[r];
            pb[i >> 1][4 * (i & 1) + j] = (__bf16)p;
            sb[i >> 1][4 * (i & 1) + j] = (__bf16)ds;
        }
    }
    // dV^T += dO^T P, dK^T += Q^T dS
#pragma unroll
    for (int sg = 0; sg < 2; ++sg)
#pragma unroll
        for (int dh = 0; dh < 2; ++dh) {
            const bf16x8 ga = tr_operand(dOs, RS, q0 + 16 * sg, 32 * dh, lane);
            const bf16x8 qa = tr_operand(Qs, RS, q0 + 16 * sg, 32 * dh, lane);
            dvT[dh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ga, pb[sg], dvT[dh], 0, 0, 0);
            dkT[dh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa, sb[sg], dkT[dh], 0, 0, 0);
        }
    // dS^T -> hand-off buffer (row = key li, 4 consecutive queries per write)
#pragma unroll
    for (int i = 0; i < 4; ++i)
        *reinterpret_cast<bf16x4*>(dst + li * SS + 8 * i + 4 * h) =
            bf16x4{sb[i >> 1][4 * (i & 1)], sb[i >> 1][4 * (i & 1) + 1], sb[i >> 1][4 * (i & 1) + 2],
                   sb[i >> 1][4 * (i & 1) + 3]};
}

// The owner of a query tile adds one key tile's share: dQ^T += K^T dS^T, with K^T read from
// the K rows of that key tile (key0) and dS^T from the hand-off buffer of the wave that
// worked on the pair.  Lane holds query li of the tile, channels 32 dh + 8 i + 4 h + j.
__device__ __forceinline__ void owner_dq(const uint16_t* Ks, const uint16_t* src, int key0, floatx16 (&dq)[2],
                                         int lane) {
    const bf16x8 sbt0 = tr_operand(src, SS, 0, 0, lane), sbt1 = tr_operand(src, SS, 16, 0, lane);
#pragma unroll
    for (int dh = 0; dh < 2; ++dh) {
        const bf16x8 k0 = tr_operand(Ks, RS, key0, 32 * dh, lane);
        const bf16x8 k1 = tr_operand(Ks, RS, key0 + 16, 32 * dh, lane);
        dq[dh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k0, sbt0, dq[dh], 0, 0, 0);
        dq[dh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k1, sbt1, dq[dh], 0, 0, 0);
    }
}

template <bool MULTI, bool KVPAD, bool ROPE>
__global__ __launch_bounds__(THREADS) void swin_bwd_bf16_window_kernel(SwinBwdArgs ba) {
    const SwinArgs& a = ba.f;
    __shared__ __attribute__((aligned(16))) unsigned char smem[LDS_BYTES];
    uint16_t* Qs = reinterpret_cast<uint16_t*>(smem + OFF_Q);
    uint16_t* dOs = reinterpret_cast<uint16_t*>(smem + OFF_DO);
    uint16_t* Ks = reinterpret_cast<uint16_t*>(smem + OFF_K);
    float* Ls = reinterpret_cast<float*>(smem + OFF_LSE);
    float* Ds = reinterpret_cast<float*>(smem + OFF_DD);
    float* DSP = reinterpret_cast<float*>(smem + OFF_DSP);
    float* KP = reinterpret_cast<float*>(smem + OFF_KP);
    uint16_t* DST = reinterpret_cast<uint16_t*>(smem + OFF_DST);

    // ---- workgroup -> unit (b, window, head), heads fastest, XCD classes rotated
    const unsigned id0 = xcd_rotate(blockIdx.x, 2);
    if (id0 >= (unsigned)ba.n_units) return;
    const unsigned id1 = a.div_heads.div(id0);
    const int head = (int)(id0 - id1 * (unsigned)a.heads);
    const unsigned id2 = a.div_nwin.div(id1);
    const int win = (int)(id1 - id2 * (unsigned)a.n_windows);
    const int b = (int)id2;

    const WindowRect wr = window_rect<MULTI>(a, win);
    const int n = wr.rows * wr.cols;          // 1 .. 256
    const int nt = (n + TL - 1) / TL;
    const long long n_pad = (long long)a.window * a.window - n;
    const bool has_pad = KVPAD && n_pad > 0;

    // ---- buffer resources at the window's first token, head `head`
    const long long win_elems = wr.tok0 * a.tok_stride + head * D;
    const long long q_base = (long long)b * a.q_batch_stride + win_elems;
    const long long kv_base = (long long)b * a.kv_batch_stride + win_elems;
    const long long q_bytes = ((long long)a.B * a.q_batch_stride - q_base) * 2;
    const long long kv_bytes = ((long long)a.B * a.kv_batch_stride - kv_base) * 2;
    const __amdgpu_buffer_rsrc_t qr = make_rsrc(static_cast<const uint16_t*>(a.q) + q_base, q_bytes);
    const __amdgpu_buffer_rsrc_t orr = make_rsrc(static_cast<const uint16_t*>(ba.out) + q_base, q_bytes);
    const __amdgpu_buffer_rsrc_t dor = make_rsrc(static_cast<const uint16_t*>(ba.dout) + q_base, q_bytes);
    const __amdgpu_buffer_rsrc_t dqr = make_rsrc(static_cast<uint16_t*>(ba.dq) + q_base, q_bytes);
    const __amdgpu_buffer_rsrc_t kr = make_rsrc(static_cast<const uint16_t*>(a.k) + kv_base, kv_bytes);
    const __amdgpu_buffer_rsrc_t vr = make_rsrc(static_cast<const uint16_t*>(a.v) + kv_base, kv_bytes);
    const __amdgpu_buffer_rsrc_t dkr = make_rsrc(static_cast<uint16_t*>(ba.dk) + kv_base, kv_bytes);
    const __amdgpu_buffer_rsrc_t dvr = make_rsrc(static_cast<uint16_t*>(ba.dv) + kv_base, kv_bytes);
    const long long lse_base = ((long long)b * a.heads + head) * a.L + wr.tok0;
    const long long lse_total = (long long)a.B * a.heads * a.L;
    const __amdgpu_buffer_rsrc_t lr = make_rsrc(ba.lse + lse_base, (lse_total - lse_base) * 4);

    WindowAddr addr;
    addr.init(wr.cols, (unsigned)((long long)wr.W * a.tok_stride * 2), (unsigned)(a.tok_stride * 2));

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int li = lane & 31;
    const int h = lane >> 5;

    // ---- 1. loads: the Q, dO and O rows first (staged first: a wait for a load waits for every
    //         load issued before it), then the wave's K and V rows.
    const int key = TL * wave + li;
    const bool key_ok = key < n;
    const unsigned krow = key_ok ? addr(key) : kOutside;
    // Q, dO, O: 8 threads per 128-byte row, rows r0 + 64 u
    const int part = tid & 7;
    const int r0 = tid >> 3;
    uint4 qv[4], gv[4], ov[4];
    float lse_raw[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int r = r0 + 64 * u;
        const unsigned off = r < n ? addr(r) + 16 * part : kOutside;
        qv[u] = bload16(qr, off);
        gv[u] = bload16(dor, off);
        ov[u] = bload16(orr, off);
        lse_raw[u] = __builtin_bit_cast(
            float, __builtin_amdgcn_raw_buffer_load_b32(lr, r < n ? 4 * addr.token(r, (unsigned)wr.W) : kOutside, 0, 0));
    }
    uint4 kp8 = {0u, 0u, 0u, 0u}, vp8 = {0u, 0u, 0u, 0u};
    if (has_pad) {
        const long long pad_elems = (long long)b * a.kv_batch_stride + a.L * a.tok_stride + head * D;
        const __amdgpu_buffer_rsrc_t kpr = make_rsrc(static_cast<const uint16_t*>(a.k) + pad_elems, D * 2);
        const __amdgpu_buffer_rsrc_t vpr = make_rsrc(static_cast<const uint16_t*>(a.v) + pad_elems, D * 2);
        kp8 = bload16(kpr, 16 * part);
        vp8 = bload16(vpr, 16 * part);
    }

    // K_w and V_w rows: lane holds row 32 * wave + li, channels 16 s + 8 h .. + 7 (the B operand
    // of S = Q K^T and dP = dO V^T)
    bf16x8 kreg[4], vreg[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        kreg[s] = __builtin_bit_cast(bf16x8, bload16(kr, krow + 32 * s + 16 * h));
        vreg[s] = __builtin_bit_cast(bf16x8, bload16(vr, krow + 32 * s + 16 * h));
    }

    // (row, col) grid coordinates of window-local index t
    auto coords = [&](int t, float& y, float& x) {
        const unsigned r = __umulhi((unsigned)t, addr.magic) + ((unsigned)t & addr.one_mask);
        y = (float)(wr.y0 + (int)r);
        x = (float)(wr.x0 + (int)((unsigned)t - r * addr.cols));
    };
    if constexpr (ROPE) {
        // RoPE on the loaded q rows (channels 8 part .. + 7: the row half for part < 4) and on
        // the wave's K rows (channels 16 s + 8 h .. + 7); the pad token is not rotated
        float y, x;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            coords(min(r0 + 64 * u, n - 1), y, x);
            qv[u] = __builtin_bit_cast(uint4, rope_rotate_bf16x8(__builtin_bit_cast(bf16x8, qv[u]),
                                                                 (part < 4 ? y : x) * a.rope_scale,
                                                                 a.rope_rev + 4 * (part & 3)));
        }
        coords(min(key, n - 1), y, x);
#pragma unroll
        for (int s = 0; s < 4; ++s)
            kreg[s] = rope_rotate_bf16x8(kreg[s], (s < 2 ? y : x) * a.rope_scale, a.rope_rev + 8 * (s & 1) + 4 * h);
    }

    // ---- LDS: Q, dO and K rows, LSE, D
    float pk[8], pv[8];   // this thread's share of the pad token's gradient (8 channels)
    for (int e = 0; e < 8; ++e) pk[e] = pv[e] = 0.f;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int r = r0 + 64 * u;
        *reinterpret_cast<uint4*>(Qs + r * RS + 8 * part) = qv[u];
        *reinterpret_cast<uint4*>(dOs + r * RS + 8 * part) = gv[u];
        const float dd = sum8(dot8(gv[u], ov[u]));
        const float lse2 = lse_raw[u] * kLog2e;
        if (part == 0) {
            Ds[r] = -dd;   // stored negated: it is the C operand of dP - D
            Ls[r] = lse2;
        }
        if (has_pad) {
            // pad token as key: P = n_pad exp(c <q, k_pad> - LSE), dS = P (<dO, v_pad> - D)
            const float zp = sum8(dot8(qv[u], kp8));
            const float dp = sum8(dot8(gv[u], vp8));
            const float p = r < n ? __builtin_amdgcn_exp2f(__builtin_fmaf(zp, a.scale_log2, log2f((float)n_pad) - lse2)) : 0.f;
            const float ds = p * (dp - dd);
            if (part == 0) DSP[r] = ds;
            const bf16x8 q8 = __builtin_bit_cast(bf16x8, qv[u]), g8 = __builtin_bit_cast(bf16x8, gv[u]);
            for (int e = 0; e < 8; ++e) {
                pk[e] = __builtin_fmaf(ds, (float)q8[e], pk[e]);
                pv[e] = __builtin_fmaf(p, (float)g8[e], pv[e]);
            }
        }
    }
    if (has_pad) {
        if (tid < 8) {
            const bf16x8 k8 = __builtin_bit_cast(bf16x8, kp8);
            for (int e = 0; e < 8; ++e) KP[8 * part + e] = (float)k8[e];
        }
        // sum over the 8 row groups of the wave (lanes part, part + 8, ...), then per wave to LDS
        float* wsum = reinterpret_cast<float*>(DST) + wave * kPadPartial;
        for (int e = 0; e < 8; ++e) {
            float x = pk[e], y = pv[e];
            x += __shfl_xor(x, 8);
            x += __shfl_xor(x, 16);
            x += __shfl_xor(x, 32);
            y += __shfl_xor(y, 8);
            y += __shfl_xor(y, 16);
            y += __shfl_xor(y, 32);
            if (lane < 8) {
                wsum[8 * part + e] = x;
                wsum[D + 8 * part + e] = y;
            }
        }
    }
#pragma unroll
    for (int s = 0; s < 4; ++s)
        *reinterpret_cast<bf16x8*>(Ks + (TL * wave + li) * RS + 16 * s + 8 * h) = kreg[s];
    __syncthreads();
    if (KVPAD && tid < kPadPartial) {
        // every workgroup writes its share (zero without virtual slots), so the reduction
        // reads a dense array
        float acc = 0.f;
        if (has_pad) {
            const float* wsum = reinterpret_cast<const float*>(DST);
            for (int w = 0; w < NW; ++w) acc += wsum[w * kPadPartial + tid];
        }
        const long long e = ((long long)b * a.heads + head) * a.n_windows + win;
        ba.ws[e * kPadPartial + tid] = tid < D ? acc * ba.scale : acc;
    }
    __syncthreads();

    // ---- 2. steps
    floatx16 dkT[2] = {floatx16{}, floatx16{}}, dvT[2] = {floatx16{}, floatx16{}};
    floatx16 dq[2] = {floatx16{}, floatx16{}};   // dQ^T of query tile `wave`, owned by this wave
    const float c2 = a.scale_log2;
    // C operand of S = Q K^T: 0, or -inf for a key past the window's last (its P is then 0)
    floatx16 s_init;
#pragma unroll
    for (int r = 0; r < 16; ++r) s_init[r] = key_ok ? 0.f : -INFINITY;
    // step t: wave w works on query tile (w + t) mod nt and hands its dS^T over (buffer t % 2);
    // during step t + 1 the owner of that tile adds its dQ^T share
    for (int t = 0; t < nt; ++t) {
        if (wave < nt) {
            if (t > 0) {
                const int w = wave - t + 1 >= 0 ? wave - t + 1 : wave - t + 1 + nt;
                owner_dq(Ks, DST + (((t - 1) & 1) * NW + w) * TL * SS, TL * w, dq, lane);
            }
            const int T = wave + t < nt ? wave + t : wave + t - nt;
            wave_step(Qs, dOs, Ds, Ls, DST + ((t & 1) * NW + wave) * TL * SS, kreg, vreg, s_init, dkT, dvT, TL * T,
                      c2, lane);
        }
        __syncthreads();
    }
    if (wave < nt) {
        const int w = wave - nt + 1 >= 0 ? wave - nt + 1 : wave + 1;
        owner_dq(Ks, DST + (((nt - 1) & 1) * NW + w) * TL * SS, TL * w, dq, lane);
    }
    __syncthreads();   // the epilogue stages dQ rows over the K rows

    // ---- 3. epilogue: each wave stages its 32 key rows of dK and dV (in the Q and dO rows)
    //         and its query tile of dQ (in that tile's accumulator space), then stores whole
    //         128-byte rows, 8 lanes per row.
    if (wave < nt) {
        const float sc = ba.scale;
        uint16_t* krow_s = Qs + (TL * wave + li) * RS;
        uint16_t* vrow_s = dOs + (TL * wave + li) * RS;
        if constexpr (ROPE) {
            // dk = R^T dk': this lane's key, channels 32 dh + 8 i + 4 h + {0..3} = pairs
            // 4 i + 2 h + {0, 1} of half dh
            float y, x;
            coords(min(key, n - 1), y, x);
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
        // dQ: this wave owns tile `wave`
        float4 x[8];
#pragma unroll
        for (int g = 0; g < 8; ++g) {
            const int dh = g >> 2, i = g & 3;
            x[g] = make_float4(dq[dh][4 * i], dq[dh][4 * i + 1], dq[dh][4 * i + 2], dq[dh][4 * i + 3]);
        }
        const int qi = TL * wave + li;
        const float dsp = has_pad ? DSP[qi] : 0.f;
        uint16_t* qrow_s = Ks + (TL * wave + li) * RS;
        [[maybe_unused]] float qy = 0.f, qx = 0.f;
        if constexpr (ROPE) coords(min(qi, n - 1), qy, qx);
#pragma unroll
        for (int g = 0; g < 8; ++g) {
            const int ch = 32 * (g >> 2) + 8 * (g & 3) + 4 * h;
            float v4[4] = {x[g].x, x[g].y, x[g].z, x[g].w};
            bf16x4 o4;
            if (has_pad)
#pragma unroll
                for (int j = 0; j < 4; ++j) v4[j] = __builtin_fmaf(dsp, KP[ch + j], v4[j]);
            if constexpr (ROPE) {
                // dq = R^T dq': pairs (ch % 32) / 2 + {0, 1} of half ch / 32
                const float pos = (ch < 32 ? qy : qx) * a.rope_scale;
                rope_unrotate_pair(v4[0], v4[1], pos, a.rope_rev[(ch & 31) / 2]);
                rope_unrotate_pair(v4[2], v4[3], pos, a.rope_rev[(ch & 31) / 2 + 1]);
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) o4[j] = (__bf16)(v4[j] * sc);
            *reinterpret_cast<bf16x4*>(qrow_s + ch) = o4;
        }
        asm volatile("" ::: "memory");   // staged rows are read back by other lanes
        const uint16_t* qbase_s = Ks + TL * wave * RS;
        const int sp = lane & 7;
        with_store_policy(ba.store_nt, [&](auto nt) {
#pragma unroll
            for (int it = 0; it < TL / 8; ++it) {
                const int rl = 8 * it + (lane >> 3);
                const int tok = TL * wave + rl;
                const unsigned off = tok < n ? addr(tok) + 16 * sp : kOutside;
                const uint4 kx = *reinterpret_cast<const uint4*>(Qs + tok * RS + 8 * sp);
                const uint4 vx = *reinterpret_cast<const uint4*>(dOs + tok * RS + 8 * sp);
                const uint4 qx = *reinterpret_cast<const uint4*>(qbase_s + rl * RS + 8 * sp);
                store_row<decltype(nt)::value>(__builtin_bit_cast(u32x4, kx), dkr, off);
                store_row<decltype(nt)::value>(__builtin_bit_cast(u32x4, vx), dvr, off);
                store_row<decltype(nt)::value>(__builtin_bit_cast(u32x4, qx), dqr, off);
            }
        });
    }
}

}  // namespace

hipError_t launch_swin_bwd_bf16_window(const SwinBwdArgs& a, hipStream_t stream) {
    SwinBwdArgs args = a;
    void* params[] = {&args};
    const bool multi = a.f.n_grids > 1, kv = a.f.pad_mode == 1;
    const void* fn;
    if (a.f.rope)   // RoPE: single grid only (the host admits no grid list with it)
        fn = kv ? reinterpret_cast<const void*>(&swin_bwd_bf16_window_kernel<false, true, true>)
                : reinterpret_cast<const void*>(&swin_bwd_bf16_window_kernel<false, false, true>);
    else
        fn = multi ? (kv ? reinterpret_cast<const void*>(&swin_bwd_bf16_window_kernel<true, true, false>)
                         : reinterpret_cast<const void*>(&swin_bwd_bf16_window_kernel<true, false, false>))
                   : (kv ? reinterpret_cast<const void*>(&swin_bwd_bf16_window_kernel<false, true, false>)
                         : reinterpret_cast<const void*>(&swin_bwd_bf16_window_kernel<false, false, false>));
    const long long groups = 8 * ((a.n_units + 7) / 8);
    return hipLaunchKernel(fn, dim3((unsigned)groups), dim3(THREADS), params, 0, stream);
}

}  // namespace fla
