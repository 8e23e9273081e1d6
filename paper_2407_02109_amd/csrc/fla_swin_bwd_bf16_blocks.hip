// Flash Swin attention backward, bf16 storage, gfx950 (CDNA4) matrix cores: the kernel for
// launches with windows of more than 256 tokens (those of up to 256 take the one-window
// kernel of fla_swin_bwd_bf16_window.hip).
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
//     in registers, while the window's queries stream through LDS in chunks of 64 (Q, dO
//     and O rows; -D and LSE log2(e) per query).  Per 32-query tile:
//        S = Q K_w^T, dP - D = dO V_w^T - D        (C operand -D)
//        P = exp2(S c log2(e) - LSE log2(e)), dS = P (dP - D), both rounded to bf16
//        dV_w^T += dO^T P, dK_w^T += Q^T dS       (dO^T, Q^T by the transposing LDS read)
//   * query role: owns 128 queries.  Wave w keeps the Q and dO rows of queries 32w .. + 31
//     in registers (B operands), their LSE and D in one register each (a lane holds one
//     query), and accumulates their dQ^T in registers, while the window's keys stream
//     through LDS in chunks of 64 (K and V rows).  Per 32-key tile:
//        S^T = K Q_w^T, dP^T - D = V dO_w^T - D
//        dS^T = P^T o (dP^T - D) in fp32, rounded to bf16
//        dQ_w^T += K^T dS^T                        (K^T by the transposing LDS read)
// No accumulator is shared between waves, so the tile loops need no barrier.
//
// Streaming.  A chunk's rows go from HBM straight into LDS (buffer loads that write LDS,
// no register staging), into one of two buffers: the next chunk's loads are issued as soon
// as a chunk is published, and land while the waves work on it.  Wave w loads rows 16 w ..
// 16 w + 15 of each chunk and, once its own loads are done, prepares exactly those rows
// (D, the LSE, RoPE, the pad token's terms), so one barrier per chunk publishes it.  LDS
// rows are 128 bytes whose 16-byte pieces are XOR-swizzled by row (piece p of row r holds
// channels 8 (p ^ (r & 7)) ..), which keeps both the row reads and the transposing reads
// free of bank conflicts.  A workgroup needs 51 KB of LDS and at most 168 VGPRs: three
// share a compute unit.  All the workgroups of one (batch entry, window, head) -- both
// roles of every block -- get ids that are equal mod 8, which the dispatcher sends to one
// XCD one after the other, so the window's rows come from HBM once and the other readers
// find them in that XCD's L2.
//
// Keys past the window's end are zero rows in LDS (query role): their dS multiplies a zero
// K row, and a partial key tile clears their P as well, so no infinity can reach the
// products.  Rows past a window's end are never stored.
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
constexpr int NMAX = kBwdBlock;        // 128 = NW * TL tokens per block
constexpr int CH = 64;                 // rows of a streamed chunk
constexpr int ROW = D;                 // bf16 per LDS row (128 bytes, swizzled pieces)
constexpr int CHE = CH * ROW;          // bf16 per chunk buffer
constexpr float kLog2e = 1.4426950408889634f;
static_assert(NW * TL == NMAX && CH == 16 * NW, "block and chunk geometry");

// LDS carve-up, bytes.  X, Y, Z: two chunk buffers each -- key role: Q, dO, O rows; query
// role: K, V rows (Z unused).  Per query of each buffered chunk (key role): LSE log2(e), -D,
// and the pad token's P and dS.  PADW: two half sums per channel of the pad token's gradient;
// PADKV: its k and v rows (key role) or its k row in fp32 (query role).  At the end X stages
// the dK (key role) or dQ rows (query role) and Y the dV rows.
constexpr int OFF_X = 0;
constexpr int OFF_Y = OFF_X + 2 * CHE * 2;
constexpr int OFF_Z = OFF_Y + 2 * CHE * 2;
constexpr int OFF_L = OFF_Z + 2 * CHE * 2;            // [2][CH] fp32
constexpr int OFF_ND = OFF_L + 2 * CH * 4;            // [2][CH] fp32
constexpr int OFF_PP = OFF_ND + 2 * CH * 4;           // [2][CH] fp32
constexpr int OFF_DSP = OFF_PP + 2 * CH * 4;          // [2][CH] fp32
constexpr int OFF_PADW = OFF_DSP + 2 * CH * 4;        // [2][128] fp32
constexpr int OFF_PADKV = OFF_PADW + 2 * kPadPartial * 4;   // [128] bf16 or [64] fp32
constexpr int LDS_BYTES = OFF_PADKV + D * 4;
static_assert(3 * LDS_BYTES <= 160 * 1024, "three workgroups per compute unit");
static_assert(2 * CHE * 2 >= NMAX * ROW * 2, "the epilogue stages a block's rows in two chunk buffers");
static_assert(THREADS == 2 * kPadPartial, "two threads per pad-gradient channel");

typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) shortx4 lds_shortx4;
typedef __attribute__((address_space(3))) void lds_void;

// bf16 index of channel c of row r in a swizzled LDS row array: 16-byte piece p of row r
// holds channels 8 (p ^ f(r)) .. + 7, f(r) = (r >> 1) & 7, so the 16 rows a 16-lane read of
// one piece touches cover all 64 banks once
__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }
__device__ __forceinline__ int sw(int r, int c) { return r * ROW + ((((c >> 3) ^ swz(r)) << 3) | (c & 7)); }

// Per-lane element offsets of the tile operands in a chunk buffer, for tiles starting at a
// multiple of 16 rows (where the swizzle of a lane's rows does not depend on the tile):
// a[s]: the row read of lane l (row l & 31, channels 16 s + 8 (l >> 5) .. + 7);
// t: the first transposing read of tr_operand at row0 = 0, col0 = 0.  tr_operand at
// (row0, 32 dh) reads base + row0 ROW + t + 32 dh and base + row0 ROW + t + 8 ROW + 32 (1 - dh)
// (the second 4-row group's swizzle differs from the first's in bit 2).
struct TileOff {
    int a[4];
    int t;
};
__device__ __forceinline__ TileOff tile_offsets(int lane) {
    TileOff o;
    const int li = lane & 31, h = lane >> 5;
#pragma unroll
    for (int s = 0; s < 4; ++s) o.a[s] = li * ROW + (((2 * s + h) ^ swz(li)) << 3);
    const int e = (lane & 15) >> 2, q = lane & 3, g1 = (lane >> 4) & 1;
    const int row = 4 * h + e;
    o.t = row * ROW + (((2 * g1 + (q >> 1)) ^ swz(row)) << 3) + 4 * (q & 1);
    return o;
}

// wait until this wave's outstanding global loads (and the LDS writes of its direct loads) are done
__device__ __forceinline__ void wait_loads() { __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8)); }

// Rows 16 w .. 16 w + 15 of a chunk (chunk-local row r = window-local token base + r, present
// when r < nrows, zero otherwise) from a buffer resource straight into the swizzled LDS
// rows `dst`: lane L writes piece L % 8 of row 8 i + L / 8 and loads the channels that piece
// holds.
__device__ __forceinline__ void load_rows(__amdgpu_buffer_rsrc_t src, uint16_t* dst, const WindowAddr& addr, int base,
                                          int nrows, int wave, int lane) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int r = 16 * wave + 8 * i + (lane >> 3);
        const int p = (lane & 7) ^ swz(r);
        const unsigned off = r < nrows ? addr(base + r) + 16 * p : kOutside;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(src, (lds_void*)(dst + (16 * wave + 8 * i) * ROW), 16, off, 0, 0, 0);
    }
}

// Transposing LDS read of a 32 x 16 operand from swizzled rows: lane l receives column
// `32 dh + (l & 31)` of rows row0 + 4 * (l >> 5) + {0..3} and row0 + 8 + 4 * (l >> 5) + {0..3}
// (row0 a multiple of 16).  Within each 16-lane group, ds_read_b64_tr_b16 has lane i name a
// 4-element piece (row i / 4, elements 4 * (i % 4) .. + 3) of a 4 x 16 block and returns to
// lane i the block's column i.  The row order matches the rows a lane holds in the accumulator
// of a 32 x 32 product, so that accumulator, rounded, is the other operand of a product summed
// over those rows.
__device__ __forceinline__ bf16x8 tr_operand(const uint16_t* base, int t, int row0, int dh) {
    const uint16_t* p = base + row0 * ROW + t;
    const shortx4 va = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_shortx4*)(const_cast<uint16_t*>(p + 32 * dh)));
    const shortx4 vb =
        __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_shortx4*)(const_cast<uint16_t*>(p + 8 * ROW + 32 * (1 - dh))));
    const bf16x4 a4 = __builtin_bit_cast(bf16x4, va), b4 = __builtin_bit_cast(bf16x4, vb);
    return bf16x8{a4[0], a4[1], a4[2], a4[3], b4[0], b4[1], b4[2], b4[3]};
}

__device__ __forceinline__ float dot8(const bf16x8& a, const bf16x8& b, float s) {
    for (int e = 0; e < 8; e += 2)
        s = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{a[e], a[e + 1]}, bf16x2{b[e], b[e + 1]}, s, false);
    return s;
}

__device__ __forceinline__ bf16x8 lds8(const uint16_t* p) { return *reinterpret_cast<const bf16x8*>(p); }

// Key role, one tile: the 32 queries whose swizzled rows start at q0 (Q, dO rows, -D and
// LSE*log2(e) of one chunk buffer in LDS) against the wave's 32 keys (kreg, vreg).  dK^T and
// dV^T add up in registers.
__device__ __forceinline__ void key_tile(const uint16_t* Qs, const uint16_t* dOs, const float* ND, const float* Ls,
                                         const bf16x8 (&kreg)[4], const bf16x8 (&vreg)[4], floatx16 (&dkT)[2],
                                         floatx16 (&dvT)[2], int q0, const TileOff& to, float c2, int lane) {
    const int h = lane >> 5;
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
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds8(Qs + q0 * ROW + to.a[s]), kreg[s], sacc, 0, 0, 0);
        pacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds8(dOs + q0 * ROW + to.a[s]), vreg[s], pacc, 0, 0, 0);
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
            dvT[dh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_operand(dOs, to.t, q0 + 16 * sg, dh), pb[sg],
                                                             dvT[dh], 0, 0, 0);
            dkT[dh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_operand(Qs, to.t, q0 + 16 * sg, dh), sb[sg],
                                                             dkT[dh], 0, 0, 0);
        }
}

// Query role, one tile: the 32 keys whose swizzled rows start at k0 (K, V rows of one chunk
// buffer) against the wave's 32 queries (qreg, greg; one query per lane column with its -D
// and LSE*log2(e)).  dQ^T adds up in registers.  MASKED: keys k0 + j with j >= nvalid get
// P = 0.
template <bool MASKED>
__device__ __forceinline__ void query_tile(const uint16_t* Ks, const uint16_t* Vs, const bf16x8 (&qreg)[4],
                                           const bf16x8 (&greg)[4], float nd, float l2, floatx16 (&dqT)[2],
                                           int k0, int nvalid, const TileOff& to, float c2, int lane) {
    const int h = lane >> 5;
    floatx16 sacc = {}, pacc;
#pragma unroll
    for (int r = 0; r < 16; ++r) pacc[r] = nd;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds8(Ks + k0 * ROW + to.a[s]), qreg[s], sacc, 0, 0, 0);
        pacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds8(Vs + k0 * ROW + to.a[s]), greg[s], pacc, 0, 0, 0);
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
            dqT[dh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_operand(Ks, to.t, k0 + 16 * s2, dh), sb[s2],
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

// RoPE on the two 8-channel pieces (channels 16 qq .. 16 qq + 15) of chunk row r, in place,
// for window-local token t
template <bool ROPE>
__device__ __forceinline__ void rope_row(const SwinArgs& a, const Block& k, uint16_t* rows, int r, int qq, int t) {
    if constexpr (ROPE) {
        float y, x;
        coords(k, min(t, k.n - 1), y, x);
#pragma unroll 1
        for (int j = 0; j < 2; ++j) {
            const int piece = 2 * qq + j;
            bf16x8* p = reinterpret_cast<bf16x8*>(rows + sw(r, 8 * piece));
            *p = rope_rotate_bf16x8(*p, (piece < 4 ? y : x) * a.rope_scale, a.rope_rev + 4 * (piece & 3));
        }
    }
}

template <bool KVPAD, bool ROPE>
__device__ __forceinline__ void key_role(const SwinBwdArgs& ba, const Block& k, unsigned char* smem) {
    const SwinArgs& a = ba.f;
    uint16_t* Xs = reinterpret_cast<uint16_t*>(smem + OFF_X);
    uint16_t* Ys = reinterpret_cast<uint16_t*>(smem + OFF_Y);
    uint16_t* Zs = reinterpret_cast<uint16_t*>(smem + OFF_Z);
    float* Ls = reinterpret_cast<float*>(smem + OFF_L);
    float* ND = reinterpret_cast<float*>(smem + OFF_ND);
    float* PP = reinterpret_cast<float*>(smem + OFF_PP);
    float* DSP = reinterpret_cast<float*>(smem + OFF_DSP);
    float* PADW = reinterpret_cast<float*>(smem + OFF_PADW);
    uint16_t* PADKV = reinterpret_cast<uint16_t*>(smem + OFF_PADKV);
    const int tid = threadIdx.x, lane = tid & 63, li = lane & 31, h = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const long long e = (((long long)k.b * a.heads + k.head) * a.n_windows + k.win) * ba.nbb + k.blk;
    const int key0 = NMAX * k.blk;
    if (key0 >= k.n) {   // the window has fewer blocks; its pad partial is still read
        if (KVPAD && tid < kPadPartial) ba.ws[e * kPadPartial + tid] = 0.f;
        return;
    }
    const int nkeys = min(NMAX, k.n - key0);
    const bool pad_here = KVPAD && k.n_pad > 0 && k.blk == 0;
    const int nqc = (k.n + CH - 1) / CH;

    // the first chunk's rows go out first, then the wave's K and V rows (lane holds key
    // key0 + 32 wave + li, channels 16 s + 8 h .. + 7), and the pad token's rows
    const int pr = 16 * wave + (lane >> 2), qq = lane & 3;   // the row this thread prepares
    auto issue = [&](int qc) {
        const int buf = qc & 1, qbase = CH * qc, nq = min(CH, k.n - qbase);
        load_rows(k.qr, Xs + buf * CHE, k.addr, qbase, nq, wave, lane);
        load_rows(k.dor, Ys + buf * CHE, k.addr, qbase, nq, wave, lane);
        load_rows(k.orr, Zs + buf * CHE, k.addr, qbase, nq, wave, lane);
        return __builtin_bit_cast(
            float, __builtin_amdgcn_raw_buffer_load_b32(
                       k.lr, pr < nq ? 4 * k.addr.token(qbase + pr, (unsigned)k.wr.W) : kOutside, 0, 0));
    };
    float lse_next = issue(0);
    const int key = TL * wave + li;
    const unsigned krow = key < nkeys ? k.addr(key0 + key) : kOutside;
    bf16x8 kreg[4], vreg[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        kreg[s] = __builtin_bit_cast(bf16x8, bload16(k.kr, krow + 32 * s + 16 * h));
        vreg[s] = __builtin_bit_cast(bf16x8, bload16(k.vr, krow + 32 * s + 16 * h));
    }
    if (pad_here && tid < 16) {
        const long long pad_elems = (long long)k.b * a.kv_batch_stride + a.L * a.tok_stride + k.head * D;
        const __amdgpu_buffer_rsrc_t prs = make_rsrc(static_cast<const uint16_t*>(tid < 8 ? a.k : a.v) + pad_elems, D * 2);
        *reinterpret_cast<uint4*>(PADKV + 8 * tid) = bload16(prs, 16 * (tid & 7));
    }
    if constexpr (ROPE) {
        float y, x;
        coords(k, min(key0 + key, k.n - 1), y, x);
        wait_loads();
#pragma unroll
        for (int s = 0; s < 4; ++s)
            kreg[s] = rope_rotate_bf16x8(kreg[s], (s < 2 ? y : x) * a.rope_scale, a.rope_rev + 8 * (s & 1) + 4 * h);
    }
    if (pad_here) __syncthreads();   // the pad rows are read by every row's preparation

    const float c2 = a.scale_log2;
    const float log2_npad = pad_here ? log2f((float)k.n_pad) : 0.f;
    float pad_sum = 0.f;   // thread (half, channel): its half of each chunk's rows, over the chunks
    const TileOff to = tile_offsets(lane);
    floatx16 dkT[2] = {floatx16{}, floatx16{}}, dvT[2] = {floatx16{}, floatx16{}};

    for (int qc = 0; qc < nqc; ++qc) {
        const int buf = qc & 1, qbase = CH * qc, nq = min(CH, k.n - qbase);
        uint16_t* Qs = Xs + buf * CHE;
        uint16_t* dOs = Ys + buf * CHE;
        const uint16_t* Os = Zs + buf * CHE;
        float* Lb = Ls + buf * CH;
        float* NDb = ND + buf * CH;
        const float lse = lse_next;
        // ---- the wave's own rows of this chunk: D, LSE, RoPE, the pad token's P and dS
        //      (4 threads per row, channels 16 qq .. 16 qq + 15)
        wait_loads();
        {
            float dd = 0.f;
#pragma unroll
            for (int j = 0; j < 2; ++j)
                dd = dot8(lds8(dOs + sw(pr, 16 * qq + 8 * j)), lds8(Os + sw(pr, 16 * qq + 8 * j)), dd);
            dd += __shfl_xor(dd, 1);
            dd += __shfl_xor(dd, 2);
            const float l2 = lse * kLog2e;
            if (qq == 0) {
                NDb[pr] = -dd;
                Lb[pr] = l2;
            }
            rope_row<ROPE>(a, k, Qs, pr, qq, qbase + pr);
            if (pad_here) {
                // pad token as key: P = n_pad exp(c <q, k_pad> - LSE), dS = P (<dO, v_pad> - D)
                asm volatile("" ::: "memory");   // the rotated q pieces are read back
                float zp = 0.f, dp = 0.f;
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const int c = 16 * qq + 8 * j;
                    zp = dot8(lds8(Qs + sw(pr, c)), lds8(PADKV + c), zp);
                    dp = dot8(lds8(dOs + sw(pr, c)), lds8(PADKV + D + c), dp);
                }
                zp += __shfl_xor(zp, 1);
                zp += __shfl_xor(zp, 2);
                dp += __shfl_xor(dp, 1);
                dp += __shfl_xor(dp, 2);
                const float p = pr < nq ? __builtin_amdgcn_exp2f(__builtin_fmaf(zp, c2, log2_npad - l2)) : 0.f;
                if (qq == 0) {
                    PP[buf * CH + pr] = p;
                    DSP[buf * CH + pr] = p * (dp - dd);
                }
            }
        }
        __syncthreads();   // the chunk is published; every wave is done with the previous one
        if (qc + 1 < nqc) lse_next = issue(qc + 1);   // lands in the other buffer meanwhile
        if (pad_here) {
            // the pad token's gradient over this chunk's rows: thread (half, c) sums channel c of
            // dS_p q (c < 64) or P_p dO (c >= 64) over rows half * 32 .. + 31 (rows past nq have
            // P = dS = 0), as four interleaved partial sums added in a fixed order
            const int c = tid & (kPadPartial - 1), half = tid / kPadPartial;
            const float* w = (c < D ? DSP : PP) + buf * CH;
            const uint16_t* rows = c < D ? Qs : dOs;
            const int ch = c & (D - 1);
            float acc4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 1
            for (int i = 0; i < CH / 2; i += 4)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int r = CH / 2 * half + i + j;
                    acc4[j] = __builtin_fmaf(w[r], __uint_as_float((unsigned)rows[sw(r, ch)] << 16), acc4[j]);
                }
            pad_sum += (acc4[0] + acc4[1]) + (acc4[2] + acc4[3]);
        }
        // ---- tiles: the wave's keys against the chunk's query tiles
        if (TL * wave < nkeys)
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const int T = (wave + t) & 1;   // the waves start on different tiles
                if (TL * T < nq) key_tile(Qs, dOs, NDb, Lb, kreg, vreg, dkT, dvT, TL * T, to, c2, lane);
            }
    }
    if (pad_here) PADW[tid] = pad_sum;
    __syncthreads();   // the chunk buffers are free for staging; the pad sums are complete

    if (KVPAD && tid < kPadPartial) {
        // every block writes its share (zero without virtual slots or past block 0), so the
        // reduction reads a dense array
        const float acc = pad_here ? PADW[tid] + PADW[kPadPartial + tid] : 0.f;
        ba.ws[e * kPadPartial + tid] = tid < D ? acc * ba.scale : acc;
    }

    // ---- dK, dV of the wave's keys: stage its 32 rows (swizzled, X and Y), store whole
    //      128-byte rows, 8 lanes per row
    if (TL * wave < nkeys) {
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
                    for (int p2 = 0; p2 < 2; ++p2) {
                        float p0 = dkT[dh][4 * i + 2 * p2], p1 = dkT[dh][4 * i + 2 * p2 + 1];
                        rope_unrotate_pair(p0, p1, (dh == 0 ? y : x) * a.rope_scale, a.rope_rev[4 * i + 2 * h + p2]);
                        dkT[dh][4 * i + 2 * p2] = p0;
                        dkT[dh][4 * i + 2 * p2 + 1] = p1;
                    }
        }
        const int row = TL * wave + li;
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
                *reinterpret_cast<bf16x4*>(Xs + sw(row, 32 * dh + 8 * i + 4 * h)) = k4;
                *reinterpret_cast<bf16x4*>(Ys + sw(row, 32 * dh + 8 * i + 4 * h)) = v4;
            }
        asm volatile("" ::: "memory");   // staged rows are read back by other lanes of the wave
        const long long kv_base = (long long)k.b * a.kv_batch_stride + k.wr.tok0 * a.tok_stride + k.head * D;
        const long long kv_bytes = ((long long)a.B * a.kv_batch_stride - kv_base) * 2;
        const __amdgpu_buffer_rsrc_t dkr = make_rsrc(static_cast<uint16_t*>(ba.dk) + kv_base, kv_bytes);
        const __amdgpu_buffer_rsrc_t dvr = make_rsrc(static_cast<uint16_t*>(ba.dv) + kv_base, kv_bytes);
        const int sp = lane & 7;
        with_store_policy(ba.store_nt, [&](auto nt) {
#pragma unroll
            for (int it = 0; it < TL / 8; ++it) {
                const int rl = TL * wave + 8 * it + (lane >> 3);
                const unsigned off = rl < nkeys ? k.addr(key0 + rl) + 16 * sp : kOutside;
                const uint4 kx = *reinterpret_cast<const uint4*>(Xs + sw(rl, 8 * sp));
                const uint4 vx = *reinterpret_cast<const uint4*>(Ys + sw(rl, 8 * sp));
                store_row<decltype(nt)::value>(__builtin_bit_cast(u32x4, kx), dkr, off);
                store_row<decltype(nt)::value>(__builtin_bit_cast(u32x4, vx), dvr, off);
            }
        });
    }
}

template <bool KVPAD, bool ROPE>
__device__ __forceinline__ void query_role(const SwinBwdArgs& ba, const Block& k, unsigned char* smem) {
    const SwinArgs& a = ba.f;
    uint16_t* Xs = reinterpret_cast<uint16_t*>(smem + OFF_X);
    uint16_t* Ys = reinterpret_cast<uint16_t*>(smem + OFF_Y);
    float* KP = reinterpret_cast<float*>(smem + OFF_PADKV);
    const int tid = threadIdx.x, lane = tid & 63, li = lane & 31, h = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int q0 = NMAX * k.blk;
    if (q0 >= k.n) return;
    const int nq = min(NMAX, k.n - q0);
    const bool has_pad = KVPAD && k.n_pad > 0;
    const int nkc = (k.n + CH - 1) / CH;
    auto issue = [&](int kc) {
        const int buf = kc & 1, kbase = CH * kc, nk = min(CH, k.n - kbase);
        load_rows(k.kr, Xs + buf * CHE, k.addr, kbase, nk, wave, lane);
        load_rows(k.vr, Ys + buf * CHE, k.addr, kbase, nk, wave, lane);
    };
    issue(0);

    // Q_w and dO_w (B operands): lane holds query q0 + 32 wave + li, channels 16 s + 8 h .. + 7;
    // O only for D = <dO, O>, and the query's LSE
    const int qi = TL * wave + li;
    const bool q_ok = qi < nq;
    const unsigned qrow = q_ok ? k.addr(q0 + qi) : kOutside;
    bf16x8 qreg[4], greg[4];
    uint4 oreg[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        qreg[s] = __builtin_bit_cast(bf16x8, bload16(k.qr, qrow + 32 * s + 16 * h));
        greg[s] = __builtin_bit_cast(bf16x8, bload16(k.dor, qrow + 32 * s + 16 * h));
        oreg[s] = bload16(k.orr, qrow + 32 * s + 16 * h);
    }
    const float l2 = __builtin_bit_cast(
                         float, __builtin_amdgcn_raw_buffer_load_b32(
                                    k.lr, q_ok ? 4 * k.addr.token(q0 + qi, (unsigned)k.wr.W) : kOutside, 0, 0)) *
                     kLog2e;
    float dd = 0.f;
#pragma unroll
    for (int s = 0; s < 4; ++s) dd = dot8(greg[s], __builtin_bit_cast(bf16x8, oreg[s]), dd);
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
    const int pr = 16 * wave + (lane >> 2), qq = lane & 3;   // the row this thread prepares
    const TileOff to = tile_offsets(lane);
    for (int kc = 0; kc < nkc; ++kc) {
        const int buf = kc & 1, kbase = CH * kc, nk = min(CH, k.n - kbase);
        uint16_t* Ks = Xs + buf * CHE;
        const uint16_t* Vs = Ys + buf * CHE;
        wait_loads();
        rope_row<ROPE>(a, k, Ks, pr, qq, kbase + pr);
        __syncthreads();   // the chunk is published; every wave is done with the previous one
        if (kc + 1 < nkc) issue(kc + 1);   // lands in the other buffer meanwhile
        // ---- tiles: the wave's queries against the chunk's key tiles; a partial tile masks its
        //      missing keys
        if (TL * wave < nq)
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const int T = (wave + t) & 1;
                const int nv = nk - TL * T;
                if (nv >= TL)
                    query_tile<false>(Ks, Vs, qreg, greg, nd, l2, dqT, TL * T, TL, to, c2, lane);
                else if (nv > 0)
                    query_tile<true>(Ks, Vs, qreg, greg, nd, l2, dqT, TL * T, nv, to, c2, lane);
            }
    }
    __syncthreads();   // the chunk buffers are free for staging

    // ---- dQ of the wave's queries: + dS_p k_pad, rotate back, scale, round; stage the 32 rows
    //      (swizzled, X) and store whole 128-byte rows, 8 lanes per row.  dqT[dh] entry r:
    //      channel 32 dh + 8 (r / 4) + 4 h + r % 4 of the lane's query.
    if (TL * wave < nq) {
        const float sc = ba.scale;
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
                *reinterpret_cast<bf16x4*>(Xs + sw(qi, ch)) = o4;
            }
        asm volatile("" ::: "memory");   // staged rows are read back by other lanes of the wave
        const long long q_base = (long long)k.b * a.q_batch_stride + k.wr.tok0 * a.tok_stride + k.head * D;
        const __amdgpu_buffer_rsrc_t dqr =
            make_rsrc(static_cast<uint16_t*>(ba.dq) + q_base, ((long long)a.B * a.q_batch_stride - q_base) * 2);
        const int sp = lane & 7;
        with_store_policy(ba.store_nt, [&](auto nt) {
#pragma unroll
            for (int it = 0; it < TL / 8; ++it) {
                const int rl = TL * wave + 8 * it + (lane >> 3);
                const unsigned off = rl < nq ? k.addr(q0 + rl) + 16 * sp : kOutside;
                const uint4 qx4 = *reinterpret_cast<const uint4*>(Xs + sw(rl, 8 * sp));
                store_row<decltype(nt)::value>(__builtin_bit_cast(u32x4, qx4), dqr, off);
            }
        });
    }
}

// Workgroup id -> (unit, role, block), unit = (batch entry, window, head): the 2 nbb
// workgroups of unit u (both roles of each of its nbb blocks) get ids
// 8 (2 nbb (u / 8) + j) + u % 8, j = 2 block + role, all on XCD u % 8 and dispatched
// one after the other there.  Units are numbered heads fastest, then windows, then batch
// entries.
template <bool MULTI, bool KVPAD, bool ROPE>
__global__ __launch_bounds__(THREADS) __attribute__((amdgpu_waves_per_eu(3, 3)))
void swin_bwd_bf16_block_kernel(SwinBwdArgs ba) {
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

hipError_t launch_swin_bwd_bf16_blocks(const SwinBwdArgs& a, hipStream_t stream) {
    SwinBwdArgs args = a;
    void* params[] = {&args};
    const bool multi = a.f.n_grids > 1, kv = a.f.pad_mode == 1;
    const void* fn;
    if (a.f.rope)   // RoPE: single grid only (the host admits no grid list with it)
        fn = kv ? reinterpret_cast<const void*>(&swin_bwd_bf16_block_kernel<false, true, true>)
                : reinterpret_cast<const void*>(&swin_bwd_bf16_block_kernel<false, false, true>);
    else
        fn = multi ? (kv ? reinterpret_cast<const void*>(&swin_bwd_bf16_block_kernel<true, true, false>)
                         : reinterpret_cast<const void*>(&swin_bwd_bf16_block_kernel<true, false, false>))
                   : (kv ? reinterpret_cast<const void*>(&swin_bwd_bf16_block_kernel<false, true, false>)
                         : reinterpret_cast<const void*>(&swin_bwd_bf16_block_kernel<false, false, false>));
    return hipLaunchKernel(fn, dim3((unsigned)bwd_bf16_groups(a.n_units, a.nbb)), dim3(THREADS), params, 0, stream);
}

}  // namespace fla
