// Flash Swin attention forward, bf16 storage, gfx950 (CDNA4) matrix cores.
//
// One workgroup = one (batch entry, window, block of up to 256 queries, head).  The
// window's rectangle comes from integer arithmetic on the shifted-window geometry
// (HRSAM Sec. 3.3 / App. A): no index table, no reordered copy.  Its real tokens are
// taken in row-major order inside the rectangle (Eq. nonshift), so the key set is dense:
// n = rows * cols keys, no masked slots except the tail of the last key tile.
//
// Per workgroup (512 threads = 8 waves):
//   1. K rows of the window -> LDS row-major; V rows -> LDS transposed (V^T, one row per
//      channel) so that P.V can take V as the A operand with keys along the reduction.
//      Every global load of a 256-key chunk is issued before the first LDS write.
//   2. Each wave owns 32 queries; Q stays in registers as the B operand.
//      For every tile of 32 keys:  S^T = K . Q^T on v_mfma_f32_32x32x16_bf16 (fp32
//      accumulation).  Each lane then holds 16 keys of one query column and the partner
//      lane (l ^ 32) the other 16, so the column max needs one v_permlane32_swap.
//      p = exp2(s * log2(e)/sqrt(d) - m) is a single FMA + v_exp_f32; P^T is rounded to
//      bf16 in the exact register layout the next MFMA reads as its B operand, and the
//      row sum adds the rounded values with v_dot2_f32_bf16.  O^T += V^T . P^T.
//      The running max is raised only when a tile exceeds it by more than 2^8 (in the
//      exp2 domain), so the O^T rescale runs on a handful of tiles, not on every one.
//      Tiles that end at or before the window's last key run a variant with no mask code.
//      The kernel is held to 128 VGPRs so that 4 waves share each SIMD (2 workgroups per
//      CU): while one wave waits on the matrix core, another runs its softmax on the
//      vector ALU, which is the busier of the two units.
//   3. Epilogue: O^T / l, round to bf16 (RNE), store each query row at its own token; if
//      asked, also the log-sum-exp m + log(l) of every query (the training forward).  The
//      result goes through LDS first so that every store writes whole 128-byte rows (8 lanes
//      x 16 B): stored straight from the MFMA layout, each instruction would write 8-byte
//      pieces of 32 rows, and those partial-line writes cost about a tenth of the layer.
//
// KV-only padding (Sec. 3.4, App. B): the pad token (row L of k, v) is loaded as key n of
// the window and its logit is raised by log2(n_pad)/scale, so in the softmax it carries
// the weight of the n_pad = window^2 - n virtual slots it stands for.
//
// Optional prologue fusion of 2-D RoPE (Sec. 3.1): q in registers, and each K row in place in
// LDS right after its write, are rotated by their token's grid coordinates, with the cos / sin
// of the window's row and column positions in a per-workgroup LDS table (windows of at most
// 32 x 32 tokens; wider ones evaluate them per rotated piece), so a rotated copy of q and k
// never goes through HBM.  The pad token has no position and is not rotated.
#include "fla_swin_device.h"

namespace fla {
namespace {

constexpr int THREADS = 512;    // 8 waves of 64
constexpr int kStoreNT = 2;     // cache policy of the output stores: non-temporal (nt)
constexpr int QW = 32;          // queries per wave
constexpr int KC = 256;         // keys staged in LDS at a time
constexpr int KT = 32;          // keys per inner tile
constexpr int KH = KC / 2;      // keys per half chunk (staged and computed in turn)
constexpr int VS = KC + 4;      // V^T row stride in LDS, bf16 elements (520 B)

// Per head_dim D (64; the plain forward also has instances for 32 and 128): the K row stride
// in LDS (D + 8 bf16: 144 B at D = 64), the threads that load one K row 16 bytes each, the K
// pieces a thread holds, the (4 keys x 8 channels) pieces of V, and the waves per SIMD the
// registers and LDS allow (at D = 128, K and V^T take 136 KB: one workgroup per CU).
template <int D>
struct Cfg {
    static constexpr int KS = D + 8;
    static constexpr int DLOG = D == 32 ? 5 : D == 64 ? 6 : 7;
    static constexpr int TPR = D / 8;               // threads per K row
    static constexpr int TPR_LOG = DLOG - 3;
    static constexpr int RPP = THREADS / TPR;       // K rows per pass of the workgroup
    static constexpr int KREG = KC / RPP;           // K pieces per thread
    static constexpr int VUNITS = (KC / 4) * (D / 8);
    static constexpr int VPT = (VUNITS + THREADS - 1) / THREADS;   // V pieces per thread
    static constexpr int WAVES = D > 64 ? 2 : 4;
};
constexpr float kLazyThreshold = 8.f;   // exp2-domain headroom before the max is raised
constexpr float kLn2 = 0.693147180559945309f;

// f(B), f(B + 1), ..., f(E - 1) as separate calls with constant arguments (the same code as
// writing the calls out; an unrolled loop is scheduled differently)
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (B < E) {
        f(B);
        static_for<B + 1, E>(f);
    }
}

template <int D, bool MASKED>
__device__ __forceinline__ void attend_tile(const uint16_t* __restrict__ Ks, const uint16_t* __restrict__ Vt,
                                            int t0, int kc0, int nk, int n, float pad_bias_raw,
                                            const bf16x8 (&qop)[D / 16], floatx16 (&o)[D / 32],
                                            float& m_run, float& neg_mc, float& l_run, float c_log2, int lane) {
    constexpr int KS = Cfg<D>::KS;
    const int li = lane & 31;
    const int h = lane >> 5;
    // ---- S^T = K . Q^T for 32 keys x 32 queries: s[r] holds key 8*(r/4) + 4*h + r%4
    //      of query li
    const uint16_t* krow = Ks + (t0 + li) * KS + 8 * h;
    floatx16 s = {};
    for (int st = 0; st < D / 16; ++st)
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8*>(krow + 16 * st),
                                                    qop[st], s, 0, 0, 0);
    if constexpr (MASKED) {
        // entry r holds key base + 8*(r/4) + r%4 with base = kc0 + t0 + 4*h
        const int lim = nk - (kc0 + t0 + 4 * h);    // entries below lim are keys of the window
        const int pad = n - (kc0 + t0 + 4 * h);     // the entry that is the pad token (if any)
        for (int r = 0; r < 16; ++r) {
            const int off = 8 * (r >> 2) + (r & 3);
            const float x = off == pad ? s[r] + pad_bias_raw : s[r];
            s[r] = off < lim ? x : -INFINITY;
        }
    }
    // 16 values -> 1 in 8 operations (v_max3_f32 takes three)
    float m0 = __builtin_fmaxf(__builtin_fmaxf(s[0], s[1]), s[2]);
    float m1 = __builtin_fmaxf(__builtin_fmaxf(s[3], s[4]), s[5]);
    float m2 = __builtin_fmaxf(__builtin_fmaxf(s[6], s[7]), s[8]);
    float m3 = __builtin_fmaxf(__builtin_fmaxf(s[9], s[10]), s[11]);
    float m4 = __builtin_fmaxf(__builtin_fmaxf(s[12], s[13]), s[14]);
    m0 = __builtin_fmaxf(__builtin_fmaxf(m0, m1), m2);
    m3 = __builtin_fmaxf(__builtin_fmaxf(m3, m4), s[15]);
    const float mx = xhalf_max(__builtin_fmaxf(m0, m3));
    const bool raise = mx > m_run + kLazyThreshold / c_log2;
    if (__builtin_amdgcn_ballot_w64(raise)) {
        const float m_new = raise ? mx : m_run;
        const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c_log2);
        m_run = m_new;
        l_run *= alpha;
        for (int db = 0; db < D / 32; ++db) o[db] *= alpha;
        neg_mc = -m_run * c_log2;
    }
    bf16x8 pb[2];
    for (int sg = 0; sg < 2; ++sg) {
        bf16x8 v8;
        for (int j = 0; j < 8; ++j)
            v8[j] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s[8 * sg + j], c_log2, neg_mc));
        pb[sg] = v8;
    }
    const bf16x2 ones = {(__bf16)1.f, (__bf16)1.f};
    for (int sg = 0; sg < 2; ++sg)
        for (int j = 0; j < 8; j += 2)
            l_run = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pb[sg][j], pb[sg][j + 1]}, ones, l_run, false);
    for (int sg = 0; sg < 2; ++sg)
        for (int db = 0; db < D / 32; ++db) {
            const uint16_t* vrow = Vt + (32 * db + li) * VS + t0 + 16 * sg + 4 * h;
            const bf16x4 va = *reinterpret_cast<const bf16x4*>(vrow);
            const bf16x4 vb = *reinterpret_cast<const bf16x4*>(vrow + 8);
            const bf16x8 vA = {va[0], va[1], va[2], va[3], vb[0], vb[1], vb[2], vb[3]};
            o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vA, pb[sg], o[db], 0, 0, 0);
        }
}

// D = 64: 4 waves per SIMD, at most 128 VGPRs, and the LDS footprint (2 x 69 KB) admits the
// two workgroups per CU that this takes.
// (row, col) of window-local index t inside the window's rectangle
__device__ __forceinline__ void window_rc(const WindowAddr& addr, int t, int& r, int& c) {
    const unsigned ru = __umulhi((unsigned)t, addr.magic) + ((unsigned)t & addr.one_mask);
    r = (int)ru;
    c = (int)((unsigned)t - ru * addr.cols);
}

// RoPE of 8 consecutive channels (4 pairs) from a table of (cos, sin) per pair
__device__ __forceinline__ void rope_rotate8_tab(uint16_t (&x)[8], const float2* cs) {
    for (int i = 0; i < 4; ++i) {
        const float2 t = cs[i];
        const float a = __uint_as_float((unsigned)x[2 * i] << 16);
        const float b = __uint_as_float((unsigned)x[2 * i + 1] << 16);
        const __bf16 ra = (__bf16)(a * t.x - b * t.y), rb = (__bf16)(b * t.x + a * t.y);
        x[2 * i] = __builtin_bit_cast(uint16_t, ra);
        x[2 * i + 1] = __builtin_bit_cast(uint16_t, rb);
    }
}

// The same rotation with (cos, sin) taken directly at position pos: the table's entries come
// from the same fp32 expression (rope_cs), so both give the same bits.
__device__ __forceinline__ void rope_rotate8_at(uint16_t (&x)[8], float pos, const float* rev) {
    float2 cs[4];
    for (int i = 0; i < 4; ++i) cs[i] = rope_cs(pos, rev[i]);
    rope_rotate8_tab(x, cs);
}

constexpr int kRopeTab = 32;   // window rows / columns covered by the per-workgroup RoPE table

template <bool MULTI, bool ROPE, int D>
__global__ __launch_bounds__(THREADS) __attribute__((amdgpu_waves_per_eu(Cfg<D>::WAVES, Cfg<D>::WAVES)))
void swin_fwd_bf16_kernel(SwinArgs a) {
    static_assert(!ROPE || D == kHeadDim, "RoPE: head_dim 64 only");
    constexpr int KS = Cfg<D>::KS, TPR = Cfg<D>::TPR, TPR_LOG = Cfg<D>::TPR_LOG, RPP = Cfg<D>::RPP;
    __shared__ __attribute__((aligned(16))) uint16_t Ks[KC * KS];
    __shared__ __attribute__((aligned(16))) uint16_t Vt[D * VS];
    // RoPE: (cos, sin) of the window's row positions [0][r][j] and column positions [1][c][j]
    __shared__ float2 Rtab[ROPE ? 2 * kRopeTab * (D / 4) : 1];

    // ---- workgroup -> (b, window, query block, head); heads vary fastest so that the
    //      workgroups of one window read adjacent 128-byte pieces of the same token rows.
    //      With one query block per window, ids go to units through xcd_rotate (every XCD
    //      takes every head).  With several query blocks per window (xcd_group), the blocks
    //      of unit u = 8 g + r (b, window, head) get ids 8 (nqb g + blk) + x with
    //      r = (x + g / 4) mod 8: the dispatcher deals ids to the 8 XCDs in turn, so the
    //      blocks run on XCD x one after the other and the window's K and V rows come from
    //      HBM once, then from that XCD's L2, and the units' classes rotate over the XCDs as
    //      in xcd_rotate.  The divisions are multiply-high by constants the host prepared.
    const unsigned id = blockIdx.x;
    unsigned id1, id2;   // id1: (b, window, query block) (raster) or (b, window) (grouped); id2: (b, window)
    int head, qblk;
    if (a.xcd_group) {
        const unsigned rest = id >> 3;
        const unsigned g = a.div_nqb.div(rest);
        qblk = (int)(rest - g * (unsigned)a.nqb);
        const unsigned unit = (g << 3) + ((id + (g >> 2)) & 7u);   // XCD classes rotated, as in xcd_rotate
        if (unit >= (unsigned)a.n_units) return;
        id2 = a.div_heads.div(unit);
        head = (int)(unit - id2 * (unsigned)a.heads);
    } else {   // one query block per window: id1 = id2
        const unsigned u = xcd_rotate(id, 4);
        if (u >= (unsigned)a.n_groups) return;
        id1 = a.div_heads.div(u);
        head = (int)(u - id1 * (unsigned)a.heads);
        id2 = a.div_nqb.div(id1);
        qblk = (int)(id1 - id2 * (unsigned)a.nqb);
    }
    const int nwin = a.n_windows;
    const unsigned id3 = a.div_nwin.div(id2);
    const int win = (int)(id2 - id3 * (unsigned)nwin);
    const int b = (int)id3;

    const WindowRect wr = window_rect<MULTI>(a, win);
    const int n = wr.rows * wr.cols;
    const int q_begin = qblk * kQueryBlock;
    if (q_begin >= n) return;   // whole workgroup: this window has fewer query blocks

    const long long n_pad = (long long)a.window * a.window - n;
    const bool has_pad = a.pad_mode == 1 && n_pad > 0;
    const int nk = n + (has_pad ? 1 : 0);
    const float pad_bias_raw = has_pad ? log2f((float)n_pad) / a.scale_log2 : 0.f;

    // ---- buffer resources based at the window's first token (y0, x0) of head `head`
    const long long L = a.L;
    const long long win_elems = wr.tok0 * a.tok_stride + head * D;
    const long long q_base = (long long)b * a.q_batch_stride + win_elems;
    const long long kv_base = (long long)b * a.kv_batch_stride + win_elems;
    const long long q_total = (long long)a.B * a.q_batch_stride;
    const long long kv_total = (long long)a.B * a.kv_batch_stride;
    const uint16_t* qp = static_cast<const uint16_t*>(a.q) + q_base;
    const uint16_t* kp = static_cast<const uint16_t*>(a.k) + kv_base;
    const uint16_t* vp = static_cast<const uint16_t*>(a.v) + kv_base;
    uint16_t* op = static_cast<uint16_t*>(a.out) + q_base;
    const __amdgpu_buffer_rsrc_t qr = make_rsrc(qp, (q_total - q_base) * 2);
    const __amdgpu_buffer_rsrc_t orr = make_rsrc(op, (q_total - q_base) * 2);
    const __amdgpu_buffer_rsrc_t kr = make_rsrc(kp, (kv_total - kv_base) * 2);
    const __amdgpu_buffer_rsrc_t vr = make_rsrc(vp, (kv_total - kv_base) * 2);
    // the pad token of KV-token mode: row L of this batch entry and head, 128 bytes
    const long long pad_elems = (long long)b * a.kv_batch_stride + L * a.tok_stride + head * D;
    const __amdgpu_buffer_rsrc_t kpr = make_rsrc(static_cast<const uint16_t*>(a.k) + pad_elems, has_pad ? D * 2 : 0);
    const __amdgpu_buffer_rsrc_t vpr = make_rsrc(static_cast<const uint16_t*>(a.v) + pad_elems, has_pad ? D * 2 : 0);

    WindowAddr addr;
    addr.init(wr.cols, (unsigned)((long long)wr.W * a.tok_stride * 2), (unsigned)(a.tok_stride * 2));

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int li = lane & 31;
    const int h = lane >> 5;

    const int wq0 = q_begin + wave * QW;
    const int nq = min(QW, n - wq0);   // queries of this wave (<= 0: the wave only loads)

    // ---- Q in registers, B-operand layout: lane holds q[query li][16*st + 8*h .. +8]
    // RoPE: windows whose rectangle fits kRopeTab x kRopeTab take (cos, sin) from one table per
    // workgroup for their row and column positions (1024 entries, two per thread, filled
    // before anything else is live in registers); wider ones compute them per rotated piece
    const bool rope_tab = ROPE && wr.rows <= kRopeTab && wr.cols <= kRopeTab;
    if constexpr (ROPE) {
        for (int e = tid; rope_tab && e < 2 * kRopeTab * (D / 4); e += THREADS) {
            const int axis = e / (kRopeTab * (D / 4)), p = (e / (D / 4)) % kRopeTab, j = e % (D / 4);
            const float pos = (float)(axis ? wr.x0 + p : wr.y0 + p) * a.rope_scale;
            float t = pos * a.rope_rev[j];
            t -= __builtin_rintf(t);   // to [-1/2, 1/2] revolution for v_sin_f32 / v_cos_f32
            Rtab[e] = make_float2(__builtin_amdgcn_cosf(t), __builtin_amdgcn_sinf(t));
        }
    }

    bf16x8 qop[D / 16];
    if (nq > 0) {
        const unsigned row = addr(min(wq0 + li, n - 1));
        for (int st = 0; st < D / 16; ++st)
            qop[st] = __builtin_bit_cast(bf16x8, bload16(qr, row + 32 * st + 16 * h));
    }
    float m_run = -INFINITY, l_run = 0.f;
    float neg_mc = 0.f;   // -m_run * log2(e) / sqrt(d); the first tile always raises the max and sets it
    floatx16 o[D / 32];   // O^T: [channel block]
    for (int db = 0; db < D / 32; ++db) o[db] = floatx16{};

    for (int kc0 = 0; kc0 < nk; kc0 += KC) {
        const int ck = min(KC, nk - kc0);
        if (kc0 > 0) __syncthreads();   // previous chunk fully consumed

        // ---- issue every global load of the chunk before the first LDS write, so a
        //      workgroup waits for one round trip to HBM, not one per load.
        //      K: D/8 threads per row of 2D bytes (coalesced; 8 per 128-byte row at D = 64),
        //      rows tid/(D/8) + RPP*it.
        //      V: a thread takes 4 consecutive keys (quad) x 8 channels (vpart) and writes
        //      them transposed: 4 keys of one channel are one 8-byte LDS store (at D = 128 a
        //      thread takes two such pieces, at D = 32 half the threads take one).
        //      The chunk is consumed in two halves of 128 keys: V and the first half of K are
        //      written to LDS and that half is computed while the K rows of the second half
        //      are still arriving (deferring V as well would exceed 128 VGPRs).  Loads are
        //      issued in the order they are consumed, since a wave waits for its loads in
        //      issue order.
        constexpr int VUNITS = Cfg<D>::VUNITS, VPT = Cfg<D>::VPT;
        uint4 kreg[Cfg<D>::KREG];
        uint4 vreg[VPT][4];
        const int part = tid & (TPR - 1);
        // V piece j of this thread: unit tid + j THREADS, whose (vpart, quad) are
        // ((unit / 8) mod D/8, unit mod 8 + 8 (unit / D)) = (vpart, quad + j 8 THREADS / D)
        const int vpart = (tid >> 3) & (D / 8 - 1);
        const int quad = (tid & 7) + ((tid >> Cfg<D>::DLOG) << 3);
        auto load_k = [&](int it) {
            const int t = kc0 + (tid >> TPR_LOG) + RPP * it;
            kreg[it] = bload16(kr, (t < n ? addr(t) : kOutside) + part * 16);
        };
        // K rows of this half (and all of V^T with the first); RoPE on the K rows in place;
        // the pad token if its slot falls in this half; then the barrier
        constexpr int kh = KH;
        constexpr int its = kh / RPP;   // K rows per thread in one half
        static_for<0, its>(load_k);
        for (int j = 0; j < VPT; ++j) {   // (plain loops here: a lambda or an unroll pragma changes the schedule)
            if (VUNITS % THREADS == 0 || tid < VUNITS) {   // (a partial last piece only at D = 32, j = 0)
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int t = kc0 + (quad + j * 8 * (THREADS >> Cfg<D>::DLOG)) * 4 + u;
                    vreg[j][u] = bload16(vr, (t < n ? addr(t) : kOutside) + vpart * 16);
                }
            }
        }
        static_for<its, 2 * its>(load_k);

        auto write_v = [&]() {
            for (int j = 0; j < VPT; ++j) {
                if (VUNITS % THREADS != 0 && tid >= VUNITS) continue;
                const int qj = quad + j * 8 * (THREADS >> Cfg<D>::DLOG);
                const uint32_t* w0 = reinterpret_cast<const uint32_t*>(&vreg[j][0]);
                const uint32_t* w1 = reinterpret_cast<const uint32_t*>(&vreg[j][1]);
                const uint32_t* w2 = reinterpret_cast<const uint32_t*>(&vreg[j][2]);
                const uint32_t* w3 = reinterpret_cast<const uint32_t*>(&vreg[j][3]);
#pragma unroll
                for (int m = 0; m < 4; ++m) {
                    uint2 lo, hi;
                    lo.x = (w0[m] & 0xffffu) | (w1[m] << 16);
                    lo.y = (w2[m] & 0xffffu) | (w3[m] << 16);
                    hi.x = (w0[m] >> 16) | (w1[m] & 0xffff0000u);
                    hi.y = (w2[m] >> 16) | (w3[m] & 0xffff0000u);
                    const int ch = vpart * 8 + 2 * m;
                    *reinterpret_cast<uint2*>(&Vt[ch * VS + qj * 4]) = lo;
                    *reinterpret_cast<uint2*>(&Vt[(ch + 1) * VS + qj * 4]) = hi;
                }
            }
        };
        auto stage_half = [&](int half) {
            for (int it = its * half; it < its * (half + 1); ++it)
                *reinterpret_cast<uint4*>(&Ks[((tid >> TPR_LOG) + RPP * it) * KS + part * 8]) = kreg[it];
            if (half == 0) write_v();
            if constexpr (ROPE) {
                // RoPE on this thread's pieces of the K rows it just wrote (8 channels per row:
                // the row half for part < 4), in place in LDS
                if (kc0 == 0 && half == 0) __syncthreads();   // the cos / sin table is complete
                for (int it = its * half; it < its * (half + 1); ++it) {
                    const int key = (tid >> TPR_LOG) + RPP * it;
                    if (kc0 + key < n) {
                        int kr_, kc_;
                        window_rc(addr, kc0 + key, kr_, kc_);
                        uint16_t e[8];
                        __builtin_memcpy(e, &Ks[key * KS + part * 8], 16);
                        if (rope_tab)
                            rope_rotate8_tab(e, Rtab + ((part < 4 ? 0 : kRopeTab) + (part < 4 ? kr_ : kc_)) * (D / 4) +
                                                    4 * (part & 3));
                        else
                            rope_rotate8_at(e, (float)(part < 4 ? wr.y0 + kr_ : wr.x0 + kc_) * a.rope_scale,
                                            a.rope_rev + 4 * (part & 3));
                        __builtin_memcpy(&Ks[key * KS + part * 8], e, 16);
                    }
                }
            }
            const int slot = n - kc0;
            if (has_pad && slot >= kh * half && slot < kh * (half + 1)) {
                // the pad token is key n of the window: its slot was zero-filled above; after
                // the barrier, 8 threads put its K row and its V^T column in place
                __syncthreads();
                if (tid < D / 8) {
                    *reinterpret_cast<uint4*>(&Ks[slot * KS + tid * 8]) = bload16(kpr, tid * 16);
                    const uint4 vv = bload16(vpr, tid * 16);
                    const uint16_t* ve = reinterpret_cast<const uint16_t*>(&vv);
                    for (int e = 0; e < 8; ++e) Vt[(tid * 8 + e) * VS + slot] = ve[e];
                }
            }
            __syncthreads();
        };

        stage_half(0);
        if constexpr (ROPE) {
            if (kc0 == 0 && nq > 0) {
                // q, once: channels 16 st + 8 h .. + 7, the row half for st < 2, the column
                // half after
                int qr_, qc_;
                window_rc(addr, min(wq0 + li, n - 1), qr_, qc_);
                for (int st = 0; st < 4; ++st) {
                    uint16_t e[8];
                    __builtin_memcpy(e, &qop[st], 16);
                    const int j0 = 8 * (st & 1) + 4 * h;
                    if (rope_tab)
                        rope_rotate8_tab(e, Rtab + ((st < 2 ? 0 : kRopeTab) + (st < 2 ? qr_ : qc_)) * (D / 4) + j0);
                    else
                        rope_rotate8_at(e, (float)(st < 2 ? wr.y0 + qr_ : wr.x0 + qc_) * a.rope_scale,
                                        a.rope_rev + j0);
                    __builtin_memcpy(&qop[st], e, 16);
                }
            }
        }
        // tiles [t_begin, t_end) of the chunk: those that end at or before key n need no mask,
        // the rest (at most the last two: past the keys, or holding the pad token) do
        auto attend_range = [&](int t_begin, int t_end) {
            const int t_plain = min(t_end, t_begin + max(0, (n - kc0 - t_begin) / KT) * KT);
            for (int t0 = t_begin; t0 < t_plain; t0 += KT)
                attend_tile<D, false>(Ks, Vt, t0, kc0, nk, n, pad_bias_raw, qop, o, m_run, neg_mc, l_run,
                                   a.scale_log2, lane);
            for (int t0 = t_plain; t0 < t_end; t0 += KT)
                attend_tile<D, true>(Ks, Vt, t0, kc0, nk, n, pad_bias_raw, qop, o, m_run, neg_mc, l_run,
                                  a.scale_log2, lane);
        };
        if (nq > 0) attend_range(0, min(ck, kh));
        if (ck > kh) {
            stage_half(1);
            if (nq > 0) attend_range(kh, ck);
        }
    }

    // ---- epilogue: normalise, round to bf16 (RNE), and store each query row at its own
    //      token.  The wave's 32 x 64 result is staged in LDS (in the K tile, free once every
    //      wave is past its last tile) so that the stores are whole rows: D/8 lanes per row
    //      (8 per 128-byte row at D = 64), 16 bytes per lane.
    __syncthreads();
    if (nq > 0) {
        const float lsum = xhalf_sum(l_run);
        const float inv = 1.f / lsum;
        if (a.lse != nullptr && h == 0 && li < nq) {
            // log of the softmax denominator over the logits q.k / sqrt(d), natural units
            const long long row = ((long long)b * a.heads + head) * L + wr.tok0 +
                                  addr.token(wq0 + li, (unsigned)wr.W);
            a.lse[row] = (m_run * a.scale_log2 + log2f(lsum)) * kLn2;
        }
        uint16_t* orow = Ks + (wave * QW + li) * KS;
        for (int db = 0; db < D / 32; ++db)
            for (int rg = 0; rg < 4; ++rg) {
                bf16x4 r4;
                for (int u = 0; u < 4; ++u) r4[u] = (__bf16)(o[db][4 * rg + u] * inv);
                *reinterpret_cast<bf16x4*>(orow + 32 * db + 8 * rg + 4 * h) = r4;
            }
        asm volatile("" ::: "memory");   // staged rows are read back by other lanes of the wave
        const int part = lane & (TPR - 1);
        constexpr int rows = 64 / TPR;   // rows per store instruction
        for (int i = 0; i < QW / rows; ++i) {
            const int r = rows * i + (lane >> TPR_LOG);
            const uint4 v = *reinterpret_cast<const uint4*>(Ks + (wave * QW + r) * KS + 8 * part);
            const unsigned off = r < nq ? addr(wq0 + r) + 16 * part : kOutside;   // tail rows: dropped
            // non-temporal: the output is not read again by this layer, and its lines should not
            // displace inputs that a layer fitting the last-level cache reads again
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), orr, off, 0, kStoreNT);
        }
    }
}

}  // namespace

template <int D>
const void* plain_kernel(const SwinArgs& a) {
    return a.n_grids > 1 ? reinterpret_cast<const void*>(&swin_fwd_bf16_kernel<true, false, D>)
                         : reinterpret_cast<const void*>(&swin_fwd_bf16_kernel<false, false, D>);
}

hipError_t launch_swin_fwd_bf16(const SwinArgs& a, hipStream_t stream) {
    SwinArgs args = a;
    void* params[] = {&args};
    const void* fn;
    if (a.rope)   // head_dim 64 only (the host checks)
        fn = a.n_grids > 1 ? reinterpret_cast<const void*>(&swin_fwd_bf16_kernel<true, true, kHeadDim>)
                           : reinterpret_cast<const void*>(&swin_fwd_bf16_kernel<false, true, kHeadDim>);
    else
        fn = a.head_dim == 32 ? plain_kernel<32>(a) : a.head_dim == 128 ? plain_kernel<128>(a) : plain_kernel<64>(a);
    return hipLaunchKernel(fn, dim3((unsigned)fwd_bf16_groups(a)), dim3(THREADS), params, 0, stream);
}

}  // namespace fla
