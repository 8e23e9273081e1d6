// C ABI of the Flash Swin attention library: argument checks, launch geometry,
// architecture probe, status strings and algorithmic work counts.
// The operation and the argument contract are stated in include/fla_swin.h.
#include "fla_swin.h"

#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstring>

#include "fla_cycle_scan.h"
#include "fla_swin_internal.h"

static_assert(fla::kScratchBytes == FLA_SCRATCH_BYTES, "static scratch size of the header and the kernels");

namespace {

constexpr int64_t kMaxElems = int64_t(1) << 40;
constexpr int64_t kLastLevelCacheBytes = int64_t(256) << 20;   // MI355X Infinity Cache
constexpr int64_t kMaxGroups = (int64_t(1) << 23) - 1;   // grid.x * 512 threads < 2^32

// Windows of a grid list: the canvas has `origin` virtual tokens in front of each axis;
// window i of an axis covers canvas [i*window, (i+1)*window) = grid [i*window - origin, ...).
struct Geometry {
    int origin, nqb, nbb, n_windows;   // nbb: bf16 backward blocks of kBwdBlock tokens
    int64_t L;                   // tokens per batch entry
    int64_t n_groups;
    fla::GridDesc grid[fla::kMaxGrids];
};

int64_t windows_along(int64_t len, int window, int origin) {
    return len > 0 ? (len + origin + window - 1) / window : 0;
}

// Largest extent of a window along an axis of `len` tokens: the first window (clipped by the
// origin), the last one (clipped by the end) and, when there are three or more, a full one.
int64_t max_extent(int64_t len, int window, int origin) {
    const int64_t n = windows_along(len, window, origin);
    if (n == 0) return 0;
    const int64_t first = len < window - origin ? len : window - origin;
    const int64_t start_last = (n - 1) * window - origin;
    const int64_t last = len - (start_last > 0 ? start_last : 0);
    int64_t m = first > last ? first : last;
    if (n >= 3 && window > m) m = window;
    return m;
}

// Fills `g` for n grids of (hw[2i], hw[2i+1]) tokens; false if a count overflows int.
bool geometry(int B, int heads, int n, const int* hw, int window, int shift, Geometry* g) {
    g->origin = (window - shift) % window;
    int64_t nmax = 0, wins = 0, L = 0;
    for (int i = 0; i < n; ++i) {
        const int H = hw[2 * i], W = hw[2 * i + 1];
        const int64_t nwy = windows_along(H, window, g->origin);
        const int64_t nwx = windows_along(W, window, g->origin);
        fla::GridDesc& d = g->grid[i];
        d.H = H;
        d.W = W;
        d.nwx = (int)nwx;
        d.win_begin = (int)wins;
        d.tok_off = L;
        d.div_nwx = fla::FastDiv::make((unsigned)(nwx > 0 ? nwx : 1));
        const int64_t rows = max_extent(H, window, g->origin), cols = max_extent(W, window, g->origin);
        if (rows * cols > nmax) nmax = rows * cols;
        wins += nwy * nwx;
        L += int64_t(H) * W;
        if (wins > (int64_t(1) << 30)) return false;
    }
    g->n_windows = (int)wins;
    g->L = L;
    g->nqb = (int)((nmax + fla::kQueryBlock - 1) / fla::kQueryBlock);
    g->nbb = (int)((nmax + fla::kBwdBlock - 1) / fla::kBwdBlock);
    g->n_groups = int64_t(B) * heads * wins * g->nqb;
    return true;
}

bool overlaps(const void* a, int64_t a_bytes, const void* b, int64_t b_bytes) {
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
    return a0 < b0 + uint64_t(b_bytes) && b0 < a0 + uint64_t(a_bytes);
}

// Size checks shared by every entry point.  Returns FLA_OK and sets *empty when there is
// nothing to compute.
int check_sizes(int B, int heads, int n, const int* hw, bool* empty) {
    *empty = false;
    if (B < 0 || heads < 0) return FLA_ERR_SHAPE;
    bool any = false;
    for (int i = 0; i < n; ++i) {
        if (hw[2 * i] < 0 || hw[2 * i + 1] < 0) return FLA_ERR_SHAPE;
        any = any || (hw[2 * i] > 0 && hw[2 * i + 1] > 0);
    }
    *empty = B == 0 || heads == 0 || !any;
    return FLA_OK;
}

// plain_forward: the head_dim instances of the plain forward kernels (32, 64, 128) are
// admitted; every other path takes 64.
int check_scalars(int head_dim, int window, int shift, int pad_mode, bool plain_forward = false) {
    if (plain_forward ? !fla::fwd_head_dim_ok(head_dim) : head_dim != fla::kHeadDim) return FLA_ERR_HEAD_DIM;
    if (window < 1) return FLA_ERR_WINDOW;
    if (shift < 0 || shift >= window) return FLA_ERR_SHIFT;
    if (pad_mode != FLA_PAD_MASK && pad_mode != FLA_PAD_KVTOKEN) return FLA_ERR_PAD_MODE;
    return FLA_OK;
}

// Per-device probe result: 0 = not probed yet, -1 = not gfx950, > 0 = gfx950 with that
// many compute units.
std::atomic<int> g_device_cus[64];

int check_arch(int* cus) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
        (void)hipGetLastError();
        return FLA_ERR_ARCH;
    }
    if (dev < 64) {
        const int st = g_device_cus[dev].load(std::memory_order_acquire);
        if (st != 0) {
            *cus = st;
            return st > 0 ? FLA_OK : FLA_ERR_ARCH;
        }
    }
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) {
        (void)hipGetLastError();
        return FLA_ERR_ARCH;
    }
    const bool ok = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 && prop.multiProcessorCount > 0;
    const int st = ok ? prop.multiProcessorCount : -1;
    if (dev < 64) g_device_cus[dev].store(st, std::memory_order_release);
    *cus = st;
    return ok ? FLA_OK : FLA_ERR_ARCH;
}

// Shape and size limits shared by the forward and backward entry points.  Assumes sizes
// and scalars were checked; fills the launch geometry.
struct Problem {
    int64_t L, tok, kv_rows;
    Geometry geo;
};

int check_limits(int B, int heads, int n_grids, const int* hw, int head_dim, int window, int shift,
                 int pad_mode, int elem_bytes, Problem* pr) {
    // sizes, in an order that cannot overflow int64 before the bound check
    int64_t L = 0;
    for (int i = 0; i < n_grids; ++i) {
        if (int64_t(hw[2 * i]) * hw[2 * i + 1] >= kMaxElems) return FLA_ERR_TOO_LARGE;
        L += int64_t(hw[2 * i]) * hw[2 * i + 1];
    }
    const int64_t tok = int64_t(heads) * head_dim;
    const int64_t kv_rows = L + (pad_mode == FLA_PAD_KVTOKEN ? 1 : 0);
    if (kv_rows >= kMaxElems || tok >= kMaxElems || kv_rows > kMaxElems / tok) return FLA_ERR_TOO_LARGE;
    if (B > kMaxElems / (kv_rows * tok)) return FLA_ERR_TOO_LARGE;
    if (!geometry(B, heads, n_grids, hw, window, shift, &pr->geo)) return FLA_ERR_TOO_LARGE;
    // one workgroup per unit or query block, in groups of 8
    if (8 * ((pr->geo.n_groups + 7) / 8) > kMaxGroups) return FLA_ERR_TOO_LARGE;
    // the bf16 forward with several query blocks per window launches them in groups of 8 units
    const int64_t units = int64_t(B) * heads * pr->geo.n_windows;
    if (pr->geo.nqb > 1 && 8 * int64_t(pr->geo.nqb) * ((units + 7) / 8) > kMaxGroups) return FLA_ERR_TOO_LARGE;
    // the kernels address a window with 32-bit byte offsets from its first token, and
    // split a window-local index into (row, col) with a 32-bit multiply-high
    for (int i = 0; i < n_grids; ++i) {
        const int H = hw[2 * i], W = hw[2 * i + 1];
        const int64_t win_rows = window < H ? window : H;
        const int64_t win_cols = window < W ? window : W;
        if (win_rows * W * tok * elem_bytes >= (int64_t(1) << 31)) return FLA_ERR_TOO_LARGE;
        if (win_rows * win_cols * win_cols > (int64_t(1) << 32)) return FLA_ERR_TOO_LARGE;
    }
    pr->L = L;
    pr->tok = tok;
    pr->kv_rows = kv_rows;
    return FLA_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

fla::SwinArgs make_args(const Problem& pr, const void* q, const void* k, const void* v, void* out,
                        float* lse, int B, int heads, int n_grids, int head_dim, int window, int shift,
                        int pad_mode, int cus) {
    const Geometry& geo = pr.geo;
    fla::SwinArgs a;
    a.q = q;
    a.k = k;
    a.v = v;
    a.out = out;
    a.lse = lse;
    a.B = B;
    a.heads = heads;
    a.window = window;
    a.shift = shift;
    a.origin = geo.origin;
    a.nqb = geo.nqb;
    a.pad_mode = pad_mode;
    a.L = pr.L;
    a.tok_stride = pr.tok;
    a.q_batch_stride = pr.L * pr.tok;
    a.kv_batch_stride = pr.kv_rows * pr.tok;
    a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)head_dim));
    a.n_groups = geo.n_groups;
    a.n_units = int64_t(B) * heads * geo.n_windows;
    a.xcd_group = geo.nqb > 1 ? 1 : 0;
    a.n_cus = cus;
    a.n_grids = n_grids;
    a.n_windows = geo.n_windows;
    for (int i = 0; i < fla::kMaxGrids; ++i) a.grid[i] = geo.grid[i < n_grids ? i : 0];
    a.div_heads = fla::FastDiv::make((unsigned)heads);
    a.div_nqb = fla::FastDiv::make((unsigned)geo.nqb);
    a.div_nwin = fla::FastDiv::make((unsigned)geo.n_windows);
    a.head_dim = head_dim;
    a.rope = 0;
    a.rope_scale = 0.f;
    for (float& f : a.rope_rev) f = 0.f;
    for (double& f : a.rope_freq) f = 0.0;
    return a;
}

// 2-D RoPE parameters of the rope entry points (theta: frequency base, scale: position unit)
struct Rope {
    double theta, scale;
};

bool rope_ok(const Rope& r) {
    return std::isfinite(r.theta) && r.theta > 0.0 && std::isfinite(r.scale);
}

void set_rope(fla::SwinArgs* a, const Rope& r) {
    a->rope = 1;
    a->rope_scale = (float)r.scale;
    const int half = fla::kHeadDim / 2;
    for (int j = 0; j < fla::kHeadDim / 4; ++j) {
        a->rope_freq[j] = std::pow(r.theta, -2.0 * j / half);
        a->rope_rev[j] = (float)(a->rope_freq[j] / (2.0 * 3.14159265358979323846));
    }
}

// lse: NULL for the plain forward; the training forward passes want_lse and its buffer.
int forward(const void* q, const void* k, const void* v, void* out, float* lse, bool want_lse, int B,
            int heads, int n_grids, const int* hw, int head_dim, int window, int shift, int pad_mode,
            hipStream_t stream, int elem_bytes, hipError_t (*launch)(const fla::SwinArgs&, hipStream_t),
            const Rope* rope = nullptr) {
    if (n_grids < 1 || n_grids > fla::kMaxGrids) return FLA_ERR_SHAPE;
    if (!hw) return FLA_ERR_NULL;
    bool empty = false;
    int st = check_sizes(B, heads, n_grids, hw, &empty);
    if (st != FLA_OK || empty) return st;
    if (!q || !k || !v || !out || (want_lse && !lse)) return FLA_ERR_NULL;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out) || (want_lse && !aligned16(lse)))
        return FLA_ERR_ALIGN;
    st = check_scalars(head_dim, window, shift, pad_mode, !rope && !want_lse);
    if (st != FLA_OK) return st;
    if (rope && !rope_ok(*rope)) return FLA_ERR_ROPE;
    Problem pr;
    st = check_limits(B, heads, n_grids, hw, head_dim, window, shift, pad_mode, elem_bytes, &pr);
    if (st != FLA_OK) return st;

    const int64_t q_bytes = int64_t(B) * pr.L * pr.tok * elem_bytes;
    const int64_t kv_bytes = int64_t(B) * pr.kv_rows * pr.tok * elem_bytes;
    if (overlaps(out, q_bytes, q, q_bytes) || overlaps(out, q_bytes, k, kv_bytes) ||
        overlaps(out, q_bytes, v, kv_bytes))
        return FLA_ERR_ALIAS;
    if (want_lse) {
        const int64_t lse_bytes = int64_t(B) * heads * pr.L * 4;
        if (overlaps(lse, lse_bytes, q, q_bytes) || overlaps(lse, lse_bytes, k, kv_bytes) ||
            overlaps(lse, lse_bytes, v, kv_bytes) || overlaps(lse, lse_bytes, out, q_bytes))
            return FLA_ERR_ALIAS;
    }

    int cus = 0;
    st = check_arch(&cus);
    if (st != FLA_OK) return st;

    fla::SwinArgs a = make_args(pr, q, k, v, out, want_lse ? lse : nullptr, B, heads, n_grids, head_dim,
                                window, shift, pad_mode, cus);
    if (rope) set_rope(&a, *rope);
    if (launch(a, stream) != hipSuccess) {
        (void)hipGetLastError();
        return FLA_ERR_LAUNCH;
    }
    return FLA_OK;
}

// Workspace bytes of a backward call: one pad-gradient partial per (b, head, window, block)
// in KV-token mode, with the bf16 kernel's blocks of kBwdBlock tokens (at least as many as
// the fp32 kernels' blocks).  Assumes the geometry is valid.
int64_t workspace_bytes(int B, int heads, const Geometry& geo, int pad_mode) {
    if (pad_mode != FLA_PAD_KVTOKEN) return 0;
    return int64_t(B) * heads * geo.n_windows * geo.nbb * fla::kPadPartial * 4;
}

// static_scratch: the workspace is the library's static device scratch (ws and ws_bytes are
// ignored), for the allocation-free entry point.
int backward(const void* q, const void* k, const void* v, const void* out, const void* dout,
             const float* lse, void* dq, void* dk, void* dv, void* ws, size_t ws_bytes, int B,
             int heads, int n_grids, const int* hw, int head_dim, int window, int shift, int pad_mode,
             hipStream_t stream, int elem_bytes, const Rope* rope = nullptr, bool static_scratch = false) {
    if (n_grids < 1 || n_grids > fla::kMaxGrids) return FLA_ERR_SHAPE;
    if (!hw) return FLA_ERR_NULL;
    bool empty = false;
    int st = check_sizes(B, heads, n_grids, hw, &empty);
    if (st != FLA_OK || empty) return st;
    if (!q || !k || !v || !out || !dout || !lse || !dq || !dk || !dv) return FLA_ERR_NULL;
    for (const void* p : {q, k, v, out, dout, static_cast<const void*>(lse), static_cast<const void*>(dq),
                          static_cast<const void*>(dk), static_cast<const void*>(dv)})
        if (!aligned16(p)) return FLA_ERR_ALIGN;
    if (static_scratch) ws = nullptr;
    if (ws && !aligned16(ws)) return FLA_ERR_ALIGN;
    st = check_scalars(head_dim, window, shift, pad_mode);
    if (st != FLA_OK) return st;
    if (rope && !rope_ok(*rope)) return FLA_ERR_ROPE;
    Problem pr;
    st = check_limits(B, heads, n_grids, hw, head_dim, window, shift, pad_mode, elem_bytes, &pr);
    if (st != FLA_OK) return st;
    // the bf16 launch: both roles of every block of every (batch entry, window, head)
    const int64_t units = int64_t(B) * heads * pr.geo.n_windows;
    if (elem_bytes == 2 && fla::bwd_bf16_groups(units, pr.geo.nbb) > kMaxGroups) return FLA_ERR_TOO_LARGE;
    // RoPE training is bf16 only (no fp32 RoPE backward entry point exists)
    if (rope && elem_bytes != 2) return FLA_ERR_UNSUPPORTED;
    const int64_t need = workspace_bytes(B, heads, pr.geo, pad_mode);
    if (static_scratch) {
        if (need > fla::kScratchBytes) return FLA_ERR_SCRATCH;
    } else if (need > 0 && (!ws || ws_bytes < uint64_t(need))) {
        return FLA_ERR_WORKSPACE;
    }

    const int64_t q_bytes = int64_t(B) * pr.L * pr.tok * elem_bytes;
    const int64_t kv_bytes = int64_t(B) * pr.kv_rows * pr.tok * elem_bytes;
    const int64_t lse_bytes = int64_t(B) * heads * pr.L * 4;
    struct Range {
        const void* p;
        int64_t n;
    };
    const Range inputs[] = {{q, q_bytes}, {k, kv_bytes}, {v, kv_bytes}, {out, q_bytes}, {dout, q_bytes},
                            {lse, lse_bytes}};
    // (the static scratch cannot overlap a caller's buffer: only its device address, which
    // the library keeps to itself, reaches it)
    const Range outputs[] = {{dq, q_bytes}, {dk, kv_bytes}, {dv, kv_bytes}, {ws, static_scratch ? 0 : need}};
    for (int i = 0; i < 4; ++i) {
        if (outputs[i].n == 0) continue;
        for (const Range& r : inputs)
            if (overlaps(outputs[i].p, outputs[i].n, r.p, r.n)) return FLA_ERR_ALIAS;
        for (int j = 0; j < i; ++j)
            if (outputs[j].n > 0 && overlaps(outputs[i].p, outputs[i].n, outputs[j].p, outputs[j].n))
                return FLA_ERR_ALIAS;
    }

    int cus = 0;
    st = check_arch(&cus);
    if (st != FLA_OK) return st;
    if (static_scratch && need > 0 && fla::scratch_address(&ws) != hipSuccess) {
        (void)hipGetLastError();
        return FLA_ERR_LAUNCH;
    }

    fla::SwinBwdArgs a;
    a.f = make_args(pr, q, k, v, nullptr, nullptr, B, heads, n_grids, head_dim, window, shift, pad_mode, cus);
    if (rope) set_rope(&a.f, *rope);
    a.out = out;
    a.dout = dout;
    a.lse = lse;
    a.dq = dq;
    a.dk = dk;
    a.dv = dv;
    a.ws = static_cast<float*>(ws);
    // bf16: windows of up to 256 tokens (one 256-query block) take the one-window kernel
    const bool window_kernel = elem_bytes == 2 && pr.geo.nqb == 1;
    a.pad_blocks = elem_bytes != 2 ? pr.geo.nqb : window_kernel ? 1 : pr.geo.nbb;
    a.nbb = pr.geo.nbb;
    a.div_2nbb = fla::FastDiv::make(2u * (unsigned)pr.geo.nbb);
    a.n_units = units;
    a.scale = (float)(1.0 / std::sqrt((double)head_dim));
    // the call's bytes (q, k, v, out, dout read; dq, dk, dv written) against the 256 MB last-level cache
    a.store_nt = 8.0 * B * double(pr.L) * double(pr.tok) * elem_bytes <= double(kLastLevelCacheBytes) ? 1 : 0;
    const hipStream_t s = stream;
    hipError_t e = elem_bytes != 2   ? fla::launch_swin_bwd_f32(a, s)
                   : window_kernel   ? fla::launch_swin_bwd_bf16_window(a, s)
                                     : fla::launch_swin_bwd_bf16_blocks(a, s);
    if (e == hipSuccess && pad_mode == FLA_PAD_KVTOKEN) e = fla::launch_swin_bwd_pad_reduce(a, elem_bytes, s);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return FLA_ERR_LAUNCH;
    }
    return FLA_OK;
}

// Algorithmic work of the windows of one grid: sum of n^2 (and n for windows with virtual
// slots in KV-token mode) over its windows.
double grid_pairs(int H, int W, int window, int shift, int pad_mode) {
    if (H <= 0 || W <= 0) return 0.0;
    const int origin = (window - shift) % window;
    const int64_t nwy = windows_along(H, window, origin), nwx = windows_along(W, window, origin);
    auto extent = [&](int64_t i, int64_t len) -> double {
        int64_t s0 = i * window - origin, s1 = s0 + window;
        if (s0 < 0) s0 = 0;
        if (s1 > len) s1 = len;
        return double(s1 - s0);
    };
    const double full = double(window) * double(window);
    double pairs = 0.0;
    for (int64_t i = 0; i < nwy; ++i) {
        const double a = extent(i, H);
        for (int64_t j = 0; j < nwx; ++j) {
            const double n = a * extent(j, W);
            pairs += n * n;
            if (pad_mode == FLA_PAD_KVTOKEN && n < full) pairs += n;
        }
    }
    return pairs;
}

// backward: five products instead of two (S, dP, dV, dK, dQ), and q, k, v, out, dout read
// with dq, dk, dv written (8 tensors instead of 4) plus the fp32 log-sum-exp per query.
int work(int B, int heads, int n_grids, const int* hw, int head_dim, int window, int shift,
         int pad_mode, int elem_bytes, bool bwd, double* flops, double* bytes) {
    if (n_grids < 1 || n_grids > fla::kMaxGrids) return FLA_ERR_SHAPE;
    if (!hw) return FLA_ERR_NULL;
    bool empty = false;
    int st = check_sizes(B, heads, n_grids, hw, &empty);
    if (st != FLA_OK) return st;
    if (window < 1) return FLA_ERR_WINDOW;
    if (shift < 0 || shift >= window) return FLA_ERR_SHIFT;
    if (pad_mode != FLA_PAD_MASK && pad_mode != FLA_PAD_KVTOKEN) return FLA_ERR_PAD_MODE;
    if (head_dim < 1 || elem_bytes < 1) return FLA_ERR_HEAD_DIM;
    double pairs = 0.0, tokens = 0.0;
    if (!empty)
        for (int i = 0; i < n_grids; ++i) {
            pairs += grid_pairs(hw[2 * i], hw[2 * i + 1], window, shift, pad_mode);
            tokens += double(hw[2 * i]) * hw[2 * i + 1];
        }
    const double pad_rows = pad_mode == FLA_PAD_KVTOKEN ? (bwd ? 4.0 : 2.0) : 0.0;
    const double rows = empty ? 0.0 : (bwd ? 8.0 : 4.0) * tokens + pad_rows;
    if (flops) *flops = (bwd ? 10.0 : 4.0) * head_dim * double(heads) * B * pairs;
    if (bytes)
        *bytes = rows * B * double(heads) * head_dim * elem_bytes + (bwd ? 4.0 * tokens * B * heads : 0.0);
    return FLA_OK;
}

}  // namespace

extern "C" {

int fla_swin_attn_fwd(const void* q, const void* k, const void* v, void* out, int B, int heads,
                      int Hgrid, int Wgrid, int head_dim, int window, int shift, int pad_mode,
                      hipStream_t stream) {
    const int hw[2] = {Hgrid, Wgrid};
    return forward(q, k, v, out, nullptr, false, B, heads, 1, hw, head_dim, window, shift, pad_mode,
                   stream, 2, fla::launch_swin_fwd_bf16);
}

int fla_swin_attn_fwd_f32(const float* q, const float* k, const float* v, float* out, int B,
                          int heads, int Hgrid, int Wgrid, int head_dim, int window, int shift,
                          int pad_mode, hipStream_t stream) {
    const int hw[2] = {Hgrid, Wgrid};
    return forward(q, k, v, out, nullptr, false, B, heads, 1, hw, head_dim, window, shift, pad_mode,
                   stream, 4, fla::launch_swin_fwd_f32);
}

int fla_swin_attn_ms_fwd(const void* q, const void* k, const void* v, void* out, int B, int heads,
                         int n_grids, const int* grid_hw, int head_dim, int window, int shift,
                         int pad_mode, hipStream_t stream) {
    return forward(q, k, v, out, nullptr, false, B, heads, n_grids, grid_hw, head_dim, window, shift,
                   pad_mode, stream, 2, fla::launch_swin_fwd_bf16);
}

int fla_swin_attn_ms_fwd_f32(const float* q, const float* k, const float* v, float* out, int B,
                             int heads, int n_grids, const int* grid_hw, int head_dim, int window,
                             int shift, int pad_mode, hipStream_t stream) {
    return forward(q, k, v, out, nullptr, false, B, heads, n_grids, grid_hw, head_dim, window, shift,
                   pad_mode, stream, 4, fla::launch_swin_fwd_f32);
}

int fla_swin_attn_fwd_lse(const void* q, const void* k, const void* v, void* out, float* lse, int B,
                          int heads, int Hgrid, int Wgrid, int head_dim, int window, int shift,
                          int pad_mode, hipStream_t stream) {
    const int hw[2] = {Hgrid, Wgrid};
    return forward(q, k, v, out, lse, true, B, heads, 1, hw, head_dim, window, shift, pad_mode, stream, 2,
                   fla::launch_swin_fwd_bf16);
}

int fla_swin_attn_fwd_lse_f32(const float* q, const float* k, const float* v, float* out, float* lse,
                              int B, int heads, int Hgrid, int Wgrid, int head_dim, int window,
                              int shift, int pad_mode, hipStream_t stream) {
    const int hw[2] = {Hgrid, Wgrid};
    return forward(q, k, v, out, lse, true, B, heads, 1, hw, head_dim, window, shift, pad_mode, stream, 4,
                   fla::launch_swin_fwd_f32);
}

int fla_swin_attn_ms_fwd_lse(const void* q, const void* k, const void* v, void* out, float* lse,
                             int B, int heads, int n_grids, const int* grid_hw, int head_dim,
                             int window, int shift, int pad_mode, hipStream_t stream) {
    return forward(q, k, v, out, lse, true, B, heads, n_grids, grid_hw, head_dim, window, shift,
                   pad_mode, stream, 2, fla::launch_swin_fwd_bf16);
}

int fla_swin_attn_ms_fwd_lse_f32(const float* q, const float* k, const float* v, float* out,
                                 float* lse, int B, int heads, int n_grids, const int* grid_hw,
                                 int head_dim, int window, int shift, int pad_mode, hipStream_t stream) {
    return forward(q, k, v, out, lse, true, B, heads, n_grids, grid_hw, head_dim, window, shift,
                   pad_mode, stream, 4, fla::launch_swin_fwd_f32);
}

int fla_swin_attn_rope_fwd(const void* q, const void* k, const void* v, void* out, int B, int heads,
                           int Hgrid, int Wgrid, int head_dim, int window, int shift, int pad_mode,
                           float rope_theta, float rope_scale, hipStream_t stream) {
    const int hw[2] = {Hgrid, Wgrid};
    const Rope r{rope_theta, rope_scale};
    return forward(q, k, v, out, nullptr, false, B, heads, 1, hw, head_dim, window, shift, pad_mode,
                   stream, 2, fla::launch_swin_fwd_bf16, &r);
}

int fla_swin_attn_rope_fwd_f32(const float* q, const float* k, const float* v, float* out, int B,
                               int heads, int Hgrid, int Wgrid, int head_dim, int window, int shift,
                               int pad_mode, float rope_theta, float rope_scale, hipStream_t stream) {
    const int hw[2] = {Hgrid, Wgrid};
    const Rope r{rope_theta, rope_scale};
    return forward(q, k, v, out, nullptr, false, B, heads, 1, hw, head_dim, window, shift, pad_mode,
                   stream, 4, fla::launch_swin_fwd_f32, &r);
}

int fla_swin_attn_rope_fwd_lse(const void* q, const void* k, const void* v, void* out, float* lse, int B,
                               int heads, int Hgrid, int Wgrid, int head_dim, int window, int shift,
                               int pad_mode, float rope_theta, float rope_scale, hipStream_t stream) {
    const int hw[2] = {Hgrid, Wgrid};
    const Rope r{rope_theta, rope_scale};
    return forward(q, k, v, out, lse, true, B, heads, 1, hw, head_dim, window, shift, pad_mode, stream, 2,
                   fla::launch_swin_fwd_bf16, &r);
}

int fla_swin_attn_rope_bwd(const void* q, const void* k, const void* v, const void* out, const void* dout,
                           const float* lse, void* dq, void* dk, void* dv, void* workspace,
                           size_t workspace_bytes, int B, int heads, int Hgrid, int Wgrid, int head_dim,
                           int window, int shift, int pad_mode, float rope_theta, float rope_scale,
                           hipStream_t stream) {
    const int hw[2] = {Hgrid, Wgrid};
    const Rope r{rope_theta, rope_scale};
    return backward(q, k, v, out, dout, lse, dq, dk, dv, workspace, workspace_bytes, B, heads, 1, hw,
                    head_dim, window, shift, pad_mode, stream, 2, &r);
}

int fla_swin_attn_bwd_workspace(int B, int heads, int n_grids, const int* grid_hw, int window,
                                int shift, int pad_mode, size_t* bytes) {
    if (n_grids < 1 || n_grids > fla::kMaxGrids) return FLA_ERR_SHAPE;
    if (!grid_hw || !bytes) return FLA_ERR_NULL;
    bool empty = false;
    int st = check_sizes(B, heads, n_grids, grid_hw, &empty);
    if (st != FLA_OK) return st;
    st = check_scalars(fla::kHeadDim, window, shift, pad_mode);
    if (st != FLA_OK) return st;
    if (empty) {
        *bytes = 0;
        return FLA_OK;
    }
    Problem pr;
    st = check_limits(B, heads, n_grids, grid_hw, fla::kHeadDim, window, shift, pad_mode, 2, &pr);
    if (st != FLA_OK) return st;
    *bytes = (size_t)workspace_bytes(B, heads, pr.geo, pad_mode);
    return FLA_OK;
}

int fla_swin_attn_bwd(const void* q, const void* k, const void* v, const void* out, const void* dout,
                      const float* lse, void* dq, void* dk, void* dv, void* workspace,
                      size_t workspace_bytes, int B, int heads, int Hgrid, int Wgrid, int head_dim,
                      int window, int shift, int pad_mode, hipStream_t stream) {
    const int hw[2] = {Hgrid, Wgrid};
    return backward(q, k, v, out, dout, lse, dq, dk, dv, workspace, workspace_bytes, B, heads, 1, hw,
                    head_dim, window, shift, pad_mode, stream, 2);
}

int fla_swin_attn_bwd_noalloc(const void* q, const void* k, const void* v, const void* out,
                              const void* dout, const float* lse, void* dq, void* dk, void* dv, int B,
                              int heads, int Hgrid, int Wgrid, int head_dim, int window, int shift,
                              int pad_mode, hipStream_t stream) {
    const int hw[2] = {Hgrid, Wgrid};
    return backward(q, k, v, out, dout, lse, dq, dk, dv, nullptr, 0, B, heads, 1, hw, head_dim, window,
                    shift, pad_mode, stream, 2, nullptr, true);
}

int fla_swin_attn_bwd_f32(const float* q, const float* k, const float* v, const float* out,
                          const float* dout, const float* lse, float* dq, float* dk, float* dv,
                          void* workspace, size_t workspace_bytes, int B, int heads, int Hgrid,
                          int Wgrid, int head_dim, int window, int shift, int pad_mode, hipStream_t stream) {
    const int hw[2] = {Hgrid, Wgrid};
    return backward(q, k, v, out, dout, lse, dq, dk, dv, workspace, workspace_bytes, B, heads, 1, hw,
                    head_dim, window, shift, pad_mode, stream, 4);
}

int fla_swin_attn_ms_bwd(const void* q, const void* k, const void* v, const void* out,
                         const void* dout, const float* lse, void* dq, void* dk, void* dv,
                         void* workspace, size_t workspace_bytes, int B, int heads, int n_grids,
                         const int* grid_hw, int head_dim, int window, int shift, int pad_mode,
                         hipStream_t stream) {
    return backward(q, k, v, out, dout, lse, dq, dk, dv, workspace, workspace_bytes, B, heads, n_grids,
                    grid_hw, head_dim, window, shift, pad_mode, stream, 2);
}

int fla_swin_attn_ms_bwd_f32(const float* q, const float* k, const float* v, const float* out,
                             const float* dout, const float* lse, float* dq, float* dk, float* dv,
                             void* workspace, size_t workspace_bytes, int B, int heads, int n_grids,
                             const int* grid_hw, int head_dim, int window, int shift, int pad_mode,
                             hipStream_t stream) {
    return backward(q, k, v, out, dout, lse, dq, dk, dv, workspace, workspace_bytes, B, heads, n_grids,
                    grid_hw, head_dim, window, shift, pad_mode, stream, 4);
}

const char* fla_status_string(int status) {
    switch (status) {
        case FLA_OK: return "ok";
        case FLA_ERR_SHAPE: return "B, heads and grid sizes must be >= 0 (1 to 8 grids)";
        case FLA_ERR_NULL: return "a tensor pointer (or the grid list) is NULL";
        case FLA_ERR_ALIGN: return "tensor pointers must be 16-byte aligned";
        case FLA_ERR_HEAD_DIM: return "head_dim must be 64";
        case FLA_ERR_WINDOW: return "window must be >= 1";
        case FLA_ERR_SHIFT: return "shift must satisfy 0 <= shift < window";
        case FLA_ERR_PAD_MODE: return "pad_mode must be FLA_PAD_MASK (0) or FLA_PAD_KVTOKEN (1)";
        case FLA_ERR_TOO_LARGE: return "problem too large (2^40 elements, 2^23 workgroups or a 2 GiB window span)";
        case FLA_ERR_ALIAS: return "an output overlaps an input or another output";
        case FLA_ERR_ARCH: return "no gfx950 (MI355X) device is current";
        case FLA_ERR_LAUNCH: return "kernel launch failed";
        case FLA_ERR_UNSUPPORTED: return "unsupported: Cycle-scan state size N not a power of two up to 32";
        case FLA_ERR_WORKSPACE: return "workspace missing or smaller than fla_swin_attn_bwd_workspace()";
        case FLA_ERR_ROPE: return "rope_theta must be finite and > 0, rope_scale finite";
        case FLA_ERR_SCRATCH: return "problem needs more workspace than the 16 MiB static scratch of the allocation-free backward";
        default: return "unknown status";
    }
}

// ---- Cycle-scan ---------------------------------------------------------------------------

// Sizes of a Cycle-scan call: FLA_ERR_SHAPE for negative sizes or N, repeats below 1; *empty
// when there is nothing to compute.
static int cycle_shape(int B, int L, int d, int N, int repeats, bool* empty) {
    if (B < 0 || L < 0 || d < 0 || N < 1 || repeats < 1) return FLA_ERR_SHAPE;
    *empty = B == 0 || L == 0 || d == 0;
    return FLA_OK;
}

static int cycle_limits(int B, int L, int d, int N) {
    if (!fla::cycle_states_supported(N)) return FLA_ERR_UNSUPPORTED;
    if (int64_t(B) * L * d >= kMaxElems || int64_t(B) * L * N >= kMaxElems) return FLA_ERR_TOO_LARGE;
    const int T = fla::cycle_chunk(L);
    const int64_t groups = int64_t(B) * ((L + T - 1) / T) * ((d + 63) / 64);
    if (groups > kMaxGroups || (int64_t(B) * d * N + 255) / 256 > kMaxGroups) return FLA_ERR_TOO_LARGE;
    return FLA_OK;
}

int fla_cycle_scan_workspace(int B, int L, int d, int N, int repeats, size_t* bytes) {
    bool empty = false;
    int st = cycle_shape(B, L, d, N, repeats, &empty);
    if (st != FLA_OK) return st;
    if (!bytes) return FLA_ERR_NULL;
    if (empty) {
        *bytes = 0;
        return FLA_OK;
    }
    st = cycle_limits(B, L, d, N);
    if (st != FLA_OK) return st;
    *bytes = (size_t)fla::cycle_workspace_floats(B, L, d, N) * 4;
    return FLA_OK;
}

int fla_cycle_scan_work(int B, int L, int d, int N, int repeats, double* exps, double* bytes) {
    bool empty = false;
    int st = cycle_shape(B, L, d, N, repeats, &empty);
    if (st != FLA_OK) return st;
    if (!exps || !bytes) return FLA_ERR_NULL;
    // one exponential exp(Delta a) per (batch entry, token, channel, state) of the
    // definition; every input read and the output written once
    *exps = double(B) * L * d * N;
    *bytes = 4.0 * (3.0 * B * L * d + 2.0 * B * L * N + double(d) * N);
    return FLA_OK;
}

int fla_cycle_scan(const float* x, const float* delta, const float* A, const float* Bm, const float* Cm,
                   float* y, void* workspace, size_t workspace_bytes, int B, int L, int d, int N,
                   int repeats, hipStream_t stream) {
    bool empty = false;
    int st = cycle_shape(B, L, d, N, repeats, &empty);
    if (st != FLA_OK) return st;
    if (empty) return FLA_OK;
    if (!x || !delta || !A || !Bm || !Cm || !y) return FLA_ERR_NULL;
    const void* ptrs[] = {x, delta, A, Bm, Cm, y, workspace};
    for (const void* p : ptrs)
        if (reinterpret_cast<uintptr_t>(p) & 3u) return FLA_ERR_ALIGN;
    st = cycle_limits(B, L, d, N);
    if (st != FLA_OK) return st;
    const int64_t need = fla::cycle_workspace_floats(B, L, d, N) * 4;
    if (!workspace || workspace_bytes < (size_t)need) return FLA_ERR_WORKSPACE;
    const int64_t xd = int64_t(B) * L * d * 4, bn = int64_t(B) * L * N * 4, an = int64_t(d) * N * 4;
    struct Range {
        const void* p;
        int64_t n;
    };
    const Range inputs[] = {{x, xd}, {delta, xd}, {A, an}, {Bm, bn}, {Cm, bn}};
    const Range outputs[] = {{y, xd}, {workspace, need}};
    for (int i = 0; i < 2; ++i) {
        for (const Range& r : inputs)
            if (overlaps(outputs[i].p, outputs[i].n, r.p, r.n)) return FLA_ERR_ALIAS;
        if (i == 1 && overlaps(outputs[1].p, outputs[1].n, outputs[0].p, outputs[0].n)) return FLA_ERR_ALIAS;
    }
    int cus = 0;
    st = check_arch(&cus);
    if (st != FLA_OK) return st;
    fla::CycleArgs a{};
    a.x = x;
    a.delta = delta;
    a.A = A;
    a.Bm = Bm;
    a.Cm = Cm;
    a.y = y;
    a.T = fla::cycle_chunk(L);
    a.nch = (L + a.T - 1) / a.T;
    a.cgroups = (d + 63) / 64;
    a.ws_h = static_cast<float*>(workspace);
    a.ws_s = a.ws_h + int64_t(B) * a.nch * d * N;
    a.B = B;
    a.L = L;
    a.d = d;
    a.N = N;
    a.repeats = repeats;
    if (fla::launch_cycle_scan(a, stream) != hipSuccess) {
        (void)hipGetLastError();
        return FLA_ERR_LAUNCH;
    }
    return FLA_OK;
}

int fla_swin_attn_work(int B, int heads, int Hgrid, int Wgrid, int head_dim, int window,
                       int shift, int pad_mode, int elem_bytes, double* flops, double* bytes) {
    const int hw[2] = {Hgrid, Wgrid};
    return work(B, heads, 1, hw, head_dim, window, shift, pad_mode, elem_bytes, false, flops, bytes);
}

int fla_swin_attn_ms_work(int B, int heads, int n_grids, const int* grid_hw, int head_dim,
                          int window, int shift, int pad_mode, int elem_bytes, double* flops,
                          double* bytes) {
    return work(B, heads, n_grids, grid_hw, head_dim, window, shift, pad_mode, elem_bytes, false, flops,
                bytes);
}

int fla_swin_attn_bwd_work(int B, int heads, int n_grids, const int* grid_hw, int head_dim,
                           int window, int shift, int pad_mode, int elem_bytes, double* flops,
                           double* bytes) {
    return work(B, heads, n_grids, grid_hw, head_dim, window, shift, pad_mode, elem_bytes, true, flops,
                bytes);
}

}  // extern "C"
