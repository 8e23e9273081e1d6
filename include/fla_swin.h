/* Flash Swin attention (forward and backward) for AMD MI355X (gfx950) -- C ABI.
 *
 * Operation (HRSAM, arXiv 2407.02109):
 *   Eq. 1 (Sec. 3.2) scaled dot-product attention, evaluated independently inside each
 *   shifted window of Sec. 3.3 ("Flash Swin"), with the KV-only padding of Sec. 3.4 /
 *   App. B as an option.  Window partition, cyclic shift, border padding and masking all
 *   happen inside one kernel launch; no reordered copy of q, k, v or out is made.
 *
 * Semantics.  Tokens sit on an Hgrid x Wgrid grid in raster order (token j at row
 * j / Wgrid, column j % Wgrid; Sec. 3.3's vanilla map).  Along each axis, coordinate c
 * belongs to region floor((c - shift) / window) (floor division).  This is the paper's
 * construction -- window - shift virtual tokens in front of the axis, unshifted windows on
 * the padded canvas, virtual tokens dropped -- extended to any 0 <= shift < window and to
 * grids that are not a multiple of the window (then the last windows are cut off by the
 * grid border, like the first ones).  For every query token (b, y, x) and head h:
 *
 *   R      = { tokens (y', x') of the grid : same row region as y, same column region as x }
 *   z_j    = <q[b, y*W + x, h, :], k[b, j, h, :]> / sqrt(head_dim)          (j in R)
 *   out    = sum_j softmax(z)_j * v[b, j, h, :]                       (FLA_PAD_MASK)
 *
 * FLA_PAD_KVTOKEN (Sec. 3.4, App. B): every key slot of the query's window x window
 * canvas square that is not a grid token reads the learnable pad token stored at row
 * L = Hgrid*Wgrid of k and v; it enters the softmax once per such slot, i.e. with
 * multiplicity n_pad = window^2 - |R|.  Queries are never padded.
 *
 * Layout.  q and out: [B, Hgrid*Wgrid, heads, head_dim], contiguous, row-major.
 * k and v: the same, or [B, Hgrid*Wgrid + 1, heads, head_dim] in FLA_PAD_KVTOKEN mode
 * (row L is the pad token of each batch entry and head).  All four are device pointers
 * owned by the caller; the library never allocates, frees, copies or synchronises.
 * q, k and v may alias each other; out must not overlap any of them.
 *
 * Errors.  Each entry point checks its arguments in this order and returns the first
 * failure without launching anything and without touching any output: FLA_ERR_SHAPE
 * (n_grids, then negative sizes), FLA_ERR_NULL, FLA_ERR_ALIGN, FLA_ERR_HEAD_DIM,
 * FLA_ERR_WINDOW, FLA_ERR_SHIFT, FLA_ERR_PAD_MODE, FLA_ERR_ROPE, FLA_ERR_TOO_LARGE,
 * FLA_ERR_UNSUPPORTED (Cycle-scan only), FLA_ERR_WORKSPACE (or FLA_ERR_SCRATCH), FLA_ERR_ALIAS,
 * FLA_ERR_ARCH, FLA_ERR_LAUNCH.
 * An empty problem (B, heads, Hgrid or Wgrid equal to 0) returns FLA_OK at once and
 * ignores the pointers.  Launches are asynchronous on `stream` (NULL = the null stream):
 * a fault during execution surfaces at the caller's next synchronisation, not here.  The
 * library is stateless apart from a per-device architecture probe and is safe to call
 * from several threads.
 */
#ifndef FLA_SWIN_H
#define FLA_SWIN_H

#include <stddef.h>

#include <hip/hip_runtime_api.h>   /* hipStream_t */

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    FLA_PAD_MASK = 0,     /* virtual / out-of-grid key slots are excluded from the softmax */
    FLA_PAD_KVTOKEN = 1   /* virtual key slots read the pad token at row L of k and v       */
} fla_pad_mode;

typedef enum {
    FLA_OK = 0,
    FLA_ERR_NULL = 1,      /* a pointer is NULL on a non-empty problem (the grid list of the
                              multi-scale entry points: always)                           */
    FLA_ERR_ALIGN = 2,     /* a pointer is not 16-byte aligned (Cycle-scan: 4-byte)         */
    FLA_ERR_SHAPE = 3,     /* B, heads, Hgrid or Wgrid negative; n_grids not in 1..8;
                              Cycle-scan: B, L, d negative, N or repeats below 1          */
    FLA_ERR_HEAD_DIM = 4,  /* head_dim is not supported (64; the plain forwards, bf16 and
                              fp32, one grid or several, also take 32 and 128)            */
    FLA_ERR_WINDOW = 5,    /* window < 1                                                   */
    FLA_ERR_SHIFT = 6,     /* shift < 0 or shift >= window                                 */
    FLA_ERR_PAD_MODE = 7,  /* pad_mode is neither FLA_PAD_MASK nor FLA_PAD_KVTOKEN         */
    FLA_ERR_ALIAS = 8,     /* an output (out, lse, dq, dk, dv, workspace) overlaps an input
                              or another output                                          */
    FLA_ERR_ARCH = 9,      /* the current device is not gfx950, or no device is present   */
    FLA_ERR_LAUNCH = 10,   /* the HIP runtime refused the kernel launch                    */
    FLA_ERR_TOO_LARGE = 11, /* a tensor has 2^40 elements or more, the launch would need
                              2^23 workgroups or more, the rows of one window span 2 GiB or
                              more (min(window, Hgrid) * Wgrid * heads * head_dim * element
                              bytes), or min(window,Hgrid) * min(window,Wgrid)^2 > 2^32     */
    FLA_ERR_UNSUPPORTED = 12, /* Cycle-scan with N not a power of two up to 32          */
    FLA_ERR_WORKSPACE = 13, /* backward, Cycle-scan: workspace NULL or smaller than the
                               matching _workspace() function reports                     */
    FLA_ERR_ROPE = 14,     /* RoPE entry points: rope_theta not finite and > 0, or
                              rope_scale not finite                                       */
    FLA_ERR_SCRATCH = 15   /* allocation-free backward: the problem needs more workspace than
                              the library's static scratch holds (FLA_SCRATCH_BYTES)      */
} fla_status;

/* bf16 forward (storage: 16-bit bfloat16, round-to-nearest-even on output).
 * Q.K^T and P.V run on bf16 matrix cores with fp32 accumulation; softmax in fp32;
 * P is rounded to bf16 before P.V.  head_dim 64 (the model's), 32 or 128.  Returns an
 * fla_status. */
int fla_swin_attn_fwd(const void* q, const void* k, const void* v, void* out,
                      int B, int heads, int Hgrid, int Wgrid, int head_dim,
                      int window, int shift, int pad_mode, hipStream_t stream);

/* fp32 forward: same operation and layout with float tensors, computed entirely in
 * fp32 (used for tight-tolerance checks on small grids); head_dim 64, 32 or 128.  Returns
 * an fla_status. */
int fla_swin_attn_fwd_f32(const float* q, const float* k, const float* v, float* out,
                          int B, int heads, int Hgrid, int Wgrid, int head_dim,
                          int window, int shift, int pad_mode, hipStream_t stream);

/* Static, NUL-terminated description of a status code (never NULL). */
const char* fla_status_string(int status);

/* Algorithmic work of one call, host arithmetic only (no device access):
 *   *flops = 4 * head_dim * heads * B * (sum over windows of n^2), plus one pad key per
 *            query of a window with virtual slots in FLA_PAD_KVTOKEN mode; n is the number
 *            of grid tokens in the window (Q.K^T and P.V, masked pairs not counted);
 *   *bytes = elem_bytes * heads * head_dim * B * (4 * Hgrid * Wgrid (+2 pad rows)):
 *            q, k, v read once and out written once.
 * Either output pointer may be NULL.  Returns FLA_OK or the argument status code. */
int fla_swin_attn_work(int B, int heads, int Hgrid, int Wgrid, int head_dim,
                       int window, int shift, int pad_mode, int elem_bytes,
                       double* flops, double* bytes);

/* Multi-scale forward (HRSAM++, Sec. 3.6 "Multi-scale Fusion" and App. C): one launch over
 * a sequence that holds the tokens of n_grids grids one after the other -- in the paper the
 * image grid followed by the anchor-map grid.  grid_hw is a host array of 2 * n_grids ints,
 * (H_0, W_0, H_1, W_1, ...); grid g's tokens are rows [off_g, off_g + H_g*W_g) of each batch
 * entry, off_g = sum of the earlier grids' H*W, each grid in raster order.
 *
 * Every grid gets the shifted-window attention defined above on its own tokens (windows never
 * span two grids; window, shift and pad_mode are shared).  In FLA_PAD_KVTOKEN mode all grids
 * share one pad token, the row L = sum of H_g*W_g of k and v (App. C's KV-only padding with a
 * shared learnable token).  With n_grids = 1 this is exactly fla_swin_attn_fwd.
 *
 * Layout: q and out [B, L, heads, head_dim]; k and v [B, L (+1), heads, head_dim].  Errors
 * as above: n_grids outside 1..8 is FLA_ERR_SHAPE, grid_hw NULL is FLA_ERR_NULL (both checked
 * before anything else), a negative H_g or W_g is FLA_ERR_SHAPE, a problem whose grids all
 * have no tokens is empty, and the size limits of FLA_ERR_TOO_LARGE apply to every grid. */
int fla_swin_attn_ms_fwd(const void* q, const void* k, const void* v, void* out,
                         int B, int heads, int n_grids, const int* grid_hw, int head_dim,
                         int window, int shift, int pad_mode, hipStream_t stream);

/* fp32 multi-scale forward: the same with float tensors, computed entirely in fp32. */
int fla_swin_attn_ms_fwd_f32(const float* q, const float* k, const float* v, float* out,
                             int B, int heads, int n_grids, const int* grid_hw, int head_dim,
                             int window, int shift, int pad_mode, hipStream_t stream);

/* Algorithmic work of one multi-scale call: fla_swin_attn_work summed over the grids, with
 * one shared pad row instead of one per grid. */
int fla_swin_attn_ms_work(int B, int heads, int n_grids, const int* grid_hw, int head_dim,
                          int window, int shift, int pad_mode, int elem_bytes,
                          double* flops, double* bytes);

/* Forward with 2-D rotary position embedding fused into its prologue (HRSAM uses RoPE in
 * place of SAM's relative position bias, Sec. 3.1).  The attention above is applied to
 * rotated q' and k' (v unchanged): for token (y, x) and channel pair (2j, 2j+1) of the
 * first half of a head, (q[2j], q[2j+1]) is turned by the angle (y * rope_scale) * f_j,
 * in the second half by (x * rope_scale) * f_j, f_j = rope_theta^(-2j / (head_dim / 2)),
 * j = 0 .. head_dim/4 - 1; likewise k.  (y, x) are grid coordinates; the pad token of
 * FLA_PAD_KVTOKEN mode has no position and is not rotated.  The rotation runs in fp32 on
 * the loaded values (bf16: rounded back to bf16 before the products), so no rotated copy of
 * q or k is written.  rope_theta = 10000, rope_scale = 1 is RoFormer's choice.  Any window:
 * the bf16 kernel takes (cos, sin) from a per-window table when the window's rectangle fits
 * 32 x 32 and computes them per rotated piece otherwise, with the same fp32 arithmetic, so
 * the result does not depend on the route.  Errors as for fla_swin_attn_fwd (head_dim 64
 * only), plus FLA_ERR_ROPE. */
int fla_swin_attn_rope_fwd(const void* q, const void* k, const void* v, void* out,
                           int B, int heads, int Hgrid, int Wgrid, int head_dim,
                           int window, int shift, int pad_mode, float rope_theta,
                           float rope_scale, hipStream_t stream);
int fla_swin_attn_rope_fwd_f32(const float* q, const float* k, const float* v, float* out,
                               int B, int heads, int Hgrid, int Wgrid, int head_dim,
                               int window, int shift, int pad_mode, float rope_theta,
                               float rope_scale, hipStream_t stream);

/* bf16 RoPE training forward: fla_swin_attn_rope_fwd, and also lse as in
 * fla_swin_attn_fwd_lse (of the rotated logits).  Errors as for fla_swin_attn_rope_fwd and
 * fla_swin_attn_fwd_lse.  (RoPE training is bf16 only: there is no fp32 variant.) */
int fla_swin_attn_rope_fwd_lse(const void* q, const void* k, const void* v, void* out, float* lse,
                               int B, int heads, int Hgrid, int Wgrid, int head_dim,
                               int window, int shift, int pad_mode, float rope_theta,
                               float rope_scale, hipStream_t stream);

/* ---------------------------------------------------------------------------------------
 * Training: the forward that keeps the log-sum-exp, and the backward pass.
 *
 * The paper trains HRSAM through Flash Swin attention (App. D); the gradients are those of
 * the operation above.  With c = 1/sqrt(head_dim), for a query i with key set R_i (plus, in
 * FLA_PAD_KVTOKEN mode, the pad token p with weight w_p = n_pad; w_j = 1 otherwise):
 *
 *   LSE_i = log sum_j w_j exp(c <q_i, k_j>)            P_ij = w_j exp(c <q_i, k_j> - LSE_i)
 *   D_i   = <dout_i, out_i>                            dS_ij = P_ij (<dout_i, v_j> - D_i)
 *   dq_i  = c sum_j dS_ij k_j     dk_j = c sum_i dS_ij q_i     dv_j = sum_i P_ij dout_i
 *
 * dk and dv of the pad token (row L) sum over every query of every window that has virtual
 * slots.  P is recomputed from q, k and LSE; nothing of size n^2 is stored.
 * --------------------------------------------------------------------------------------- */

/* Training forward: fla_swin_attn_fwd, and also lse [B, heads, L] (fp32, contiguous):
 * LSE_i above, the natural log of each query's softmax denominator.  Training (this, the
 * backward and RoPE) takes head_dim 64 only.  lse is a device
 * pointer, non-NULL, 16-byte aligned, and must not overlap q, k, v or out.  In bf16 the
 * denominator is the sum of the bf16-rounded probabilities the output uses. */
int fla_swin_attn_fwd_lse(const void* q, const void* k, const void* v, void* out, float* lse,
                          int B, int heads, int Hgrid, int Wgrid, int head_dim,
                          int window, int shift, int pad_mode, hipStream_t stream);
int fla_swin_attn_fwd_lse_f32(const float* q, const float* k, const float* v, float* out,
                              float* lse, int B, int heads, int Hgrid, int Wgrid, int head_dim,
                              int window, int shift, int pad_mode, hipStream_t stream);
int fla_swin_attn_ms_fwd_lse(const void* q, const void* k, const void* v, void* out, float* lse,
                             int B, int heads, int n_grids, const int* grid_hw, int head_dim,
                             int window, int shift, int pad_mode, hipStream_t stream);
int fla_swin_attn_ms_fwd_lse_f32(const float* q, const float* k, const float* v, float* out,
                                 float* lse, int B, int heads, int n_grids, const int* grid_hw,
                                 int head_dim, int window, int shift, int pad_mode, hipStream_t stream);

/* Workspace the backward needs, in bytes (host arithmetic only): in FLA_PAD_KVTOKEN mode 512
 * bytes per (batch entry, head, window, block), each block's share of the pad token's
 * gradient, where the blocks are the 128-token pieces of the largest window (nbb =
 * ceil(max window tokens / 128)); 0 in FLA_PAD_MASK mode.  The fp32 entry points need at most
 * as much.  Single-grid callers pass n_grids = 1 and grid_hw = {Hgrid, Wgrid}.  Argument
 * errors as for the forward; bytes must be non-NULL (FLA_ERR_NULL). */
int fla_swin_attn_bwd_workspace(int B, int heads, int n_grids, const int* grid_hw, int window,
                                int shift, int pad_mode, size_t* bytes);

/* bf16 backward.  Inputs: q, k, v and dout as for the forward, out and lse as the training
 * forward wrote them.  Outputs: dq (layout of q), dk and dv (layout of k and v; in
 * FLA_PAD_KVTOKEN mode row L holds the pad token's gradient).  Every output element is
 * written; nothing is accumulated into what the buffers held.  workspace: device memory
 * of at least fla_swin_attn_bwd_workspace() bytes (may be NULL when that is 0), contents
 * ignored on entry.  All pointers are device pointers, 16-byte aligned.  Inputs may alias
 * each other; dq, dk, dv and the workspace must not overlap any input or each other.
 * S = Q.K^T, dP = dO.V^T, dV = P^T.dO, dK = dS^T.Q and dQ = dS.K run on bf16 matrix cores
 * with fp32 accumulation (P and dS rounded to bf16 before their products); outputs are
 * rounded to bf16 (RNE).  The result does not depend on scheduling (fixed summation
 * order).  Any window size: windows of up to 256 tokens are taken whole by one workgroup;
 * wider ones in 128-token blocks, one workgroup per block computing dK and dV of its keys
 * over all the window's queries and another dQ of its queries over all the keys.
 * Errors: checked in the order
 * stated at the top of this header (FLA_ERR_WORKSPACE after FLA_ERR_TOO_LARGE, before
 * FLA_ERR_ALIAS); nothing is launched and no output is touched on error.
 * Asynchronous on `stream`: one kernel, and the pad-gradient reduction in FLA_PAD_KVTOKEN
 * mode. */
int fla_swin_attn_bwd(const void* q, const void* k, const void* v, const void* out,
                      const void* dout, const float* lse, void* dq, void* dk, void* dv,
                      void* workspace, size_t workspace_bytes, int B, int heads, int Hgrid,
                      int Wgrid, int head_dim, int window, int shift, int pad_mode, hipStream_t stream);

/* Allocation-free bf16 backward, for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): fla_swin_attn_bwd
 * with the same kernels and results, whose workspace is instead a static device array of
 * FLA_SCRATCH_BYTES inside the library.  The library and its callers allocate nothing for it:
 * each device holds its own copy from the moment the library is loaded on it until the process
 * ends; its device address is looked up once per device, on this entry point's first call there.
 * No part of it needs clearing between calls (every workgroup writes its whole share before it
 * is read).  All calls on one device share that device's array: calls that may run at the same
 * time on one device (on different streams, or from several host threads without ordering)
 * race on it and must be serialised by the caller.  Arguments, layout, results and errors as
 * for fla_swin_attn_bwd, with FLA_ERR_SCRATCH (in place of FLA_ERR_WORKSPACE) when
 * fla_swin_attn_bwd_workspace() exceeds FLA_SCRATCH_BYTES. */
#define FLA_SCRATCH_BYTES (16u << 20)
int fla_swin_attn_bwd_noalloc(const void* q, const void* k, const void* v, const void* out,
                              const void* dout, const float* lse, void* dq, void* dk, void* dv, int B,
                              int heads, int Hgrid, int Wgrid, int head_dim, int window, int shift,
                              int pad_mode, hipStream_t stream);

/* fp32 backward: the same with float tensors, computed entirely in fp32, any window size. */
int fla_swin_attn_bwd_f32(const float* q, const float* k, const float* v, const float* out,
                          const float* dout, const float* lse, float* dq, float* dk, float* dv,
                          void* workspace, size_t workspace_bytes, int B, int heads, int Hgrid,
                          int Wgrid, int head_dim, int window, int shift, int pad_mode,
                          hipStream_t stream);

/* Multi-scale backward (App. C): the backward of fla_swin_attn_ms_fwd; the shared pad
 * token's gradient sums over all grids. */
int fla_swin_attn_ms_bwd(const void* q, const void* k, const void* v, const void* out,
                         const void* dout, const float* lse, void* dq, void* dk, void* dv,
                         void* workspace, size_t workspace_bytes, int B, int heads, int n_grids,
                         const int* grid_hw, int head_dim, int window, int shift, int pad_mode,
                         hipStream_t stream);
int fla_swin_attn_ms_bwd_f32(const float* q, const float* k, const float* v, const float* out,
                             const float* dout, const float* lse, float* dq, float* dk, float* dv,
                             void* workspace, size_t workspace_bytes, int B, int heads,
                             int n_grids, const int* grid_hw, int head_dim, int window, int shift,
                             int pad_mode, hipStream_t stream);

/* bf16 RoPE backward: the gradients of fla_swin_attn_rope_fwd with respect to the unrotated q, k
 * and v.  Inside, q and k are rotated as they are loaded (as in the forward) and the
 * gradients at the rotated values are rotated back by the transpose of each token's
 * rotation (dq = R^T dq', dk = R^T dk'); dv is unchanged, and the pad token, which is never
 * rotated, gets its gradient as in fla_swin_attn_bwd.  out and lse are those of
 * fla_swin_attn_rope_fwd_lse.  Arguments and errors as for fla_swin_attn_bwd, plus
 * FLA_ERR_ROPE (checked after FLA_ERR_PAD_MODE). */
int fla_swin_attn_rope_bwd(const void* q, const void* k, const void* v, const void* out,
                           const void* dout, const float* lse, void* dq, void* dk, void* dv,
                           void* workspace, size_t workspace_bytes, int B, int heads, int Hgrid,
                           int Wgrid, int head_dim, int window, int shift, int pad_mode,
                           float rope_theta, float rope_scale, hipStream_t stream);

/* Algorithmic work of one backward call:
 *   *flops = 10 * head_dim * heads * B * pairs (pairs as in fla_swin_attn_work: the five
 *            products S, dP, dV, dK, dQ over the unmasked pairs and pad keys);
 *   *bytes = elem_bytes * heads * head_dim * B * (8 * L (+4 pad rows)) + 4 * B * heads * L:
 *            q, k, v, out, dout read once, dq, dk, dv written once, lse read once. */
int fla_swin_attn_bwd_work(int B, int heads, int n_grids, const int* grid_hw, int head_dim,
                           int window, int shift, int pad_mode, int elem_bytes,
                           double* flops, double* bytes);

/* ---- Cycle-scan (HRSAM Sec. 3.5) -------------------------------------------------------
 *
 * The Cycle-scan module's state space model over the token sequence, fp32.  Every channel
 * c of a d-channel sequence is scanned on its own with N states, a diagonal A, and the
 * zero-order hold of the SSM equations of Sec. 3.5 (Delta, B and C given per token, as in
 * the selective scan of Mamba, which the paper uses):
 *   h_t = Abar_t h_{t-1} + Bbar_t x_t,   y_t = sum_n C_t[n] h_t[n],
 *   Abar_t[n] = exp(delta_t[c] A[c][n]),  Bbar_t[n] = (exp(delta_t[c] A[c][n]) - 1) / A[c][n] * B_t[n].
 * Cycle-scan lays the sequence out `repeats` times one after the other (the paper uses 3),
 * scans the repeats * L tokens in that order from h = 0 (the state runs on from one copy
 * into the next), cuts the output into the copies and sums them:
 *   y[b, t, c] = sum_{k<repeats} (scan output at position k L + t).
 * The copies are never formed; the kernels take two passes over the data (see the kernel
 * source for the algebra).
 *
 * Layout (fp32, contiguous, row-major, device pointers, 4-byte aligned):
 *   x, delta, y [B, L, d]  (token-major, channels contiguous: the attention's token layout);
 *   A [d, N]               (the diagonal of each channel's A: negative, as Mamba's -exp(A_log);
 *                           A = 0 is not supported and yields NaN);
 *   Bm, Cm [B, L, N]       (B_t and C_t of each token, shared by the channels).
 * delta holds the step sizes (positive; softplus already applied).  N (states per channel)
 * is one of 1, 2, 4, 8, 16, 32 (the paper's Cycle-scan uses 32).
 * Errors, in this order: FLA_ERR_SHAPE (B, L or d negative, N or repeats below 1); then an
 * empty problem (B, L or d equal to 0) returns FLA_OK and ignores the pointers;
 * FLA_ERR_NULL; FLA_ERR_ALIGN (4 bytes); FLA_ERR_UNSUPPORTED (N not one of those); FLA_ERR_TOO_LARGE
 * (x or Bm of 2^40 elements or more, or 2^23 workgroups or more); FLA_ERR_WORKSPACE;
 * FLA_ERR_ALIAS (y or the workspace overlapping an input or each other; inputs may alias
 * each other); FLA_ERR_ARCH; FLA_ERR_LAUNCH.  Nothing is launched and y is not touched on
 * error.  Asynchronous on `stream` (three kernels). */

/* Workspace of fla_cycle_scan, in bytes: N + 1 floats (4 (N + 1) bytes) per (batch entry,
 * chunk, channel), with chunks of 32 to 256 tokens.  Errors as for fla_cycle_scan up to FLA_ERR_TOO_LARGE
 * (bytes must be non-NULL). */
int fla_cycle_scan_workspace(int B, int L, int d, int N, int repeats, size_t* bytes);

/* The Cycle-scan described above.  workspace: device memory of at least
 * fla_cycle_scan_workspace() bytes, contents ignored on entry and overwritten. */
int fla_cycle_scan(const float* x, const float* delta, const float* A, const float* Bm,
                   const float* Cm, float* y, void* workspace, size_t workspace_bytes, int B,
                   int L, int d, int N, int repeats, hipStream_t stream);

/* Algorithmic work of one fla_cycle_scan call (host arithmetic only):
 *   *exps  = B * L * d * N: the exponentials exp(delta A) of the definition, one per
 *            (batch entry, token, channel, state) -- the copies repeat them;
 *   *bytes = 4 * (3 B L d + 2 B L N + d N): x, delta, Bm, Cm, A read once, y written once.
 * Errors: FLA_ERR_SHAPE as for fla_cycle_scan; FLA_ERR_NULL for a NULL output. */
int fla_cycle_scan_work(int B, int L, int d, int N, int repeats, double* exps, double* bytes);

#ifdef __cplusplus
}
#endif

#endif /* FLA_SWIN_H */
