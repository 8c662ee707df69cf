/*
 * gradlev.h - C ABI of the GradLev fast-weight scan library for MI355X (gfx950).
 *
 * GradLev (arXiv 2609.34174) adapts a linear map y_t = W_t x_t by online
 * gradient descent with unit retention (Section 3, Eq. 2):
 *
 *     W_{t+1} = W_t - eta_t g_t x_t^T,      W_t = W_0 + Delta_t,   Delta_0 = 0.
 *
 * Given every token's input x_t and proposed costate g_t up front (Section 3,
 * step 1), the adapted weights are a prefix sum of rank-1 writes and the whole
 * sequence is evaluated in parallel (Section 3, steps 2-3; Appendix C, Eq. 16).
 * This library computes that scan, its backward, and the token-by-token
 * deployment update on the GPU.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - All array arguments are caller-owned DEVICE pointers, row-major and
 *   contiguous, 16-byte aligned.  The library never allocates device memory,
 *   never frees caller memory and keeps no pointer after a call returns.
 * - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL is the
 *   default stream).  Results are valid once the stream has been synchronised.
 * - Every entry point validates its arguments on the host BEFORE touching the
 *   HIP runtime, and returns a status code; nothing is thrown across the ABI.
 *   On any error no work has been enqueued, except GRADLEV_ERR_HIP, which
 *   reports a failed launch.
 * - Outputs must not overlap inputs or each other (decode's W is in/out).
 * - Floating point: X, G and dY are fp32 or bf16 (values as stored, bf16 being
 *   round-to-nearest-even storage).  W_0, eta, fast states and every output are
 *   fp32, following the paper's precision contract of 16-bit activations with
 *   32-bit parameters and fast states (Appendix E, "Numerical implementation").
 *   Contractions run on the MFMA units with fp32 accumulation; fp32 states are
 *   split into two bf16 terms when they meet bf16 operands.
 */
#ifndef GRADLEV_H
#define GRADLEV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Storage type of X, G and dY. */
enum { GRADLEV_F32 = 0, GRADLEV_BF16 = 1 };

/* Read convention of the scans.
 * EXCLUSIVE (the paper's, Section 3 step 2 and Appendix C): token t reads the
 *   weights before its own write, y_t = (W_0 + Delta_t) x_t.
 * INCLUSIVE: token t reads after its own write, y_t = (W_0 + Delta_{t+1}) x_t. */
enum { GRADLEV_EXCLUSIVE = 0, GRADLEV_INCLUSIVE = 1 };

/* Status codes. */
enum {
  GRADLEV_OK = 0,
  GRADLEV_ERR_INVALID = -1,     /* NULL required pointer, non-positive size, bad enum */
  GRADLEV_ERR_UNSUPPORTED = -2, /* valid but outside the compiled shapes */
  GRADLEV_ERR_ALIGN = -3,       /* a pointer is not 16-byte aligned */
  GRADLEV_ERR_WORKSPACE = -4,   /* workspace NULL or smaller than required */
  GRADLEV_ERR_HIP = -5,         /* a HIP launch failed */
  GRADLEV_ERR_SCRATCH = -6      /* gradlev_scan_fwd_static: the call needs more scratch
                                   than GRADLEV_STATIC_SCRATCH_BYTES */
};

/* Problem description for the scans.
 *   B, H      batch and heads; each (b, h) is an independent sequence (>= 1)
 *   T         tokens per sequence (>= 1, any value; a partial last chunk is masked)
 *   d_in      input width d of the adapted map  (64 or 128, or wide: see below)
 *   d_out     output width m of the adapted map (64 or 128, or wide: see below)
 *   chunk     intra-chunk tile length hint: 0 (library default), 64 or 128.
 *             It changes the rounding order only, never the result in exact
 *             arithmetic; the library may use a smaller tile where a kernel's
 *             LDS budget requires it.
 *   segment   tokens per workgroup segment hint: 0 (library default) or a
 *             positive multiple of 64.  Segments of one sequence run in
 *             parallel and are joined by an fp32 carry of their aggregated
 *             writes; like `chunk` it changes the rounding order only.  At
 *             most 16 segments per sequence: a hint giving more is
 *             GRADLEV_ERR_UNSUPPORTED (the default never does), and so is
 *             a plan whose grid, 8 * n_seg * ceil(B*H / 8) workgroups of up
 *             to 1024 work-items, would reach 2^32 work-items.
 *   in_dtype  GRADLEV_F32 or GRADLEV_BF16
 *   prefix    GRADLEV_EXCLUSIVE or GRADLEV_INCLUSIVE */
/* Wide maps.  When d_in or d_out is above 128 (both multiples of 128, at most
 * 8192 - the paper's adapted MLP is 1024 -> 4096 -> 1024) the scans run the
 * parallel form: the chunked form of Appendix C with one chunk spanning the
 * sequence, i.e. y_t = W0 x_t + sum_{s<t} F_ts c_s (x_s . x_t) g_s with
 * c_s = -eta_s and F_ts the retention product (1 without gates), and the
 * transpose read alike.  Results are those of the sequential definition up to
 * rounding.  Limits: exclusive reads only, T <= 16384 (the workspace holds
 * the causal B*H*T*T score matrix: gradlev_scan_workspace_bytes), chunk and
 * segment hints are ignored (the plan reports one chunk of T rounded up to
 * 128).  The backward returns every output of the narrow scans: gtilde and
 * the write side of dX (S_read and its transpose, S_read = F c (dY G^T),
 * contracted with X), dG (the transpose of the forward's scores contracted
 * with dY), deta and dalpha (masked column sums over the pairs of reads and
 * writes; dalpha through Z = K F^T with K = c (dY G^T) o (X X^T)) and dW0.
 * Calls are deterministic: every reduction, including the split of long score
 * contractions, runs in a fixed order. */
typedef struct gradlev_shape {
  int64_t B, H, T, d_in, d_out;
  int64_t chunk;
  int64_t segment;
  int32_t in_dtype;
  int32_t prefix;
} gradlev_shape;

/* How a call will be executed (for callers sizing grids or counting work). */
typedef struct gradlev_plan {
  int64_t fwd_chunk, fwd_segment, fwd_nseg; /* tile, tokens/segment, segments per sequence */
  int64_t bwd_chunk, bwd_segment, bwd_nseg;
  size_t workspace_bytes;                   /* bytes needed by fwd and by bwd */
} gradlev_plan;

/* Fills *plan for shape *s.  Pure host computation, no HIP call.
 * Returns GRADLEV_OK, GRADLEV_ERR_INVALID or GRADLEV_ERR_UNSUPPORTED. */
int gradlev_scan_plan(const gradlev_shape* s, gradlev_plan* plan);

/* Workspace bytes that gradlev_scan_fwd and gradlev_scan_bwd need for *s
 * (written to *bytes; may be 0).  Pure host computation.
 * The workspace is scratch: its contents on entry are ignored and on exit are
 * unspecified.  One workspace must not be shared by calls that may overlap. */
int gradlev_scan_workspace_bytes(const gradlev_shape* s, size_t* bytes);

/* Forward scan (Section 3 step 2, Eq. 3; Appendix C, Eq. 16, first line).
 *
 *   Y[b,h,t,:] = (W0[h] + Delta_t) X[b,h,t,:],
 *   Delta_t    = - sum_{s<t} eta[b,h,s] G[b,h,s,:] X[b,h,s,:]^T   (s<=t if INCLUSIVE)
 *
 *   W0   [H, m, d]     fp32   slow weights W_0, shared over the batch
 *   X    [B, H, T, d]  in_dtype  map inputs x_t
 *   G    [B, H, T, m]  in_dtype  proposed costates g_hat_t
 *   eta  [B, H, T]     fp32   per-token step sizes, or NULL to use eta_scalar
 *   Y    [B, H, T, m]  fp32   output (fully overwritten)
 *   workspace / workspace_bytes: device scratch of at least
 *        gradlev_scan_workspace_bytes(s) bytes (may be NULL if that is 0). */
int gradlev_scan_fwd(const gradlev_shape* s, const float* W0, const void* X,
                     const void* G, const float* eta, float eta_scalar, float* Y,
                     void* workspace, size_t workspace_bytes, void* stream);

/* Forward scan that allocates nothing and takes no workspace, for callers
 * that cannot allocate device memory or pass one: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments, results and kernels as gradlev_scan_fwd; the scratch that
 * gradlev_scan_fwd takes from its workspace argument (segment aggregates, or
 * the wide maps' gate prefixes and score tiles) comes instead from a static
 * device array of GRADLEV_STATIC_SCRATCH_BYTES that the library keeps on
 * each GPU it runs on until the process ends.
 *   - The array of the CURRENT device (hipGetDevice) is used; `stream` must
 *     belong to that device.  Its address is looked up once per device, on
 *     that device's first call.
 *   - Calls whose workspace (gradlev_scan_workspace_bytes) exceeds the array
 *     return GRADLEV_ERR_SCRATCH before any HIP call.
 *   - Every call on one GPU shares that GPU's array, and each call leaves its
 *     contents behind (nothing in it needs to start at zero).  Calls that can
 *     overlap on one GPU - on different streams, or from several host threads
 *     without ordering - race on it: order them on one stream or synchronise
 *     between them. */
#define GRADLEV_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
int gradlev_scan_fwd_static(const gradlev_shape* s, const float* W0, const void* X,
                            const void* G, const float* eta, float eta_scalar, float* Y,
                            void* stream);

/* Backward of the forward scan for an upstream gradient dY = dL/dY.
 *
 * Read side (Section 3 step 3, Eq. 4; Appendix C, Eq. 16, second line) - the
 * paper's grounded costate target for the map input:
 *   gtilde[b,h,t,:] = (W0[h] + Delta_t)^T dY[b,h,t,:]     (Delta_{t+1} if INCLUSIVE)
 * Reverse-time terms (vector-Jacobian product through the prefix sums, with
 * suffix R_t = sum_{u>t} dY_u X_u^T, u>=t if INCLUSIVE):
 *   u_t      = -R_t X_t
 *   dG[t]    = eta_t u_t                       dL/dG
 *   deta[t]  = <G_t, u_t>                      dL/deta
 *   dX[t]    = gtilde_t - eta_t R_t^T G_t      total dL/dX (read + write side)
 *   dW0[h]   = sum_b sum_t dY_t X_t^T          dL/dW0, summed over the batch
 * The paper's own training detaches writes (Appendix E, "Initialization and
 * gradients") and uses gtilde only; pass NULL for outputs you do not need and
 * their work is skipped.  At least one output must be non-NULL.
 *
 *   dY      [B, H, T, m] in_dtype
 *   gtilde  [B, H, T, d] fp32 or NULL      dX [B, H, T, d] fp32 or NULL
 *   dG      [B, H, T, m] fp32 or NULL      deta [B, H, T] fp32 or NULL
 *   dW0     [H, m, d]    fp32 or NULL (overwritten)
 * Other arguments as in gradlev_scan_fwd.  Reductions are in a fixed order, so
 * repeated calls are bitwise identical. */
int gradlev_scan_bwd(const gradlev_shape* s, const float* W0, const void* X,
                     const void* G, const float* eta, float eta_scalar,
                     const void* dY, float* gtilde, float* dX, float* dG,
                     float* deta, float* dW0, void* workspace,
                     size_t workspace_bytes, void* stream);

/* Save-for-backward pair.  A training step that runs the forward and then the
 * backward on the same inputs can let the forward keep the fast weights at the
 * end of each of its token segments (the prefix sums of Section 3 step 2,
 * Eq. 3, at the segment boundaries); the backward then starts every segment
 * from the saved state instead of re-reading X and G to rebuild it, which
 * removes one of its two streaming passes over the inputs.
 *
 * gradlev_scan_saved_bytes: bytes of the saved state (*saved_bytes) and of the
 *   workspace both calls need (*workspace_bytes) for *s.  Pure host
 *   computation.  Both calls of a pair take the same shape, the same segment
 *   hint, and a workspace of at least *workspace_bytes.
 * gradlev_scan_fwd_save: as gradlev_scan_fwd, and also writes the state to
 *   saved [B*H][n_seg][m][d] fp32 (W after the last write of each segment,
 *   row-major; n_seg is private to the plan, only the byte count is public).
 * gradlev_scan_bwd_saved: as gradlev_scan_bwd, reading the state that
 *   gradlev_scan_fwd_save wrote for the same W0, X, G and eta; the caller
 *   keeps that buffer unmodified between the two calls.  Its results equal
 *   gradlev_scan_bwd's up to float32 rounding order.
 * saved must be 16-byte aligned device memory of at least the returned size
 * (GRADLEV_ERR_WORKSPACE otherwise).  Shapes that gradlev_scan_fwd runs in
 * the parallel form (a width above 128) return GRADLEV_ERR_UNSUPPORTED: that
 * form has no segment states. */
int gradlev_scan_saved_bytes(const gradlev_shape* s, size_t* saved_bytes,
                             size_t* workspace_bytes);
int gradlev_scan_fwd_save(const gradlev_shape* s, const float* W0, const void* X,
                          const void* G, const float* eta, float eta_scalar,
                          float* Y, float* saved, size_t saved_bytes,
                          void* workspace, size_t workspace_bytes, void* stream);
int gradlev_scan_bwd_saved(const gradlev_shape* s, const float* W0, const void* X,
                           const void* G, const float* eta, float eta_scalar,
                           const void* dY, const float* saved, size_t saved_bytes,
                           float* gtilde, float* dX, float* dG, float* deta,
                           float* dW0, void* workspace, size_t workspace_bytes,
                           void* stream);

/* Save-for-backward pair with document resets, at unit retention (the
 * paper's LM configuration: retention one, fast state reset at document and
 * packed-row boundaries; Section 3, Eq. 2 holds within each reset segment;
 * Appendix E).  A reset flag at token t starts a new document: t reads W_0
 * plus the writes of its own document, and the backward's suffix of a token
 * ends before the next document.  Results are those of the gated scans with
 * alpha = 1 and the same flags (the tokens a reset overrides have dG = 0,
 * deta = 0 and no write-side dX), computed by the unit-retention kernels:
 * within a 64-token chunk a reset becomes masks (scores pair tokens of one
 * document, rows after the chunk's first reset read W_0, only its last
 * document's writes and reads cross the chunk boundary), and the forward
 * stores the fast weights at the start of each chunk that holds a reset,
 * where the backward cannot take writes back.
 *   reset  [B, T] uint8 (0 or 1, shared by the heads of a batch row), or NULL
 *          (no document starts); a flag at t = 0 changes nothing.
 * Supported: d_in = d_out = 64, exclusive reads (GRADLEV_ERR_UNSUPPORTED
 * otherwise; other widths use the gated pair).  The chunk hint is ignored
 * (both directions use 64-token tiles); segment hints as for the plain pair.
 * gradlev_scan_reset_saved_bytes: bytes of the saved state (segment-end
 *   weights plus room for a state at every chunk start) and of the workspace
 *   both calls need.  Other arguments, ownership and the saved buffer's
 *   rules as in gradlev_scan_fwd_save / gradlev_scan_bwd_saved (dW0 is the
 *   full sum_b sum_t dY_t X_t^T: every read sees W_0). */
int gradlev_scan_reset_saved_bytes(const gradlev_shape* s, size_t* saved_bytes,
                                   size_t* workspace_bytes);
int gradlev_scan_fwd_reset_save(const gradlev_shape* s, const float* W0, const void* X,
                                const void* G, const float* eta, float eta_scalar,
                                const uint8_t* reset, float* Y, float* saved,
                                size_t saved_bytes, void* workspace, size_t workspace_bytes,
                                void* stream);
int gradlev_scan_bwd_reset_saved(const gradlev_shape* s, const float* W0, const void* X,
                                 const void* G, const float* eta, float eta_scalar,
                                 const void* dY, const uint8_t* reset, const float* saved,
                                 size_t saved_bytes, float* gtilde, float* dX, float* dG,
                                 float* deta, float* dW0, void* workspace,
                                 size_t workspace_bytes, void* stream);

/* One deployment step for S sequences x H heads (Section 3, "Training
 * objective", last sentences; Appendix A, last sentence): score with the
 * current weights, then write the true costate.
 *
 *   y[s,h,:]   = W[s,h] x[s,h,:]                       (before the write)
 *   W[s,h]    <- W[s,h] - eta[s,h] g[s,h,:] x[s,h,:]^T
 *
 *   W    [S, H, d_out, d_in] fp32  fast weights, updated in place
 *   x    [S, H, d_in]  fp32        g [S, H, d_out] fp32
 *   eta  [S, H] fp32 or NULL (then eta_scalar)
 *   y    [S, H, d_out] fp32 output
 * Supported: d_in in {16, 32, 64, 128, 256} with d_out in [1, 1024] and
 * S * H < 2^24, or wide states, d_in in {512, 1024, 2048, 4096, 8192} with
 * d_out in [1, 65536] and d_in * d_out * 4 < 2^31 (the paper's LM-width MLP
 * maps are 1024 -> 4096 and 4096 -> 1024).  Larger calls would exceed the
 * 2^32 work-items of one launch and return GRADLEV_ERR_UNSUPPORTED.
 * Exclusive only: deployment needs y before the costate g exists. */
int gradlev_decode_step(int64_t S, int64_t H, int64_t d_in, int64_t d_out,
                        float* W, const float* x, const float* g,
                        const float* eta, float eta_scalar, float* y,
                        void* stream);

/* ------------------------------------------------------------------------
 * Gated scans: retention and document resets (Section 3, Eq. 2, general form)
 * ------------------------------------------------------------------------
 * With a retention alpha_t in [0, 1] per token the write is centered weight
 * decay,
 *
 *     W_{t+1} = W_0 + alpha_t (W_t - W_0) - eta_t g_t x_t^T,
 *     Delta_t = - sum_{i<t} eta_i (prod_{i<j<t} alpha_j) g_i x_i^T,
 *
 * so every earlier write is discounted by the retentions after it and decay
 * pulls towards W_0, not towards zero.  Eq. 2 holds within each reset
 * segment: a token flagged as a reset reads W_0 again (Delta_t = 0).  That
 * is the recurrence with alpha_{t-1} = eta_{t-1} = 0, which is how the kernels
 * apply it; the gate gradients (dalpha, deta) of such a token t-1 are 0.
 *
 *   alpha   [B, H, T] fp32 in [0, 1], or NULL to use alpha_scalar for every token
 *   reset   [B, T] uint8 (0 or 1, shared by the heads of a batch row), or NULL
 *
 * Only the exclusive read is supported (GRADLEV_ERR_UNSUPPORTED otherwise),
 * and one sequence's chunk-start states must stay under 2 GiB:
 * ceil(T / chunk) * d_in * d_out * 4 < 2^31 with the backward's chunk of 32
 * tokens (64 for bf16 64 x 64 maps): T below 2^20 at 128 x 128. */
typedef struct gradlev_gates {
  const float* alpha;
  float alpha_scalar;
  const uint8_t* reset;
} gradlev_gates;

/* Workspace bytes for gradlev_scan_fwd_gated and gradlev_scan_bwd_gated
 * (same rules as gradlev_scan_workspace_bytes).  The backward keeps the
 * fast-weight state at every chunk start of its plan (fp32, B*H*ceil(T/chunk)
 * matrices): retention makes the writes impossible to take back stably. */
int gradlev_scan_gated_workspace_bytes(const gradlev_shape* s, size_t* bytes);

/* Gated forward scan: Y[b,h,t,:] = (W0[h] + Delta_t) X[b,h,t,:] with Delta_t
 * as above.  Arguments as in gradlev_scan_fwd; gates must not be NULL. */
int gradlev_scan_fwd_gated(const gradlev_shape* s, const gradlev_gates* gates,
                           const float* W0, const void* X, const void* G,
                           const float* eta, float eta_scalar, float* Y,
                           void* workspace, size_t workspace_bytes, void* stream);

/* Backward of the gated forward scan.  With Lambda_t = dL/dDelta_t, carried
 * in reverse time as Lambda_t = dY_t X_t^T + alpha_t Lambda_{t+1}:
 *   gtilde[t] = (W0 + Delta_t)^T dY_t
 *   u_t       = -Lambda_{t+1} X_t,   dG[t] = eta_t u_t,   deta[t] = <G_t, u_t>
 *   dX[t]     = gtilde_t - eta_t Lambda_{t+1}^T G_t
 *   dalpha[t] = <Lambda_{t+1}, Delta_t>_F           dL/dalpha (Appendix E keeps gate derivatives)
 *   dW0[h]    = sum_b sum_t dY_t X_t^T              (the decay is centered on W0)
 *   dalpha  [B, H, T] fp32 or NULL; other arguments as in gradlev_scan_bwd. */
int gradlev_scan_bwd_gated(const gradlev_shape* s, const gradlev_gates* gates,
                           const float* W0, const void* X, const void* G,
                           const float* eta, float eta_scalar, const void* dY,
                           float* gtilde, float* dX, float* dG, float* deta,
                           float* dalpha, float* dW0, void* workspace,
                           size_t workspace_bytes, void* stream);

/* Gated save-for-backward pair.  With retention the backward needs Delta at
 * the start of every one of its tiles (Section 3, Eq. 2 with alpha; the
 * writes cannot be taken back, so they are carried forward), which the plain
 * gated backward recomputes in a state pass over X and G.  Here the forward
 * runs on the backward's tile and stores those states as it passes them, and
 * the backward reads them: no state pass, and no write aggregates, so its
 * aggregate pass reads X, dY and the gates but not G.
 *
 * gradlev_scan_gated_saved_bytes: bytes of the saved states (*saved_bytes:
 *   B*H * ceil(T / tile) * m * d * 4, tile 64 for bf16 64 x 64 maps, else 32)
 *   and of the workspace both calls need (*workspace_bytes).  Pure host
 *   computation.  Both calls of a pair take the same shape, the same
 *   segment hint, the same gates and a workspace of at least that size.
 * gradlev_scan_fwd_gated_save: as gradlev_scan_fwd_gated, and also writes
 *   the states into saved (layout private to the library).
 * gradlev_scan_bwd_gated_saved: as gradlev_scan_bwd_gated, reading the
 *   states that gradlev_scan_fwd_gated_save wrote for the same inputs and
 *   gates; the caller keeps that buffer unmodified in between.  Results equal
 *   gradlev_scan_bwd_gated's up to float32 rounding order.
 * saved must be 16-byte aligned device memory of at least the returned size
 * (GRADLEV_ERR_WORKSPACE otherwise).  Wide shapes return
 * GRADLEV_ERR_UNSUPPORTED (the parallel form keeps no states). */
int gradlev_scan_gated_saved_bytes(const gradlev_shape* s, size_t* saved_bytes,
                                   size_t* workspace_bytes);
int gradlev_scan_fwd_gated_save(const gradlev_shape* s, const gradlev_gates* gates,
                                const float* W0, const void* X, const void* G,
                                const float* eta, float eta_scalar, float* Y,
                                float* saved, size_t saved_bytes, void* workspace,
                                size_t workspace_bytes, void* stream);
int gradlev_scan_bwd_gated_saved(const gradlev_shape* s, const gradlev_gates* gates,
                                 const float* W0, const void* X, const void* G,
                                 const float* eta, float eta_scalar, const void* dY,
                                 const float* saved, size_t saved_bytes,
                                 float* gtilde, float* dX, float* dG, float* deta,
                                 float* dalpha, float* dW0, void* workspace,
                                 size_t workspace_bytes, void* stream);

/* Gated deployment step: score with the current weights, then write with
 * centered decay,
 *   y[s,h,:]  = W[s,h] x[s,h,:]            (W[s,h] replaced by W0[h] first if reset[s])
 *   W[s,h]   <- W0[h] + alpha[s,h] (W[s,h] - W0[h]) - eta[s,h] g[s,h,:] x[s,h,:]^T
 *   W0     [H, d_out, d_in] fp32 slow weights
 *   alpha  [S, H] fp32 or NULL (then alpha_scalar)
 *   reset  [S] uint8 or NULL: 1 = this step starts a new document
 * Other arguments and supported sizes as in gradlev_decode_step. */
int gradlev_decode_step_gated(int64_t S, int64_t H, int64_t d_in, int64_t d_out,
                              float* W, const float* W0, const float* x,
                              const float* g, const float* eta, float eta_scalar,
                              const float* alpha, float alpha_scalar,
                              const uint8_t* reset, float* y, void* stream);

/* ------------------------------------------------------------------------
 * Two-map online MLP (Appendix A)
 * ------------------------------------------------------------------------
 *   z_t = W1_t x_t,   h_t = sigma(z_t),   y_t = W2_t h_t,
 * both maps written with centered decay, the shared retention alpha_t and the
 * shared write strength mu_t divided by each map's input width:
 *   eta_1 = mu_t / d_in,   eta_2 = mu_t / hidden.
 * Given costate proposals g_z (for W1) and g_y (for W2) the forward is two
 * gated exclusive scans in layer order, and the reverse target of the hidden
 * layer is sigma'(z_hat) times the transpose read of the second scan,
 *   g_z~ = sigma'(z_hat_t) (W2_0 + Delta2_t)^T g_y~,
 * optionally continued to the input: g_x~ = (W1_0 + Delta1_t)^T g_z~. */
/* GRADLEV_ACT_GELU_TANH is the tanh-approximate GELU,
 *   z/2 (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3))),
 * which the paper's backbone uses (Appendix E, "Model and prefiller"). */
enum { GRADLEV_ACT_TANH = 0, GRADLEV_ACT_GELU = 1 /* z Phi(z), erf form */, GRADLEV_ACT_GELU_TANH = 2 };

/* d_in, hidden, d_out in {64, 128}; in_dtype is the storage of X, Gz, Gy,
 * the hidden activations between the scans and gY; segment as in
 * gradlev_shape; act a GRADLEV_ACT_* value. */
typedef struct gradlev_mlp_shape {
  int64_t B, H, T, d_in, hidden, d_out;
  int64_t segment;
  int32_t in_dtype;
  int32_t act;
} gradlev_mlp_shape;

/* Workspace for gradlev_mlp_fwd and gradlev_mlp_reverse (same rules as
 * gradlev_scan_workspace_bytes). */
int gradlev_mlp_workspace_bytes(const gradlev_mlp_shape* s, size_t* bytes);

/* Forward.
 *   W1_0 [H, hidden, d_in], W2_0 [H, d_out, hidden] fp32 slow weights
 *   X [B,H,T,d_in], Gz [B,H,T,hidden], Gy [B,H,T,d_out]   in_dtype
 *   mu [B,H,T] fp32 or NULL (then mu_scalar)
 *   Z   [B,H,T,hidden] fp32 out: z_hat
 *   Hid [B,H,T,hidden] in_dtype out: h_hat = sigma(z_hat) as stored for the second scan
 *   Y   [B,H,T,d_out]  fp32 out: y_hat */
int gradlev_mlp_fwd(const gradlev_mlp_shape* s, const gradlev_gates* gates,
                    const float* W1_0, const float* W2_0, const void* X,
                    const void* Gz, const void* Gy, const float* mu, float mu_scalar,
                    float* Z, void* Hid, float* Y, void* workspace,
                    size_t workspace_bytes, void* stream);

/* Reverse targets, from the forward's Z and Hid and the output costate
 *   gY [B,H,T,d_out] in_dtype.
 *   gZ [B,H,T,hidden] fp32 out: g_z~
 *   gX [B,H,T,d_in]   fp32 out or NULL: g_x~ (the hidden target is stored in
 *                     in_dtype before it queries the first scan)
 * Training gradients of L = sum_t <gY_t, y_t> with the writes detached, as
 * the paper trains (Appendix E: costates and write inputs detached; gate and
 * read derivatives remain), each fp32 out or NULL:
 *   dMu   [B,H,T]          dL/dmu_t = deta_1 / d_in + deta_2 / hidden, where
 *                          deta_k is map k's write-strength gradient for its
 *                          own upstream costate (gY for the second map, the
 *                          hidden target g_z~ for the first); for a scalar mu
 *                          its gradient is the sum over tokens
 *   dAlpha [B,H,T]         dL/dalpha_t, the two maps' retention gradients added
 *   dW1_0 [H,hidden,d_in]  sum_b sum_t g_z~ x^T (overwritten)
 *   dW2_0 [H,d_out,hidden] sum_b sum_t gY h^T (overwritten)
 * The first map's outputs use the in_dtype copy of g_z~, as gX does. */
int gradlev_mlp_reverse(const gradlev_mlp_shape* s, const gradlev_gates* gates,
                        const float* W1_0, const float* W2_0, const void* X,
                        const void* Gz, const void* Gy, const float* mu, float mu_scalar,
                        const float* Z, const void* Hid, const void* gY, float* gZ,
                        float* gX, float* dMu, float* dAlpha, float* dW1_0, float* dW2_0,
                        void* workspace, size_t workspace_bytes, void* stream);

/* Kernel timing for benchmarks and tracing.  While a family's bit is set in
 * the mask given to gradlev_timing_enable (bit f = family f; 0 turns timing
 * off), every launch of that family is bracketed by HIP events recorded on the
 * caller's stream (events are created by the library on first use and reused;
 * no device memory is allocated).  Recording works under stream capture: the
 * events become nodes of the captured graph and are read after it has run.
 * gradlev_timing_read waits for the recorded events and returns, for one
 * family, the summed duration in milliseconds and the number of launches
 * since the last reset.  Not thread-safe: use from one host thread.  At most
 * 65536 launches per family are kept between reads: past that, an eager
 * launch first waits for the recorded events and folds them into the sum,
 * while a launch under stream capture (whose events have not run yet) is
 * simply not timed.
 * Families: */
enum {
  GRADLEV_K_FWD_AGG = 0,   /* per-segment write aggregates (forward)      */
  GRADLEV_K_FWD_MAIN = 1,  /* chunked forward scan                         */
  GRADLEV_K_BWD_AGG = 2,   /* per-segment aggregates (backward)           */
  GRADLEV_K_BWD_MAIN = 3,  /* chunked backward scan                        */
  GRADLEV_K_BWD_DW0 = 4,   /* batch reduction of dW0                       */
  GRADLEV_K_DECODE = 5,    /* deployment step                              */
  GRADLEV_K_GATED_AGG = 6, /* gated scans: per-segment aggregates          */
  GRADLEV_K_GATED_FWD = 7, /* gated forward scan                           */
  GRADLEV_K_GATED_STATES = 8, /* gated backward: chunk-start states        */
  GRADLEV_K_GATED_BWD = 9, /* gated backward scan                          */
  GRADLEV_K_WIDE_SCORE = 10, /* wide maps: gates and causal score tiles   */
  GRADLEV_K_WIDE_OUT = 11,   /* wide maps: W_0 term plus score-weighted sum */
  GRADLEV_K_COUNT = 12
};
int gradlev_timing_enable(int mask); /* returns the previous mask */
int gradlev_timing_reset(void);
int gradlev_timing_read(int family, double* ms, int64_t* launches);

/* Static, human-readable text for a status code. */
const char* gradlev_error_string(int code);

/* Library version as MAJOR*10000 + MINOR*100 + PATCH. */
int gradlev_version(void);

#ifdef __cplusplus
}
#endif

#endif /* GRADLEV_H */
