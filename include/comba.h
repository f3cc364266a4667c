/*
 * comba.h -- C ABI of the MI355X (gfx950) chunk-wise Comba operator.
 *
 * Comba (arXiv 2506.02475) is a bilinear RNN whose per-head state S_t (dv x dk)
 * follows, for tokens t = 1..T of one sequence (Eq. comba-S, Section 3):
 *
 *     S_t = S_{t-1} (alpha_t I - beta~_t k_t k_t^T) + beta_t v_t k_t^T
 *     o_t = S_t (q_t - d k_t)
 *
 * with forget gate alpha_t = exp(g_t) in (0, 1], input gate beta_t, state
 * feedback strength beta~_t, and a per-head output-feedback scalar d.  beta~ is
 * an optional per-token input (Section 3.2 forms it as b * beta with a learned
 * b in (0, 1); Comba-iplr, alpha (I - 2 beta~ k k^T), is the same recurrence
 * with beta~' = 2 alpha beta~, Section 3 SPLR/IPLR); when it is omitted
 * (NULL) it is tied to beta, the paper's ablation without the factor b
 * (Section 4).  The library evaluates this recurrence with the chunk-wise
 * parallel algorithm of Section 3.3 (chunks of 64 tokens, WY/UT transform with
 * one unit-lower-triangular inverse per chunk, inter-chunk state passing), and
 * its reverse-mode derivative (derived from the same chunk form; the paper
 * states no backward).
 *
 * Conventions shared by every entry point
 *  - `shape` (and shape->cu_seqlens_host) points to host memory; every other
 *    pointer (including shape->cu_seqlens) is a DEVICE pointer on the current
 *    HIP device.  The caller owns every buffer; the library allocates no
 *    device memory and keeps no data between calls.  It keeps one helper
 *    stream (default priority) and two events per device, created on the
 *    first comba_chunk_bwd call that uses them: the stateless backward runs
 *    its two independent scans side by side, the second on the helper stream,
 *    forked from and joined back to `stream` (under graph capture of `stream`
 *    the helper joins the capture; a first call that is itself captured
 *    creates nothing and runs the two scans in turn).
 *  - Layouts are C-contiguous.  Token-major tensors are [B, T, H, D]; in the
 *    variable-length mode B == 1, T is the packed token count and sequence s
 *    covers tokens [cu_seqlens[s], cu_seqlens[s+1]).  A sequence's last chunk
 *    may be partial; states never cross sequences.
 *  - The recurrent state is stored transposed, H = S^T, as [N, H, dk, dv] fp32
 *    (N = number of sequences), the orientation of the paper's recurrent
 *    pseudocode (Appendix B.1).
 *  - q, k, v, beta, beta_tilde and dO have dtype shape->in_dtype (bf16 or
 *    fp32); g (log alpha), d, states and every output are fp32.
 *  - Head sizes: dk, dv in {64, 128}; with bf16 inputs also dk, dv in {128, 256}
 *    (256, the paper's models, for every chunk entry point).  fp32 inputs: 64.
 *  - beta_tilde [B,T,H] may be NULL: beta~ = beta.  The backward's dbeta_tilde
 *    [B,T,H] fp32 may be NULL only when beta_tilde is: dbeta then holds the
 *    total derivative through both roles of beta.  When dbeta_tilde is given,
 *    dbeta holds the derivative through the write strength only and
 *    dbeta_tilde that through the feedback strength (the per-head b of Section
 *    3.2 then gets db_h = sum over tokens of beta * dbeta_tilde).
 *  - g must be <= 0 (alpha in (0, 1]); other values are outside the contract
 *    (results may overflow) but never cause out-of-bounds accesses.
 *  - Calls are asynchronous on `stream` (a hipStream_t passed as void*; NULL is
 *    the default stream).  Argument errors are detected before any launch and
 *    then nothing is written.  A failed launch returns COMBA_ERR_HIP.
 *  - Alignment: q, k, v, dO and every fp32 tensor whose last dimension is dk
 *    or dv (h0, ht, o, dht, dh0, dq, dk, dv) need 16 bytes, the workspace 256
 *    bytes, the other fp32 tensors 4 bytes and beta, beta_tilde their element
 *    size; any other pointer is rejected with COMBA_ERR_ALIGN.
 *  - Outputs must not alias inputs (the one exception: ht == h0 in
 *    comba_recurrent_fwd); outputs are overwritten, never accumulated.
 *  - A call without tokens (T == 0 or B == 0) is valid: the per-token tensors
 *    (q, k, v, g, beta, o, dO, dq, dk, dv, dg, dbeta, dbeta_tilde) may then be
 *    NULL, and the states pass through (ht = h0, dh0 = dht, dd = 0).  Empty
 *    sequences inside a packed batch behave the same way for their own states.
 *  - Variable-length offsets: when shape->cu_seqlens_host (a HOST copy of the
 *    same N + 1 offsets) is given, every entry point checks
 *    0 = cu[0] <= cu[1] <= ... <= cu[N] = T on it and returns COMBA_ERR_SHAPE
 *    before any launch when it fails.  Without the host copy the device
 *    offsets are trusted: malformed ones are clamped into [0, T] on the device
 *    (never an out-of-bounds access), and the outputs are then undefined.
 *  - Non-finite inputs propagate: a NaN or Inf in q, k, v, dO (or the
 *    states) makes the affected outputs and gradients of its sequence and
 *    head non-finite; other sequences and heads are unaffected (dd sums over
 *    all sequences of a head and so takes it up too).
 *  - Few long rows (rows whose state scans would have fewer chains, N H dv /
 *    32, than half the device's CUs; packed batches only with
 *    cu_seqlens_host): the bf16 chunk entry points cut every row into P
 *    segments scanned side by side (the state
 *    recurrence is affine in the state entering a segment; Section 3.3's
 *    chunk form, applied between segments).  P is chosen from the shape and
 *    the device; the environment variable COMBA_SCAN_SEGMENTS, read at every
 *    call, overrides it: 1 never, P in 2..64 P segments (fixed-length rows:
 *    when P divides the row's chunks, else none), unset or 0 the automatic
 *    choice.  The workspace sizes include the segments' buffers; a smaller
 *    workspace that still holds the plain layout runs the plain scans.  The
 *    result equals the plain scans' up to rounding.  A saved pair
 *    (comba_chunk_fwd_save, comba_chunk_bwd_saved) must see the same
 *    COMBA_SCAN_SEGMENTS and workspace size in both calls.
 *  - Calls on different streams with distinct workspaces may run concurrently;
 *    a workspace must not be shared by calls that overlap in time.
 */
#ifndef COMBA_H
#define COMBA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  COMBA_OK = 0,
  COMBA_ERR_NULL = 1,      /* a required pointer is NULL                         */
  COMBA_ERR_SHAPE = 2,     /* unsupported or inconsistent sizes                  */
  COMBA_ERR_DTYPE = 3,     /* unknown dtype                                      */
  COMBA_ERR_ALIGN = 4,     /* a pointer breaks the alignment rules above         */
  COMBA_ERR_WORKSPACE = 5, /* workspace smaller than the *_workspace_bytes value */
  COMBA_ERR_HIP = 6,       /* a kernel launch failed                             */
  COMBA_ERR_SCRATCH = 7    /* too large for the static scratch of the no-allocation
                              entry point (comba_noalloc_scratch_bytes)           */
} comba_status;

typedef enum { COMBA_F32 = 0, COMBA_BF16 = 1 } comba_dtype;

typedef struct {
  int32_t B;                  /* batch rows (1 in variable-length mode)                 */
  int32_t T;                  /* tokens per row; packed total in variable-length mode   */
  int32_t H;                  /* heads                                                  */
  int32_t dk;                 /* key/query head dim: 64, 128, 256 (see above)           */
  int32_t dv;                 /* value head dim: 64, 128, 256 (see above)               */
  int32_t chunk;              /* chunk length; must be 64                               */
  int32_t num_seqs;           /* N: sequences; must equal B when cu_seqlens == NULL     */
  const int32_t *cu_seqlens;  /* device [N+1] offsets (0 = cu[0] <= ... <= cu[N] = T),
                                 or NULL for fixed-length rows                           */
  const int32_t *cu_seqlens_host; /* optional HOST copy of the same offsets, or NULL:
                                 when given, checked before any launch (COMBA_ERR_SHAPE
                                 on a malformed table; requires cu_seqlens)              */
  comba_dtype in_dtype;       /* dtype of q, k, v, beta, beta_tilde, dO                 */
} comba_shape;

/* Workspace sizes in bytes for one call of the matching entry point. */
size_t comba_fwd_workspace_bytes(const comba_shape *shape);
size_t comba_bwd_workspace_bytes(const comba_shape *shape);

/*
 * Forward of the chunk-wise recurrence (Section 3.3: UT transform with one
 * inverse M per chunk, Eq. prepare-WY_M; inter-chunk state update and output of
 * the closing matrix form).
 *   q, k  [B,T,H,dk] in_dtype      v   [B,T,H,dv] in_dtype
 *   g     [B,T,H] fp32 (log alpha) beta [B,T,H] in_dtype    d [H] fp32
 *   beta_tilde [B,T,H] in_dtype feedback strength, or NULL (tied to beta)
 *   h0    [N,H,dk,dv] fp32 initial states, or NULL for zero states
 *   o     [B,T,H,dv] fp32 output   ht  [N,H,dk,dv] fp32 final states, or NULL
 *   ws    device workspace of at least comba_fwd_workspace_bytes(shape), 256-B aligned
 */
comba_status comba_chunk_fwd(const comba_shape *shape, const void *q, const void *k,
                             const void *v, const float *g, const void *beta,
                             const void *beta_tilde, const float *d, const float *h0, float *o,
                             float *ht, void *ws, size_t ws_bytes, void *stream);

/*
 * Backward: gradients of L = <dO, o> + <dht, ht> with respect to every input.
 * Recomputes the forward internally (no saved state is needed from a forward
 * call); the recomputed chunk states and the reverse state-gradient scan do
 * not depend on each other and run side by side (see the conventions).
 * Inputs as comba_chunk_fwd plus
 *   dO    [B,T,H,dv] in_dtype     dht [N,H,dk,dv] fp32 or NULL (zero)
 * Outputs (fp32): dq, dk [B,T,H,dk]; dv [B,T,H,dv]; dg, dbeta [B,T,H];
 *   dbeta_tilde [B,T,H] (see the conventions: NULL only with beta_tilde NULL);
 *   dd [H] (summed over all sequences and tokens); dh0 [N,H,dk,dv] or NULL.
 */
comba_status comba_chunk_bwd(const comba_shape *shape, const void *q, const void *k,
                             const void *v, const float *g, const void *beta,
                             const void *beta_tilde, const float *d, const float *h0,
                             const void *dO, const float *dht, float *dq, float *dk, float *dv,
                             float *dg, float *dbeta, float *dbeta_tilde, float *dd, float *dh0,
                             void *ws, size_t ws_bytes, void *stream);

/*
 * Training pair.  comba_chunk_fwd_save computes exactly what comba_chunk_fwd
 * computes and, in addition, leaves in `ws` everything the backward would
 * otherwise recompute (chunk tables, the per-chunk UT-transform operands and
 * the chunk-boundary states); `ws` must hold comba_bwd_workspace_bytes(shape).
 * comba_chunk_bwd_saved then returns the same gradients as comba_chunk_bwd
 * while skipping that recomputation.  The caller must pass the same shape and
 * inputs (q, k, v, g, beta, beta_tilde, d, h0) and the same, unmodified `ws` to both calls,
 * with the backward ordered after the forward (same stream, or synchronised);
 * otherwise the results are undefined (never out of bounds).
 */
comba_status comba_chunk_fwd_save(const comba_shape *shape, const void *q, const void *k,
                                  const void *v, const float *g, const void *beta,
                                  const void *beta_tilde, const float *d, const float *h0,
                                  float *o, float *ht, void *ws, size_t ws_bytes, void *stream);
comba_status comba_chunk_bwd_saved(const comba_shape *shape, const void *q, const void *k,
                                   const void *v, const float *g, const void *beta,
                                   const void *beta_tilde, const float *d, const float *h0,
                                   const void *dO, const float *dht, float *dq, float *dk,
                                   float *dv, float *dg, float *dbeta, float *dbeta_tilde,
                                   float *dd, float *dh0, void *ws, size_t ws_bytes,
                                   void *stream);

/*
 * Forward without any device allocation, for callers that cannot allocate:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Computes what comba_chunk_fwd computes with the same kernels
 * (bitwise-equal results; the one exception: few long rows whose segmented
 * scans, see the conventions, need more than the array holds run the plain
 * scans here, equal up to rounding), with its workspace in a static device array of
 * comba_noalloc_scratch_bytes() bytes (80 MiB) that every device the library
 * runs on holds until the process ends; the caller passes only inputs and
 * outputs.  A shape whose comba_fwd_workspace_bytes exceeds it (more than about
 * 4,900 chunk-heads, e.g. beyond the 1.3B layer's B4 T4096 H16 at d = 128) is
 * rejected with COMBA_ERR_SCRATCH before any launch; invalid shapes with
 * COMBA_ERR_SHAPE.  Calls that overlap in time on one device share the array
 * and race: order them on one stream.  Nothing in it needs clearing between
 * calls (each call writes every byte it reads).
 */
size_t comba_noalloc_scratch_bytes(void);
comba_status comba_chunk_fwd_noalloc(const comba_shape *shape, const void *q, const void *k,
                                     const void *v, const float *g, const void *beta,
                                     const void *beta_tilde, const float *d, const float *h0,
                                     float *o, float *ht, void *stream);

/*
 * Token-by-token recurrence (Eq. comba-S evaluated one token at a time: the
 * constant-memory inference form of Section 3), for decoding and short
 * segments.  Per sequence, head and token, with H = S^T:
 *     u_t = beta_t v_t - beta~_t H_{t-1}^T k_t,  H_t = alpha_t H_{t-1} + k_t u_t^T,
 *     o_t = H_t^T (q_t - d k_t).
 * Arguments and layouts are those of comba_chunk_fwd (same shape struct; its
 * `chunk` field is not used, and fp32 inputs also allow dk, dv = 128), without
 * a workspace: the call needs no device memory of its own.  h0 may be NULL
 * (zero states) and ht NULL (states not returned); ht may be the same buffer
 * as h0, which updates the states in place (the usual decoding step, T = 1);
 * any other overlap of ht with an input is undefined.  The work per token is a
 * dependent chain, so long sequences belong to comba_chunk_fwd; results agree
 * with it to rounding.
 */
comba_status comba_recurrent_fwd(const comba_shape *shape, const void *q, const void *k,
                                 const void *v, const float *g, const void *beta,
                                 const void *beta_tilde, const float *d, const float *h0,
                                 float *o, float *ht, void *stream);

/*
 * Layer input prologue (Section 3.4, Neural Architecture): turns the projected
 * pre-activations xq, xk [B,T,H,dk] and xv [B,T,H,dv] (in_dtype) into the
 * operator's q, k, v (in_dtype, same layouts):
 *     u_t = sum_{j<4} w[h][c][j] x_{t-3+j}[c]   (causal depthwise conv, zero before
 *                                               each sequence start)
 *     s_t = SiLU(u_t);  q, k: y_t = s_t / sqrt(|s_t|^2 + 1e-6) over the head's
 *     channels;  v: y_t = s_t.
 * Taps wq, wk [H][dk][4] and wv [H][dv][4] fp32; the newest token takes tap 3.
 * Shape rules of comba_recurrent_fwd (chunk not used; dk, dv in {64, 128, 256},
 * 64 not paired with 256).  The forward needs no workspace.  bf16 outputs are
 * rounded to nearest even.
 */
comba_status comba_prologue_fwd(const comba_shape *shape, const void *xq, const void *xk,
                                const void *xv, const float *wq, const float *wk, const float *wv,
                                void *q, void *k, void *v, void *stream);

/*
 * Backward of the prologue: given gq, gk, gv (fp32 gradients of q, k, v, same
 * layouts), writes dxq, dxk, dxv (fp32, layouts of x) and dwq, dwk, dwv (fp32,
 * layouts of w; summed over every token of every sequence in a fixed order).
 * Recomputes the forward.  ws: device workspace of at least
 * comba_prologue_workspace_bytes(shape) bytes, 256-byte aligned.
 */
size_t comba_prologue_workspace_bytes(const comba_shape *shape);
comba_status comba_prologue_bwd(const comba_shape *shape, const void *xq, const void *xk,
                                const void *xv, const float *wq, const float *wk, const float *wv,
                                const float *gq, const float *gk, const float *gv, float *dxq,
                                float *dxk, float *dxv, float *dwq, float *dwk, float *dwv,
                                void *ws, size_t ws_bytes, void *stream);

/*
 * Output gate of the layer (Section 3.4, sigmoid gating), applied to the
 * operator's output before the output projection: y = o * sigmoid(z), with o
 * [B,T,H,dv] fp32 (as comba_chunk_fwd writes it), the gate pre-activation z and
 * y [B,T,H,dv] in_dtype (bf16 y rounded to nearest even).  Backward from dy
 * (fp32): do = dy sigmoid(z), dz = dy o sigmoid(z) (1 - sigmoid(z)), both
 * fp32.  Shape rules of comba_recurrent_fwd (dk is checked but not used).  All
 * pointers 16-byte aligned; no workspace.
 */
comba_status comba_gate_fwd(const comba_shape *shape, const float *o, const void *z, void *y,
                            void *stream);
comba_status comba_gate_bwd(const comba_shape *shape, const float *o, const void *z,
                            const float *dy, float *dout, float *dz, void *stream);

/*
 * Stage timing, for benchmarks (not part of the method).  comba_profile_enable(1)
 * starts a recording session on the calling host thread: every following
 * comba_chunk_fwd / comba_chunk_bwd call on this thread records a HIP event on
 * its stream before each kernel stage and after its last stage (at most 4096
 * events per session; calls beyond that are not recorded).  Events are created
 * on first use on the current device and reused until the process ends.
 * comba_profile_read waits for the last recorded event and writes, in call
 * order, up to `capacity` stage durations in milliseconds (`ms`) and static
 * stage names (`names`; either may be NULL).  It returns the number written,
 * or -1 on a HIP error.  comba_profile_enable(0) stops recording (the default).
 */
comba_status comba_profile_enable(int enable);
int comba_profile_read(float *ms, const char **names, int capacity);

/*
 * Stage selection for the timing above (benchmarks only).  With a stage name
 * (for example "intra_bwd"; the name is copied), the calling thread's
 * recording sessions record only two events per call: one before that stage
 * and one right after it, so comba_profile_read returns that stage's
 * durations alone and the other stages run without event records between
 * them.  NULL (the default) records every stage.  The selection holds until
 * the next call of this function on the thread.  Always returns COMBA_OK.
 */
comba_status comba_profile_select(const char *stage);

/* Human-readable name of a status code (static storage). */
const char *comba_status_string(comba_status status);

#ifdef __cplusplus
}
#endif

#endif /* COMBA_H */
