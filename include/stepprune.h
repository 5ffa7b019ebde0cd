/*
 * stepprune.h -- C ABI of the StepPrune inference-time selection library for
 * AMD MI355X (gfx950).
 *
 * The library runs the three stages of the paper's inference procedure
 * (Algorithm 1):
 *   stepprune_project  step 1: project visual tokens, START/STOP embeddings and
 *                      the text context once (Section "Conditional Sequential
 *                      Pointer Policy": text projection, LayerNorm, gain g_text;
 *                      the pointer decoder's key/query/value projections);
 *   stepprune_select   steps 2-4: the sequential pointer policy with STOP (Eq. 2,
 *                      Eq. 4), every group of every image run as an independent
 *                      episode, kept indices restored to native order;
 *   stepprune_compact  step 5: physical gather of the kept tokens ahead of the
 *                      prompt into a padded or packed prefill buffer.
 * Beside them: stepprune_encode, the cross-modal input encoder of Eq. 3 that
 * turns X into the candidate tokens H ahead of step 1; and, for the training
 * pathway (Section "Trajectory-Aware Differentiable Optimization"),
 * stepprune_select_trajectory (the trajectory sums of Eqs. 5-7) and
 * stepprune_gate_denoise (the noise gate of Eq. 9 and the locally masked
 * denoiser).
 *
 * Conventions shared by every call
 *  - Pointers are DEVICE pointers unless marked (host).  All row-major.
 *  - Rows of visual tokens of all images are packed back to back; image b owns
 *    rows [img_off[b], img_off[b+1]).  Indices in the outputs are image-local.
 *  - Every call validates its host-side arguments first and returns a status
 *    before launching anything.  On SP_OK the work is enqueued on `stream` and
 *    the call returns; outputs are valid once the stream has been synchronised.
 *  - The library allocates no memory and keeps no state besides kernel handles
 *    and the fixed device scratch of stepprune_select_noalloc.  The caller owns
 *    every buffer, including the workspace `ws` whose size
 *    stepprune_workspace_bytes() gives; a workspace may be reused by later calls
 *    on the same stream.
 *  - Errors that depend on device-resident data (inconsistent offsets, a group
 *    larger than the stated maximum, counts that do not fit the output) are
 *    recorded in a device error word, the first 4 bytes of `ws`; the affected
 *    outputs are then undefined.  The word keeps the first error recorded
 *    until stepprune_read_device_error() reads and clears it, so it covers
 *    every call made with that workspace since the last read.  A new
 *    workspace must be zero-filled (its first 256 bytes at least) before its
 *    first use.
 *  - No C++ exception crosses this interface.
 *  - `events` (host) is NULL or points to caller-created hipEvent_t handles that
 *    the call records on `stream` around its main kernels, for timing:
 *      project: [0] before, [1] after the projection GEMM;
 *      select:  [0] before, [1] after the Gram products, [2] before, [3] after
 *               the pointer recurrence;
 *      compact: [0] before, [1] after the gather.
 *    A NULL entry is skipped.  The library neither creates nor destroys events.
 *
 * Numerics: projections accumulate in float32 and are stored once, rounded to
 * nearest-even, in the dtype of sp_dims (bfloat16 or float32); the text context
 * and all selection arithmetic are float32.  sigma = h^(-1/2) is applied to the
 * history-attention scores and to the pointer logits; the STOP bias b_stop is
 * added to the STOP logit unscaled.  Exact ties go to the lowest token index and
 * STOP loses ties against tokens (it is last in the candidate memory).
 */
#ifndef STEPPRUNE_H
#define STEPPRUNE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SP_OK = 0,
  SP_EINVAL = 1,        /* a host-side argument is invalid (null, size, alignment) */
  SP_EUNSUPPORTED = 2,  /* valid but not supported by this library (dtype, g > 5, sizes) */
  SP_EWORKSPACE = 3,    /* ws_bytes smaller than stepprune_workspace_bytes() */
  SP_EHIP = 4,          /* a HIP launch or runtime call failed */
  SP_EDEVICE = 5        /* the device error word is set (read_device_error) */
} sp_status;

typedef enum { SP_F32 = 0, SP_BF16 = 1 } sp_dtype;

enum {
  SP_TRACE = 1u,       /* stepprune_select writes the per-step trace */
  SP_NO_HISTORY = 2u,  /* pointer query frozen at its first value (diagnostic:
                          the selector collapses to top-K of the first scores, Eq. 1) */
  SP_FULL_ROLLOUT = 4u,/* the rollout that the trajectory sums of Eqs. 5-7 run over:
                          STOP is scored but not taken while a token is left, so
                          every episode runs to its cap (or out of tokens) */
  /* The two phases of stepprune_select, for callers that overlap batches:
     SP_GRAM_ONLY computes the per-group Gram products (the matrix-core part)
     into the workspace and returns; a later call with SP_REUSE_GRAM and the
     same arguments and workspace runs the recurrence on them.  Between the
     two, KQV, ctx, the offsets and the workspace must not change. */
  SP_GRAM_ONLY = 8u,
  SP_REUSE_GRAM = 16u,
  /* Diagnostic, with SP_TRACE: every trace record is followed by the step's
     whole logit vector (see stepprune_select's `trace`). */
  SP_LOGITS = 32u
};

enum { SP_LAYOUT_PADDED = 0, SP_LAYOUT_PACKED = 1 };

/* Device error word values (stepprune_read_device_error). */
enum {
  SP_DEV_OK = 0,
  SP_DEV_BAD_OFFSETS = 1,   /* an offset array is not non-decreasing or exceeds its total */
  SP_DEV_GROUP_TOO_LARGE = 2,/* a group has more tokens than max_group */
  SP_DEV_BAD_CAP = 3,       /* a group cap is negative or exceeds max_cap */
  SP_DEV_OUTPUT_OVERFLOW = 4 /* kept or prefill rows exceed the capacity given */
};

/* Shapes shared by the calls (host). d, d_text and h are multiples of 64,
   h <= 1024 (h <= 512 for SP_F32).  dtype applies to X, E_text, s_start,
   s_stop, W_kqv, W_text, KQV and the compaction output. */
typedef struct {
  int32_t d;        /* visual feature width */
  int32_t d_text;   /* text embedding width */
  int32_t h;        /* selector hidden width */
  int32_t dtype;    /* sp_dtype */
} sp_dims;

/*
 * Algorithm 1 step 1.  Projects every visual row and the START and STOP
 * embeddings with one weight matrix, and pools the text context per image.
 *
 *  X        [T_vis, d]        visual tokens of all images, packed
 *  s_start  [d], s_stop [d]   learned START / STOP embeddings
 *  W_kqv    [3h, d]           output-major: rows [0,h) key, [h,2h) query,
 *                             [2h,3h) value features (x -> x W_kqv^T)
 *  E_text   [T_txt, d_text]   text embeddings of all images, packed by
 *  text_off [B+1]             text_off (device); T_txt = text_off[B] (host copy)
 *  W_text   [h, d_text]       text projection into the pointer query space
 *  g_text, ln_eps             c_b = g_text * mean_l LN(E_{b,l} W_text^T),
 *                             LayerNorm without affine, biased variance;
 *                             an image without text gets c_b = 0
 *  KQV      out [T_vis+2, 3h] row T_vis = START, row T_vis+1 = STOP
 *  ctx      out [B, h] float32
 *  ws       workspace of stepprune_workspace_bytes(0, ...)
 */
sp_status stepprune_project(const sp_dims* dims,
                            const void* X, int64_t T_vis,
                            const void* s_start, const void* s_stop,
                            const void* W_kqv,
                            const void* E_text, const int32_t* text_off,
                            int32_t B, int64_t T_txt,
                            const void* W_text, float g_text, float ln_eps,
                            void* KQV, float* ctx,
                            void* ws, size_t ws_bytes,
                            const hipEvent_t* events, hipStream_t stream);

/*
 * Algorithm 1 steps 2-4 (Eq. 2, Eq. 4; Eq. 11 for g > 1).  Every group (a
 * contiguous run of one image's visual rows) is an independent episode:
 * history [START], then per round t = 1..cap the pointer query
 *     u_t = c_b + q_e + sum_tau softmax_tau(sigma <q_e, k_tau>) v_tau
 * (e the newest history entry, tau over the history), logits
 * l_t(j) = sigma <u_t, k_j> over the group's unselected tokens and
 * l_t(STOP) = sigma <u_t, k_stop> + b_stop; the first maximal candidate is
 * taken; STOP ends the episode; a token is masked and appended to the history.
 * At the cap the episode ends without a STOP step.
 *
 * With g > 1 tokens per round (Section "Grouped Execution for High-Resolution
 * Inputs", Eq. 11) a round ends the episode only when STOP is strictly above
 * every unselected token; otherwise it takes the min(g, unselected) tokens of
 * largest logit (equal logits: lower index first), appends them to the
 * history in descending-logit order, and the next query q_e is the mean of
 * their q rows.  The cap counts rounds, so a group keeps at most min(cap g, n).
 *
 *  KQV, ctx       outputs of stepprune_project (T_vis visual rows + START + STOP)
 *  img_off [B+1]  visual row offsets per image
 *  grp_off [G+1]  visual row offsets per group; groups of an image are
 *                 contiguous and in row order, grp_img [G] their image,
 *                 grp_cap [G] their round cap (>= 0)
 *  max_group      (host) upper bound on any group's size, <= 1022
 *  max_cap        (host) upper bound on any group's kept capacity
 *                 min(cap g, n); a group above it is a device error
 *  kept_off [B+1] offsets of each image's slice of kept_idx; the slice must
 *                 hold sum over its groups of min(cap g, n)
 *  b_stop         additive STOP bias (may be +-inf)
 *  g              tokens kept per non-STOP round, 1 <= g <= 5
 *                 (SP_EUNSUPPORTED above 5)
 *  flags          SP_TRACE (with SP_LOGITS), SP_NO_HISTORY, SP_FULL_ROLLOUT, SP_GRAM_ONLY or
 *                 SP_REUSE_GRAM (not both; SP_GRAM_ONLY writes none of the
 *                 outputs and is refused by stepprune_select_trajectory)
 *  kept_idx  out  image-local kept indices, ascending per image, at kept_off[b]
 *  kept_cnt  out  [B] kept count per image (0 for an image whose slice of
 *                 kept_idx overflows, with SP_DEV_OUTPUT_OVERFLOW)
 *  grp_cnt   out  [G] kept count per group, or NULL
 *  trace     out  with SP_TRACE, NULL otherwise.  g = 1: [G, trace_steps, 4]
 *                 float32 records per step: {taken candidate (int32 bits;
 *                 -1 = STOP), its logit, the runner-up candidate logit (-inf
 *                 if none), STOP logit}.  g > 1: [G, trace_steps, g + 3] per
 *                 round: {g slots of taken tokens in appended order (int32
 *                 bits; slot 0 = -1 for STOP, unused slots -3), the smallest
 *                 taken logit (the STOP logit for STOP), the largest logit
 *                 left out (STOP included when not taken; -inf if none), STOP
 *                 logit}.  Either way records past the end hold -2 in slot 0.
 *                 With SP_LOGITS (which needs SP_TRACE) each record is
 *                 followed by max_group + 1 float32: the step's (round's)
 *                 logit of every token slot 0..max_group-1 (-inf for tokens
 *                 already selected and for slots past the group), then the
 *                 STOP logit; records are then 4 + max_group + 1 (g = 1) or
 *                 g + 3 + max_group + 1 floats wide (-inf past the end).
 */
sp_status stepprune_select(const sp_dims* dims,
                           const void* KQV, const float* ctx, int64_t T_vis,
                           const int32_t* img_off, int32_t B,
                           const int32_t* grp_off, const int32_t* grp_img,
                           const int32_t* grp_cap, int32_t G,
                           int32_t max_group, int32_t max_cap,
                           const int32_t* kept_off,
                           float b_stop, int32_t g, uint32_t flags,
                           int32_t* kept_idx, int32_t* kept_cnt, int32_t* grp_cnt,
                           float* trace, int32_t trace_steps,
                           void* ws, size_t ws_bytes,
                           const hipEvent_t* events, hipStream_t stream);

/*
 * stepprune_select for callers that cannot allocate device memory (code under
 * HIP graph capture, serving loops or harnesses that forbid allocation): the
 * same selection, decisions and outputs, with no caller workspace.  The
 * scratch (the Gram blocks, the context split and the group-local kept lists
 * that stepprune_select keeps in `ws`) is a fixed array of
 * STEPPRUNE_NOALLOC_SCRATCH_BYTES in the library's device memory, one copy per
 * GPU, held until the process ends.  The call itself allocates nothing; its
 * first call on a GPU looks up that GPU's copy.
 *
 * Arguments as for stepprune_select, without ws / ws_bytes, plus
 *  err   out  device pointer to a caller-owned, 4-byte-aligned int32 error
 *             word, zero before the first call; it plays the role of the
 *             workspace's error word (the first SP_DEV_* code sticks until
 *             stepprune_read_device_error(err, ...) reads and clears it).
 *  stream     must belong to the current device (SP_EINVAL otherwise).
 * Sizes whose stepprune_workspace_bytes(1, ...) exceeds
 * STEPPRUNE_NOALLOC_SCRATCH_BYTES return SP_EWORKSPACE before any launch
 * (64 MiB holds, for example, 24 groups of 576 tokens at h = 1024).
 * Every call on a GPU uses that GPU's one array, which keeps the last call's
 * contents: calls that overlap on one GPU (different streams, or several
 * host threads) race and must be serialised by the caller.  SP_REUSE_GRAM
 * reads the Gram products that the last SP_GRAM_ONLY call on the GPU left
 * there.
 */
#define STEPPRUNE_NOALLOC_SCRATCH_BYTES (64u << 20)
sp_status stepprune_select_noalloc(const sp_dims* dims,
                                   const void* KQV, const float* ctx, int64_t T_vis,
                                   const int32_t* img_off, int32_t B,
                                   const int32_t* grp_off, const int32_t* grp_img,
                                   const int32_t* grp_cap, int32_t G,
                                   int32_t max_group, int32_t max_cap,
                                   const int32_t* kept_off,
                                   float b_stop, int32_t g, uint32_t flags,
                                   int32_t* kept_idx, int32_t* kept_cnt, int32_t* grp_cnt,
                                   float* trace, int32_t trace_steps,
                                   int32_t* err,
                                   const hipEvent_t* events, hipStream_t stream);

/*
 * Trajectory sums of the training surrogate (Section "Trajectory-Aware
 * Differentiable Optimization"), computed along the pointer trajectory that
 * stepprune_select_trajectory executes (g = 1):
 *     p_t   = softmax(l_t / tau) over the step's candidates (unselected
 *             tokens and STOP; Eq. 4)
 *     A_1 = 1, A_{t+1} = A_t (1 - p_t(STOP))                       (Eq. 5)
 *     s_i   = sum_t A_t p_t(i) beta^t                               (Eq. 6)
 *     K_bar = sum_t A_t (1 - p_t(STOP))                             (Eq. 7)
 * over the executed steps: up to and including the STOP step, or, with
 * SP_FULL_ROLLOUT, every step up to the cap (T_max).  Caller-owned device
 * buffers:
 *  s          out [T_vis] float32, s_i of every token of every group (rows
 *             outside all groups are not written)
 *  kbar       out [G] float32, K_bar per group
 *  pstop      out [G, pstop_steps] float32, p_t(STOP) per step (NaN past
 *             the episode's end), or NULL
 */
typedef struct {
  float tau;            /* pointer temperature, > 0 */
  float beta;           /* discount, 0 < beta <= 1 */
  float* s;
  float* kbar;
  float* pstop;
  int32_t pstop_steps;  /* >= 0; 0 with pstop = NULL */
} sp_trajectory;

/*
 * stepprune_select, and along the same trajectory the sums described with
 * sp_trajectory (Eqs. 5-7).  Arguments as for stepprune_select plus `traj`
 * (host pointer, required).  g must be 1 (SP_EUNSUPPORTED otherwise);
 * tau <= 0, beta outside (0, 1] or a NULL s / kbar give SP_EINVAL.  Runs a
 * selection kernel built with the sums (one exp per candidate and a wave sum
 * per step); it takes the same decisions as stepprune_select.
 */
sp_status stepprune_select_trajectory(const sp_dims* dims,
                                      const void* KQV, const float* ctx, int64_t T_vis,
                                      const int32_t* img_off, int32_t B,
                                      const int32_t* grp_off, const int32_t* grp_img,
                                      const int32_t* grp_cap, int32_t G,
                                      int32_t max_group, int32_t max_cap,
                                      const int32_t* kept_off,
                                      float b_stop, int32_t g, uint32_t flags,
                                      int32_t* kept_idx, int32_t* kept_cnt, int32_t* grp_cnt,
                                      float* trace, int32_t trace_steps,
                                      const sp_trajectory* traj,
                                      void* ws, size_t ws_bytes,
                                      const hipEvent_t* events, hipStream_t stream);

/*
 * Algorithm 1 step 5.  Gathers each image's kept visual rows (ascending) and
 * then its text rows into the prefill buffer.  Requires d_text == d.  X and
 * E_text must be valid device pointers even when the batch holds no visual or
 * no text row (the offsets are device data; nothing is read past them).
 *
 *  layout SP_LAYOUT_PADDED: image b owns out rows [b*rows_per_image,
 *         (b+1)*rows_per_image); rows past K_b + L_b are left untouched;
 *         seq_info [B] = K_b + L_b.
 *  layout SP_LAYOUT_PACKED: sequences back to back; seq_info [B+1] =
 *         cu_seqlens, cu[0] = 0, cu[b+1] = cu[b] + K_b + L_b; rows_per_image
 *         is ignored.
 *  out_rows (host) rows of `out`; writes beyond it set SP_DEV_OUTPUT_OVERFLOW.
 */
sp_status stepprune_compact(const sp_dims* dims,
                            const void* X, const int32_t* img_off,
                            const void* E_text, const int32_t* text_off,
                            const int32_t* kept_idx, const int32_t* kept_off,
                            const int32_t* kept_cnt, int32_t B,
                            int32_t layout, int32_t rows_per_image, int64_t out_rows,
                            void* out, int32_t* seq_info,
                            void* ws, size_t ws_bytes,
                            const hipEvent_t* events, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Training pathway: the variance-preserving noise gate and the locally masked
 * denoiser (Section "Trajectory-Aware Differentiable Optimization": Eq. 9 and
 * the denoiser paragraph).  Per visual token i (row of X):
 *
 *   x~_i = sqrt(a_i) x_i + sqrt(1 - a_i) eps_i
 *   h_i  = x~_i + W_o (W_v LN1(x~_i) + b_v) + b_o
 *   y_i  = h_i + W_2 GELU(W_1 LN2(h_i) + b_1) + b_2
 *
 * The denoiser is one pre-norm transformer block whose self-attention is
 * restricted to the diagonal: each token attends only to itself, so its
 * attention output is the value projection and no information moves between
 * tokens.  LN is LayerNorm over d with scale and shift (eps 1e-6, biased
 * variance); GELU is the exact x Phi(x); the hidden width is 4d.  The gate's
 * weights a_i come from Eq. 8's differentiable top-k in the paper and are an
 * input here; eps holds the caller's N(0, 1) draws.
 *
 * bfloat16 only (SP_EUNSUPPORTED otherwise).  Weights use the [out, in]
 * layout; vectors are float32.  Every array is 16-byte aligned (SP_EINVAL
 * otherwise).  The residual stream is float32; every product
 * operand and result is rounded once to bfloat16.  d <= 4096.
 */
typedef struct {
  const float* ln1_g;  /* [d] */
  const float* ln1_b;  /* [d] */
  const void* W_v;     /* [d, d] bfloat16 */
  const float* b_v;    /* [d] */
  const void* W_o;     /* [d, d] bfloat16 */
  const float* b_o;    /* [d] */
  const float* ln2_g;  /* [d] */
  const float* ln2_b;  /* [d] */
  const void* W_1;     /* [4d, d] bfloat16 */
  const float* b_1;    /* [4d] */
  const void* W_2;     /* [d, 4d] bfloat16 */
  const float* b_2;    /* [d] */
} sp_denoiser;

/*  X      [T, d] bfloat16 visual rows;  alpha [T] float32 in [0, 1] (values
 *         outside give NaN rows);  eps [T, d] bfloat16
 *  p      (host) the block's parameters, all device pointers, none NULL
 *  out    [T, d] bfloat16 (may not alias X or eps)
 *  ws     workspace of stepprune_workspace_bytes(3, dims, T, ...): float32
 *         [T, d] and bfloat16 [T, d] x 2 and [T, 4d] intermediates
 *  events [0] before, [1] after the whole block (or NULL)
 */
sp_status stepprune_gate_denoise(const sp_dims* dims, const void* X, int64_t T,
                                 const float* alpha, const void* eps, const sp_denoiser* p,
                                 void* out, void* ws, size_t ws_bytes,
                                 const hipEvent_t* events, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * The cross-modal input encoder of Eq. 3 (Section "Conditional Sequential
 * Pointer Policy", paragraph "Cross-Modal Input Encoder"):
 *
 *   E~_b = g_text LN(E_b W_p^T)                (LayerNorm without scale or
 *                                               shift, biased variance, eps 1e-5)
 *   H_b  = Enc([X_b; E~_b])[first N_b rows]
 *
 * for every image b.  Enc is two pre-norm transformer blocks of width d:
 *   h = x + W_o MHA(LN1(x)) + b_o,   y = h + W_2 GELU(W_1 LN2(h) + b_1) + b_2,
 * LayerNorm with scale and shift (eps 1e-6), multi-head attention with heads
 * of width 128 over q, k, v = LN1(x) W_qkv^T + b_qkv (rows [0, d) query,
 * [d, 2d) key, [2d, 3d) value of W_qkv; head j takes columns [128 j, 128 j +
 * 128) of each), scores scaled by 128^(-1/2), over the image's whole sequence
 * (bidirectional, the paper's default; SP_ENC_CAUSAL: token i attends to
 * tokens j <= i, visual tokens first), the MLP 4d wide with the exact GELU.
 * Images never attend to each other; the text rows are not output.  H takes
 * the place of X as stepprune_project's input (the compaction still gathers
 * the original X).
 *
 * bfloat16 only, d a multiple of 128 up to 4096, d_text a multiple of 64
 * (SP_EUNSUPPORTED / SP_EINVAL otherwise).  Weights are bfloat16 [out, in],
 * vectors float32, every array 16-byte aligned.  The residual stream is
 * float32; the text product, LayerNorm outputs, products, biased q/k/v,
 * attention probabilities weighting the values, head outputs, the GELU output
 * and H are rounded once to bfloat16.
 */
typedef struct {
  const float* ln1_g;  /* [d] */
  const float* ln1_b;  /* [d] */
  const void* W_qkv;   /* [3d, d] bfloat16 */
  const float* b_qkv;  /* [3d] */
  const void* W_o;     /* [d, d] bfloat16 */
  const float* b_o;    /* [d] */
  const float* ln2_g;  /* [d] */
  const float* ln2_b;  /* [d] */
  const void* W_1;     /* [4d, d] bfloat16 */
  const float* b_1;    /* [4d] */
  const void* W_2;     /* [d, 4d] bfloat16 */
  const float* b_2;    /* [d] */
} sp_encoder_block;

enum { SP_ENC_CAUSAL = 1u };

/*  X        [T_vis, d] visual tokens, packed by img_off [B+1] (device)
 *  E_text   [T_txt, d_text] text tokens, packed by text_off [B+1] (device)
 *  W_p      [d, d_text] bfloat16 text projection; g_text its gain
 *  blocks   (host) [2] the blocks' parameters, device pointers, none NULL
 *  max_seq  (host) upper bound on any image's N_b + L_b; an image above it is
 *           a device error (SP_DEV_GROUP_TOO_LARGE) and its rows of H are
 *           undefined
 *  flags    0 or SP_ENC_CAUSAL
 *  H        out [T_vis, d] bfloat16
 *  ws       workspace of stepprune_workspace_bytes(4, dims, T_vis, T_txt, B,
 *           0, max_seq, 0); its first 4 bytes are the device error word
 *  events   [0] before, [1] after the whole encoder (or NULL)
 */
sp_status stepprune_encode(const sp_dims* dims, const void* X, int64_t T_vis,
                           const int32_t* img_off, int32_t B,
                           const void* E_text, const int32_t* text_off, int64_t T_txt,
                           const void* W_p, float g_text,
                           const sp_encoder_block* blocks, int32_t max_seq, uint32_t flags,
                           void* H, void* ws, size_t ws_bytes,
                           const hipEvent_t* events, hipStream_t stream);

/* Workspace bytes for stage `which` (0 project, 1 select, 2 compact, 3 gate
   and denoiser, 4 input encoder; for 3, T_vis is the token count T; for 4,
   max_group is max_seq) at the given sizes (host).  Returns 0 for invalid
   arguments. */
size_t stepprune_workspace_bytes(int32_t which, const sp_dims* dims, int64_t T_vis,
                                 int64_t T_txt, int32_t B, int32_t G,
                                 int32_t max_group, int32_t max_cap);

/* Synchronises `stream`, then copies the device error word of `ws` to *code
   (host) and clears it.  Returns SP_EDEVICE if it was set. */
sp_status stepprune_read_device_error(void* ws, hipStream_t stream, int32_t* code);

/* Static description of a status code. */
const char* stepprune_status_string(sp_status status);

#ifdef __cplusplus
}
#endif
#endif /* STEPPRUNE_H */
