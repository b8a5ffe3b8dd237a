/*
 * ee_tuning.h -- C ABI of the MI355X (gfx950) early-exit head training step.
 *
 * EE-Tuning (arXiv 2402.00518) converts a frozen pre-trained LLM into an
 * early-exit one by attaching exit heads to intermediate hidden states and
 * tuning only those heads.  This library runs the hot part of one tuning
 * iteration (Sec. 2.2, "Computational efficiency", item 2): for every exit,
 * the forward pass, the next-token loss, and the backward pass into the
 * exit's own parameters.  The backbone is frozen, so no gradient is produced
 * for the hidden states (Sec. 2.2, first paragraph).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Device pointers are HIP device addresses on the current device; host
 *    pointers are marked "host".  Every device pointer must be 16-byte
 *    aligned.  The caller owns all memory; the library allocates nothing per
 *    call and keeps no state besides its loaded kernels and a thread-local
 *    error string.
 *  - `stream` is a hipStream_t (NULL = the null stream).  Work is enqueued
 *    asynchronously on it; scalars written to device memory are valid once
 *    the stream has been synchronised.
 *  - Every error that the host can detect (NULL pointers, bad shapes, bad
 *    dtype, misalignment, small workspace, aliased outputs, unsupported exit
 *    kind) is reported before anything is enqueued: nothing runs.  A detail
 *    string is then available from ee_last_error().
 *  - Targets outside [0, V) are a precondition violation that only the
 *    device sees: the kernels never access memory with them, record the
 *    fault in the workspace, and ee_check_device_error() reports it.
 *  - Matrices are row-major.  The output embedding, an h x V matrix in the
 *    paper (Sec. 2.1, Embedding exit), is stored as W_out[V][h], the common
 *    checkpoint layout; it is the same matrix.
 *  - Mixed precision (EE_BF16): hidden states and weights are bf16; norms,
 *    softmax and losses run in fp32; GEMMs take bf16 operands with fp32
 *    accumulation; weight gradients are written in fp32.  EE_F32 keeps every
 *    operand in fp32.
 */
#ifndef EE_TUNING_H
#define EE_TUNING_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define EE_ABI_VERSION 2

/* Each enum below also spans every int value (the *_RANGE_* enumerators are
 * never passed or returned): a caller may hand the library any int in one of
 * these types, an unknown value is rejected with an error, and reading it is
 * defined behaviour in the C++ library as well. */
typedef enum ee_status {
  EE_OK = 0,
  EE_ERR_NULL = 1,        /* a required pointer is NULL                       */
  EE_ERR_SHAPE = 2,       /* a size is out of range or not a multiple of 64   */
  EE_ERR_DTYPE = 3,       /* unknown dtype, or dtypes of exits disagree       */
  EE_ERR_ALIGN = 4,       /* a device pointer is not 16-byte aligned          */
  EE_ERR_WORKSPACE = 5,   /* workspace smaller than ee_workspace_bytes()      */
  EE_ERR_ALIAS = 6,       /* an output overlaps another output or an input    */
  EE_ERR_UNSUPPORTED = 7, /* exit kind or flag not implemented (Layer exit)   */
  EE_ERR_TARGET = 8,      /* device saw a target outside [0, V)               */
  EE_ERR_HIP = 9,         /* a HIP runtime call or launch failed              */
  EE_STATUS_RANGE_MIN = -0x7FFFFFFF - 1,
  EE_STATUS_RANGE_MAX = 0x7FFFFFFF
} ee_status;

typedef enum ee_dtype {
  EE_F32 = 0,
  EE_BF16 = 1,
  EE_DTYPE_RANGE_MIN = -0x7FFFFFFF - 1,
  EE_DTYPE_RANGE_MAX = 0x7FFFFFFF
} ee_dtype;

/* Exit architectures of Sec. 2.1 ("Architectures of early exits"):
 *  EMBEDDING  logits = X W_out^T                                  (one matrix)
 *  NORM       logits = RMSNorm_gamma(X) W_out^T       (RMSNorm as in Sec. 3.2)
 *  MLP        Y = X + SwiGLU(RMSNorm_gamma_mlp(X)) W_down^T   (pre-norm residual
 *             module, Fig. 2 caption), logits = RMSNorm_gamma(Y) W_out^T
 *  LAYER      a full Transformer layer in front of Norm: EE_ERR_UNSUPPORTED.
 * RMSNorm: s_hat = s (mean_j s_j^2 + eps)^(-1/2), then times the gain.
 * SwiGLU:  A = silu(U W_gate^T) * (U W_up^T), silu(t) = t / (1 + exp(-t)). */
typedef enum ee_exit_kind {
  EE_EXIT_EMBEDDING = 0,
  EE_EXIT_NORM = 1,
  EE_EXIT_MLP = 2,
  EE_EXIT_LAYER = 3,
  EE_EXIT_KIND_RANGE_MIN = -0x7FFFFFFF - 1,
  EE_EXIT_KIND_RANGE_MAX = 0x7FFFFFFF
} ee_exit_kind;

/* Normalisation of a Norm exit (Sec. 2.1: "a LayerNorm or RMSNorm module").
 *  RMS    s_hat = s (mean_j s_j^2 + eps)^(-1/2)                    (default)
 *  LAYER  s_hat = (s - mean_j s_j) (mean_j (s_j - mean)^2 + eps)^(-1/2),
 *         z = s_hat * gamma + beta, with beta optional (NULL: no bias).
 * LAYER is available for NORM exits; MLP exits use RMSNorm. */
typedef enum ee_norm {
  EE_NORM_RMS = 0,
  EE_NORM_LAYER = 1,
  EE_NORM_RANGE_MIN = -0x7FFFFFFF - 1,
  EE_NORM_RANGE_MAX = 0x7FFFFFFF
} ee_norm;

/* Step flags. */
#define EE_FLAG_DYNAMIC_TOKEN_WEIGHTS 1u
/* Sec. 2.3 "Dynamic token-wise loss weights" (loss in Appendix A.3,
 * "Dynamic token-wise loss weighting"): weight each token's NLL by its
 * detached confidence c_n = max_v softmax(S[n, :]).  The paper weights by
 * c_n alone; caller token weights, when given, multiply it (m_n = token_w[n]
 * * c_n), so a row masked by weight 0 stays masked. */

/* One exit's parameters (read-only; may alias another exit's, e.g. after
 * the "copy" initialisation of Sec. 2.1). */
typedef struct ee_exit {
  int32_t kind;          /* ee_exit_kind                                     */
  int32_t dtype;         /* ee_dtype of the hidden states and all weights    */
  int64_t hidden;        /* h: multiple of 64, 64 <= h <= 32768 (MLP: 8192)  */
  int64_t vocab;         /* V: 1 <= V <= 1048576                             */
  int64_t intermediate;  /* I (MLP only): multiple of 64, <= 65536; else 0   */
  float rms_eps;         /* norm epsilon, >= 0 (Llama-2 uses 1e-5)           */
  int32_t norm;          /* ee_norm; EE_NORM_LAYER only for NORM exits       */
  const void *w_out;     /* [V][h]                                           */
  const void *gamma;     /* [h] exit RMSNorm gain (NORM, MLP)                */
  const void *gamma_mlp; /* [h] MLP pre-norm gain (MLP)                      */
  const void *w_gate;    /* [I][h] (MLP)                                     */
  const void *w_up;      /* [I][h] (MLP)                                     */
  const void *w_down;    /* [h][I] (MLP)                                     */
  const void *beta;      /* [h] LayerNorm bias (NORM + LAYER), or NULL       */
} ee_exit;

/* Gradients of one exit's parameters, fp32, same shapes as the parameters.
 * Pointers for parameters the exit kind does not have are ignored. */
typedef struct ee_exit_grads {
  float *d_w_out;
  float *d_gamma;
  float *d_gamma_mlp;
  float *d_w_gate;
  float *d_w_up;
  float *d_w_down;
  float *d_beta;         /* required when the exit has a bias                */
} ee_exit_grads;

/* Bytes of device workspace needed to run the given exits over n_tokens
 * rows, forward and backward.  One workspace serves every exit of
 * ee_multi_exit_step (they run one after another on the stream).  Returns 0
 * if the arguments are invalid (ee_last_error() says why). */
size_t ee_workspace_bytes(int n_exits, const ee_exit *exits, int64_t n_tokens);

/* Forward pass and loss of one exit (Sec. 2 loss; Sec. 2.1 architectures).
 *
 *   L_e = (1/N) sum_n m_n * ( logsumexp_v S[n, v] - S[n, y_n] ),
 *   S   = exit(hidden) W_out^T,
 *
 * with m_n = token_w[n] (all ones when token_w is NULL), times the detached
 * confidence with EE_FLAG_DYNAMIC_TOKEN_WEIGHTS.  The mean over the N rows
 * reads the paper's sum over tokens as a per-token average.
 *
 *   hidden    device [N][h], dtype of the exit: the frozen backbone's hidden
 *             states at this exit; row n predicts targets[n] (already
 *             shifted by one position).
 *   targets   device [N] int32 token ids in [0, V).
 *   token_w   device [N] fp32, or NULL.
 *   exit_weight  w_e, scales the gradients that ee_head_backward produces.
 *   loss      device [1] fp32: L_e (not multiplied by w_e).
 *   row_loss  device [N] fp32 per-row NLL, or NULL.
 *   ws        device workspace of ws_bytes >= ee_workspace_bytes(1, e, N).
 *
 * Leaves in ws everything ee_head_backward needs, including the logit
 * gradient seed w_e m_n / N * (softmax(S[n]) - onehot(y_n)).  The workspace
 * must not be touched between the two calls. */
ee_status ee_head_forward_loss(const ee_exit *e, const void *hidden,
                               const int32_t *targets, const float *token_w,
                               int64_t n_tokens, float exit_weight,
                               uint32_t flags, void *ws, size_t ws_bytes,
                               float *loss, float *row_loss, void *stream);

/* Backward pass of one exit into its own parameters only (Sec. 2.2): writes
 * w_e * dL_e/dtheta_e for every parameter of the exit kind, consuming the
 * workspace a preceding ee_head_forward_loss left for the same exit and N.
 * accumulate = 0 overwrites the gradient buffers, 1 adds to them. */
ee_status ee_head_backward(const ee_exit *e, int64_t n_tokens, void *ws,
                           size_t ws_bytes, const ee_exit_grads *g,
                           int accumulate, void *stream);

/* One full step over all exits (Sec. 2.2: exits are tuned independently and
 * their losses combine as a weighted sum, Sec. 1):
 *
 *   L = sum_e exit_weights[e] * L_e,
 *
 * equal to ee_head_forward_loss + ee_head_backward for each exit in turn.
 * All exits share N, V, targets, token_w and flags; each has its own hidden
 * states hidden[e] (device pointers in a host array) and parameters.
 *   exit_weights   host [n_exits]
 *   grads          host [n_exits] gradient buffer sets
 *   loss_total     device [1];  loss_per_exit device [n_exits] or NULL. */
ee_status ee_multi_exit_step(int n_exits, const ee_exit *exits,
                             const void *const *hidden, const int32_t *targets,
                             const float *token_w, int64_t n_tokens,
                             const float *exit_weights, uint32_t flags,
                             const ee_exit_grads *grads, int accumulate,
                             void *ws, size_t ws_bytes, float *loss_total,
                             float *loss_per_exit, void *stream);

/* Synchronises `stream`, then reports EE_ERR_TARGET if the latest
 * ee_head_forward_loss or ee_multi_exit_step call on this workspace saw a
 * target outside [0, V) (each such call starts with a clean record), and
 * clears the record.  EE_OK otherwise. */
ee_status ee_check_device_error(void *ws, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------- decode
 * Confidence-based exit decision at decode time (Sec. 3, "Inference":
 * greedy decoding; an exit emits its most likely token as soon as the
 * maximum next-token probability there is above a threshold, and a
 * threshold of 1 disables early exits).  Forward only, for n_rows hidden
 * states at one exit (typically the batch of sequences being decoded):
 *
 *   S_n          = exit(hidden_n) W_out^T          (the architectures above)
 *   token[n]     = argmax_v S_n[v], the lowest id among tied maxima
 *   confidence[n]= max_v softmax(S_n)[v]           (fp32)
 *   exit_flag[n] = confidence[n] > threshold ? 1 : 0   ("above": strict)
 *
 *   hidden      device [n_rows][h], dtype of the exit.
 *   token, exit_flag  device int32 [n_rows];  confidence device fp32 [n_rows].
 *   ws          device workspace of ws_bytes >= ee_decode_workspace_bytes().
 * Errors as for the training entry points (nothing is enqueued); threshold
 * must not be NaN.  Logits are accumulated in fp32 from the exit's dtype;
 * no logit tensor is written (each 32-row slice of W_out is reduced to
 * per-token max / argmax / sum of exponentials on the fly). */
size_t ee_decode_workspace_bytes(const ee_exit *e, int64_t n_rows);

ee_status ee_exit_decide(const ee_exit *e, const void *hidden, int64_t n_rows,
                         float threshold, int32_t *token, float *confidence,
                         int32_t *exit_flag, void *ws, size_t ws_bytes,
                         void *stream);

/* The same decision for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): no workspace argument and nothing allocated per call.  The
 * workspace is a fixed array of EE_STATIC_SCRATCH_BYTES (32 MiB) that the
 * library holds on each GPU it runs on until the process ends; its device
 * address is looked up on the first call on a device.
 *  - Runs on the current device; `stream` must belong to it.
 *  - EE_ERR_WORKSPACE (nothing enqueued) when ee_decode_workspace_bytes(e,
 *    n_rows) exceeds EE_STATIC_SCRATCH_BYTES (e.g. a bf16 Norm exit with
 *    h = 8192 and V = 32000 fits about 1100 rows).
 *  - All calls on one GPU share its one array: calls whose work overlaps on
 *    that GPU (other streams, or threads without an order between them)
 *    race and their results are undefined.  Calls in order on one stream are
 *    safe; every workspace word a call reads it has written first, so what
 *    an earlier call left there does not matter.
 * Arguments, other errors and results as ee_exit_decide; outputs must not
 * overlap each other or the inputs (EE_ERR_ALIAS). */
#define EE_STATIC_SCRATCH_BYTES ((size_t)32 << 20)

ee_status ee_exit_decide_static(const ee_exit *e, const void *hidden,
                                int64_t n_rows, float threshold,
                                int32_t *token, float *confidence,
                                int32_t *exit_flag, void *stream);

/* ---------------------------------------------------------------- update
 * Adam update of exit parameters: the optimiser of Sec. 3 ("Tuning": Adam
 * with beta1 = 0.9, beta2 = 0.95, eps = 1e-5), the last part of a tuning
 * iteration (Sec. 2.2, "Computational efficiency").  For every element, in
 * fp32, with t = step:
 *
 *   m <- beta1 m + (1 - beta1) g
 *   v <- beta2 v + (1 - beta2) g^2
 *   p <- p - lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)
 *
 * (Kingma and Ba's update; no weight decay, no clipping: the paper names
 * neither).  p is the fp32 master copy when `master` is given, and the
 * stored parameter then receives p rounded to its dtype (bf16: to nearest
 * even); without a master the stored parameter is read, updated and written
 * back.  One call updates any number of tensors (fused, up to 8 per kernel
 * launch). */
typedef struct ee_adam_tensor {
  void *param;         /* device [numel] of `dtype`, updated in place            */
  float *master;       /* device fp32 [numel] master weights, or NULL            */
  const float *grad;   /* device fp32 [numel], e.g. from ee_head_backward        */
  float *exp_avg;      /* device fp32 [numel] first moment m (zeros before t=1)  */
  float *exp_avg_sq;   /* device fp32 [numel] second moment v (zeros before t=1) */
  int64_t numel;       /* >= 0; 0 skips the tensor (its pointers may be NULL)    */
  int32_t dtype;       /* ee_dtype of param                                      */
  int32_t reserved;    /* must be 0                                              */
} ee_adam_tensor;

/* tensors: host array of n_tensors descriptors (n_tensors >= 0).
 * lr: this update's step size (finite, e.g. from ee_lr_schedule); beta1,
 * beta2 in [0, 1); eps >= 0; step >= 1 counts this update.
 * Errors (nothing is enqueued): EE_ERR_NULL for a missing pointer of a
 * non-empty tensor, EE_ERR_ALIGN, EE_ERR_DTYPE, EE_ERR_SHAPE (numel < 0, a
 * reserved field set, hyper-parameters out of range), EE_ERR_ALIAS when a
 * written buffer (param, master, exp_avg, exp_avg_sq of any tensor)
 * overlaps another buffer of the call. */
ee_status ee_adam_update(int n_tensors, const ee_adam_tensor *tensors, float lr,
                         float beta1, float beta2, float eps, int64_t step,
                         void *stream);

/* Learning rate of update `step` (1-based) under the schedule of Sec. 3
 * ("Tuning": linear warmup over a fraction of the iterations, then linear
 * decay from lr_max to lr_min).  With W = floor(warmup_fraction *
 * total_steps):  lr_max * step / W for step <= W;  lr_min + (lr_max - lr_min)
 * (total_steps - step) / (total_steps - W) up to total_steps;  lr_min after.
 * Host function.  Returns NaN (and sets ee_last_error) if step < 1,
 * total_steps < 1 or warmup_fraction is outside [0, 1). */
double ee_lr_schedule(int64_t step, int64_t total_steps, double warmup_fraction,
                      double lr_max, double lr_min);

/* Kernel timing, for diagnostics.  Between ee_profile_start() and
 * ee_profile_stop(), every kernel the step and update functions launch is
 * bracketed by a pair of HIP events recorded on the launch stream (the
 * events cost a few microseconds per launch; keep them out of headline
 * timings).
 * ee_profile_stop() waits for the recorded events, fills up to `capacity`
 * entries of `out` (host array) with per-kernel launch counts and summed
 * durations, in first-launch order, and returns the number of entries, or -1
 * on a HIP error.  Names are static strings owned by the library.  Process-
 * wide; not meant for concurrent use from several threads. */
typedef struct ee_kernel_time {
  const char *name;
  int32_t launches;
  double total_ms;
} ee_kernel_time;

ee_status ee_profile_start(void);
int ee_profile_stop(ee_kernel_time *out, int capacity);

/* Static description of a status code. */
const char *ee_status_string(ee_status s);

/* Detail of the last failure on the calling thread ("" if none). */
const char *ee_last_error(void);

/* EE_ABI_VERSION of the loaded library. */
int ee_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* EE_TUNING_H */
