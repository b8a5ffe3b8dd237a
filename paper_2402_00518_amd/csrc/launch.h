// Host-callable launchers of the exit-head kernels (defined in kernels.hip).
// Every launcher enqueues on `stream` and returns the launch status; shapes
// have been validated by the caller.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ee {

constexpr int kTokenPad = 64;     // padding of the token dimension

// Split-K tail of the MLP exit's token-by-feature products (the down
// projection and dZ): the outputs of tokens >= tok0 and features >= feat0
// (one of the two is 0) are computed as `splits` partial sums over slices of
// K, slice z at z * n * h floats from slice 0; the rest take all of K.
// split_tail(f32, n, h, K) picks one for a shape.
struct SplitTail {
  int tok0;
  int feat0;
  int splits;  // 1: no split
};

// Width of the column slices over which the logits and weight-gradient
// GEMMs keep their softmax and gain-gradient partials (one wave's columns).
int gemm_part_cols(bool f32);

// Row statistics of the exit norm.  RMSNorm (mu == NULL): r[n] =
// (mean_j x[n][j]^2 + eps)^(-1/2).  LayerNorm: mu[n] = mean_j x[n][j] and
// r[n] = (mean_j (x[n][j] - mu[n])^2 + eps)^(-1/2).
// clear, clear_exit (optional): the device error flag and an exit's
// range-check flag, set to 0 by the launch (the first kernel of a step, or
// of an exit, clears them instead of a launch of its own).
hipError_t launch_row_rms(bool x_f32, const void *x, int64_t ldx, int n, int h, float eps,
                          float *r, hipStream_t stream, float *mu = nullptr, int *clear = nullptr,
                          int *clear_exit = nullptr);
// RMSNorm statistics of the fp32 rows the split down projection leaves
// (see gemm_down_residual): the split outputs are first replaced by the sum
// of their slices, in slice order.
hipError_t launch_row_rms_split(float *x, int n, int h, float eps, float *r, SplitTail sp, hipStream_t stream);

// Apply the row statistics, a gain and a bias: x_hat = (x - mu[n]) * r[n]
// (mu == NULL: no centring; r == NULL: no scale), z = x_hat * gain + bias
// (bias may be NULL).  Writes any of z [n][h], x_hat [n][h] (row-major) and
// x_hat^T [h][ldn] (token-contiguous, columns n..ldn-1 zero).  Output
// element type = `f32`.  clear, clear_exit: as for launch_row_rms.
hipError_t launch_norm_apply(bool x_f32, bool f32, const void *x, int64_t ldx, const float *r,
                             const void *gain, int n, int ldn, int h, void *z, void *x_hat,
                             void *x_hat_t, hipStream_t stream, const float *mu = nullptr,
                             const void *bias = nullptr, int *clear = nullptr, int *clear_exit = nullptr);

// launch_row_rms followed by launch_norm_apply (z and x_hat^T, a gain, an
// optional bias) as one pass over x, for rows that fit a block's LDS
// (norm_rows(h, f32): 8 rows of h inputs in at most 128 KB).  Same results;
// x and the outputs are of the exit's element type `f32`.
bool norm_rows(int h, bool f32);
hipError_t launch_norm_rows(bool f32, const void *x, int64_t ldx, int n, int ldn, int h, float eps, const void *gain,
                            const void *bias, float *r, float *mu, void *z, void *x_hat_t, hipStream_t stream,
                            int *clear = nullptr, int *clear_exit = nullptr);

// The exit norm of a few rows in one launch (decode): z[n][h] = (x - mu) r *
// gain (+ bias), with mu the row mean when `centre` (LayerNorm), else 0, and
// r = (mean (x - mu)^2 + eps)^(-1/2).  x is fp32 when x_f32, z is `f32`.
hipError_t launch_row_norm(bool x_f32, bool f32, const void *x, int n, int h, float eps, const void *gain,
                           const void *bias, bool centre, void *z, hipStream_t stream);

// Combine the per-tile softmax partials of each token into LSE, the row NLL
// and the loss weight s_n.  Also flags targets outside [0, V).
struct CeReduceArgs {
  const float *part_m;
  const float *part_l;
  const float *tgt;
  const int32_t *targets;
  const float *token_w;   // or NULL
  float *lse;             // [ldn] log-sum-exp
  float *sn;              // [ldn] s_n = w_e m_n / N
  float *row_loss;        // [n] or NULL
  float *block_sums;      // [cdiv(n, 32)]
  int *flag;
  int n, ldn, vocab, tiles;
  float exit_weight;
  int dynamic_weights;
  int shift0;             // the partials are of exp(S) (EpiLogits shift0 1 or 2), see kernels.hip
  int *fallback;          // shift0: set to 1 if a row is outside the unshifted range
  float *coef;            // shift0: [ldn] s_n exp(-LSE_n)
  const int *run_if;      // or NULL: run only if *run_if is non-zero
};
hipError_t launch_ce_reduce(const CeReduceArgs &a, hipStream_t stream);

// In place: G[v][n] = P[v][n] * s_n exp(m[v / vtile][n] - LSE_n) - (v == y_n) * s_n
// (0 for n >= N).  With gsum_part, also the fp32 row sums of G over each
// chunk of 2048 tokens: gsum_part[chunk][v] (seed_chunks(ldn) chunks).
int seed_chunks(int ldn);
hipError_t launch_seed(bool f32, void *P, const float *part_m, const float *lse, const float *sn,
                       const int32_t *targets, int n, int ldn, int vocab, int vtile, hipStream_t stream,
                       float *gsum_part = nullptr);

// After the unshifted cross-entropy reduce: if *fallback is set, the seed
// (as launch_seed, with G's row sums into gsum_part if it is not NULL); else
// the operand scale, x_hat_t[j][c] *= coef[c] (c < n) and, at each token's
// target, P[y_c][c] -= exp(lse[c]), so that P holds P' with
// G = diag(coef) P'.  x_hat_t [h][ldn], P [V][ldn], element type `f32`.
// The same launch also does launch_final_loss's work (block_sums .. first).
hipError_t launch_seed_or_scale(bool f32, void *P, void *x_hat_t, const float *part_m, const float *lse,
                                const float *sn, const float *coef, const int32_t *targets, int n, int ldn, int h,
                                int vocab, int vtile, const int *fallback, const float *block_sums, int blocks,
                                float *loss, float *total, float w, int first, hipStream_t stream,
                                float *gsum_part = nullptr);
// After launch_seed_or_scale, for an exit with a bias: unless *fallback is
// set (the seed wrote them), the row sums of G = diag(coef) P' per chunk of
// 2048 tokens, gsum_part[chunk][v] = sum_{c in chunk, c < n} coef[c] P'[v][c],
// as launch_seed's.
hipError_t launch_gsum_unshifted(bool f32, const void *P, const float *coef, int n, int ldn, int vocab,
                                 const int *fallback, float *gsum_part, hipStream_t stream);

// loss[0] = sum(block_sums) / n;  total[0] = (first ? 0 : total[0]) + w * loss[0].
hipError_t launch_final_loss(const float *block_sums, int blocks, int n, float *loss, float *total,
                             float w, int first, hipStream_t stream);

// out[j] (=|+=) sum_t part_a[t][j] (+ sum_t part_b[t][j]).
hipError_t launch_gain_reduce(const float *part_a, int tiles_a, const float *part_b, int tiles_b,
                              int h, float *out, int accumulate, hipStream_t stream);

// RMSNorm backward through the exit norm of an MLP exit:
//   dz_hat = dZ * gain,  z_hat = y * r,  dY = r (dz_hat - z_hat mean_j(dz_hat z_hat)),
// with dZ as gemm_dz leaves it for the split sp (its slices added in order),
// each row first scaled by row_scale[n] unless *scale_off is non-zero (dZ
// computed from P', see launch_seed_or_scale).
hipError_t launch_norm_bwd(bool f32, const float *dz, const float *y, const float *r, const void *gain,
                           int n, int h, void *dy, hipStream_t stream, SplitTail sp = SplitTail{0, 0, 1},
                           const float *row_scale = nullptr, const int *scale_off = nullptr);


// ------------------------------------------------------------------ GEMMs
// Logits^T = W_out Z^T with the softmax-partials epilogue: shift0 = 0,
// P = exp(S - m); 1, P = exp(S) and the slice maxima; 2, P = exp(S) and no
// maxima.  With run_if, a launch that runs only if *run_if is non-zero (one
// block per CU looping over the tiles).
hipError_t gemm_logits(bool f32, const void *w_out, const void *z, int vocab, int n, int h, void *P,
                       int ldn, float *part_m, float *part_l, float *tgt, const int32_t *targets,
                       hipStream_t stream, int shift0 = 0, const int *run_if = nullptr);
// dW[M][h] = (G^T X_hat) * gain with gain-gradient partials (K = tokens, both operands
// token-contiguous with leading dimension ldn).  With a LayerNorm bias:
// dW += gsum b^T and bias-gradient partials part_b (gsum[v] = sum_n G[n][v]).
hipError_t gemm_weight_grad_kk(bool f32, const void *g_t, const void *xhat_t, int m, int h, int ldn,
                               const void *gain, const void *w, float *dw, float *part, int accumulate,
                               hipStream_t stream, const float *gsum = nullptr, const void *bias = nullptr,
                               float *part_b = nullptr);
// Two such weight gradients that share x_hat and the gain (no bias), all
// operands token-contiguous with leading dimension ldn (g1_t, g2_t [m][ldn],
// xhat_t [h][ldn]): the gate and up gradients of the MLP exit, one launch
// (the second problem's tiles follow the first's, filling the CUs its last
// round leaves idle).
hipError_t gemm_weight_grad_kk_pair(bool f32, const void *g1_t, const void *g2_t, const void *xhat_t, int m, int h,
                                    int ldn, const void *gain, const void *w1, const void *w2, float *dw1, float *dw2,
                                    float *part1, float *part2, int accumulate, hipStream_t stream);
// One product for both projections of the SwiGLU MLP (W_gate and W_up rows
// interleaved in blocks of 32 on their way into LDS): H_g = U W_gate^T and
// H_u = U W_up^T, stored side by side per element (hgu [n][I] pairs of the
// element type), and A = silu(H_g) H_u [n][I].  inter: a multiple of 32.
hipError_t gemm_gate_up_swiglu(bool f32, const void *u, const void *w_gate, const void *w_up, int n, int inter,
                               int h, void *hgu, void *act, hipStream_t stream);
// K values per slice when a product of depth K runs as `splits` partial sums.
int split_kchunk(int K, int splits);
// Y[n][h] = X + A W_down^T  (fp32 out).  With sp.splits > 1 the outputs in
// sp's region are sp.splits partial sums over slices of I: slice 0 (which
// adds X) in place, slice z at Y + z n h, so Y holds splits n h floats;
// launch_row_rms_split with the same split adds them up.
// split_tail: the split for n tokens by h features over a sum of depth K (a
// shape-only rule that simulates the dispatch of a few candidates).
SplitTail split_tail(bool f32, int n, int h, int K);
hipError_t gemm_down_residual(bool f32, const void *act, const void *w_down, const void *x, int n,
                              int h, int inter, float *y, hipStream_t stream, SplitTail sp = SplitTail{0, 0, 1});
// dZ[n][h] = G W_out with G stored transposed [V][ldn]  (fp32 out), with
// the split sp of its vocabulary sum (the buffer holds sp.splits n h floats).
// (With the unshifted logits the operand is P' and G = diag(coef) P': the
// norm backward applies coef, see launch_norm_bwd.)
hipError_t gemm_dz(bool f32, const void *g_t, const void *w_out, int n, int ldn, int h, int vocab,
                   float *dz, hipStream_t stream, SplitTail sp = SplitTail{0, 0, 1});
// One launch of two independent products of the MLP backward:
//   dA = dY W_down with the SwiGLU backward epilogue (dH_g, dH_u, stored
//   token-contiguous: dhg_t, dhu_t [I][ldn], columns n..ldn-1 zero), and
//   dW_down[h][I] (=|+=) dY^T A.
hipError_t gemm_da_swiglu_dw_down(bool f32, const void *dy, const void *w_down, int n, int inter, int h,
                                 const void *hgu, void *dhg_t, void *dhu_t, int ldn, const void *act, float *dwd,
                                 int accumulate, hipStream_t stream);

// ------------------------------------------------------------- optimizer
// One tensor of a fused Adam launch (optim.hip).  Pointers are device
// addresses, 16-byte aligned; master may be NULL.
constexpr int kAdamMaxTensors = 8;
struct AdamTensorArgs {
  void *param;            // [numel], bf16 when `bf16`, else fp32
  float *master;          // [numel] or NULL
  const float *grad;      // [numel]
  float *exp_avg;         // [numel]
  float *exp_avg_sq;      // [numel]
  int64_t numel;
  int64_t first_block;    // set by launch_adam
  int32_t bf16;
  int32_t pad;
};
struct AdamBatchArgs {
  AdamTensorArgs t[kAdamMaxTensors];
  int32_t count;
  float beta1, beta2, eps;
  float lr_bc1;           // lr / (1 - beta1^step)
  float inv_bc2;          // 1 / (1 - beta2^step)
};
// ---------------------------------------------------------------- decode
// Skinny products of the decode-time exit head (decode.hip): n token rows
// (any n; 32 per pass) against a weight of `rows` K-contiguous rows, K a
// multiple of 64.  Outputs are token-major, [n][rows].
int decode_tiles(int rows);  // partial rows per token of decode_logits
hipError_t decode_store(bool f32, const void *w, int rows, const void *z, int n, int k, void *out,
                        hipStream_t stream);
hipError_t decode_swiglu(bool f32, const void *w, int rows, const void *z, int n, int k, const void *hg,
                         void *act, hipStream_t stream);
hipError_t decode_residual(bool f32, const void *w, int rows, const void *z, int n, int k, const void *x,
                           float *y, hipStream_t stream);
// Softmax partials of S = Z W_out^T: [decode_tiles(vocab)][n] max, sum exp, lowest argmax.
hipError_t decode_logits(bool f32, const void *w_out, int vocab, const void *z, int n, int h, float *part_m,
                         float *part_l, int32_t *part_arg, hipStream_t stream);
// Greedy token, its probability, and confidence > threshold, per token row.
hipError_t decode_decide(const float *part_m, const float *part_l, const int32_t *part_arg, int tiles, int n,
                         float threshold, int32_t *token, float *confidence, int32_t *exit_flag,
                         hipStream_t stream);

// Blocks one tensor of `numel` elements occupies in a launch.
int64_t adam_blocks(int64_t numel);
hipError_t launch_adam(AdamBatchArgs b, hipStream_t stream);

}  // namespace ee
