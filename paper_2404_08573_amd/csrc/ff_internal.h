// Internal interface between the host API (ff_api.cpp) and the gfx950 kernels
// (ff_kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace ffk {

// Largest operand row length (layer width) of the forward product: a 256-row
// tile of it spans under 2^31 bytes, the range of one buffer descriptor.
constexpr int kMaxWidth = 1 << 20;

// Where row r of a layer-0 input comes from.
//   ROWS:     row r of `base` (already embedded or a hidden activity).
//   PAIRS:    rows [0, n_pos) are base rows base_off+r with label lab_a[base_off+r];
//             rows [n_pos, ..) are base rows base_off+r-n_pos with label lab_b[...]
//             (a chunk's positives, then its negatives).
//   EXPAND:   row r is base row base_off + r / n_classes under label r % n_classes
//             (every candidate label of every input, for scoring).
//   MASKED:   row r is base row base_off + r with the n_classes label features
//             zeroed, normalised as if one label feature were 1: the part that
//             every label embedding of the row shares (same norm for every label).
//   NEUTRAL:  row r is base row base_off + r with every label feature 0.1 (the
//             neutral label of Softmax prediction).
enum RowMode : int32_t { ROWS = 0, PAIRS = 1, EXPAND = 2, MASKED = 3, NEUTRAL = 4 };

struct RowMap {
  const float *base;
  const int32_t *lab_a;
  const int32_t *lab_b;
  int32_t mode;
  int32_t n_pos;
  int32_t base_off;
  int32_t n_classes;
};

// Label expansion of a shared-base layer-0 product (scoring).  Base row r
// (normalised, label features zeroed) gives n_classes output rows, row
// r * n_classes + c under label c.  The label feature of the normalised row is
// scale[r], so output row (r, c) is relu(P_r + scale[r] * W[:, c] + b) with
// P = X W^T on the masked rows.
struct LabelExpand {
  int32_t n_classes;
  const float *scale;  // [M]
};
constexpr int kMaxExpand = 16;  // label counts up to this take the shared-base path

// Adam update t: the bias corrections bc1 = 1 - beta1^t and bc2 = 1 - beta2^t
// enter as lr / bc1 and 1 / bc2 (computed in double on the host).
struct AdamArgs {
  float lr, beta1, beta2, eps;
  float lr_bc1, inv_bc2;
};

// Loss scalar finished by the dW kernel from the per-workgroup partials of
// the loss-rows kernel: loss = sum(pos partials)/n_pos + sum(neg partials)/n_neg.
struct LossFinish {
  const float *lpart;  // [nblk][2]
  int32_t nblk;
  int32_t n_pos, n_neg;
  float *loss;         // null: not wanted
};

// Features of a softmax classifier: the concatenation of layer blocks
// A_l[r][j] = s_l[r] * H_l[r][j], block l of width d[l] (s_l null: scale 1).
// Block l's classifier weights are w[l] [C][d[l]] with row stride ldw[l];
// logits = sum over blocks of A_l w_l^T + sum of the n_bias bias vectors.
constexpr int kHeadMaxBlocks = 8;
constexpr int kHeadMaxClasses = 16;
struct HeadFeatures {
  int32_t n_blocks;
  const float *h[kHeadMaxBlocks];
  const float *s[kHeadMaxBlocks];
  int32_t d[kHeadMaxBlocks];
  const float *w[kHeadMaxBlocks];
  int32_t ldw[kHeadMaxBlocks];
  int32_t n_bias;
  const float *bias[kHeadMaxBlocks];
};

// Softmax classifier forward on n rows (C classes), then the softmax.  Writes
// logits [n][C] and pred [n] (argmax, lowest class on ties) when non-null;
// with labels (training) also G[n][C] = (p - onehot) / n, the gradient of the
// mean cross-entropy with respect to the logits, and the per-row loss lrow [n].
hipError_t launch_head_logits(const HeadFeatures &f, int n, int C, const int32_t *labels,
                              float *logits, int32_t *pred, float *G, float *lrow,
                              hipStream_t s);

// Performance-optimised layer backprop through its classifier:
// dZ[r][j] = [H[r][j] > 0] * sum_c G[r][c] Wc[c][j] (H [R][D], Wc [C][D]),
// and ones[r] = 1 (the row scale of the weight-gradient product).
hipError_t launch_po_dz(const float *H, const float *G, const float *Wc, int R, int D, int C,
                        float *dZ, float *ones, hipStream_t s);

// Row splits of the head's weight-gradient reduction.
int head_grad_splits(int n);

// Classifier weight-gradient partials: part[split][C][D] = sum over the
// split's rows of G[r][c] * A[r][f] (the weights in f are not read).
hipError_t launch_head_grad(const HeadFeatures &f, const float *G, int n, int C, int D,
                            int splits, float *part, hipStream_t s);

// Sum of the partials (fixed order), db = sum_r G[r] and loss = mean of lrow
// (fixed order), and one Adam update of W [C][D] and b [C].
hipError_t launch_head_adam(const float *part, int splits, const float *G, const float *lrow,
                            int n, int C, int D, float *W, float *mW, float *vW, float *b,
                            float *mb, float *vb, const AdamArgs &a, float *loss,
                            hipStream_t s);

// Number of per-workgroup loss partial pairs for `rows` rows.
int loss_blocks(int rows);

// Number of column tiles of the forward product on rows x n_cols, which is
// the number of goodness partials per row (one per column tile), and its
// upper bound over all row counts (for sizing scratch).
int fwd_col_tiles(int rows, int n_cols, int dtype);
int fwd_col_tiles_max(int n_cols);
int fwd_expand_col_tiles(int rows, int n_cols, int dtype);

// Embedding (optional) + L2 normalisation (optional) into fp32 or bf16 rows.
// scale_out [rows] (optional): each row's normalisation factor (rounded to
// bf16 when bf16_out), i.e. the value a one-hot label feature takes.
hipError_t launch_embed_norm(const RowMap &m, int rows, int d, float eps, bool normalise,
                             bool bf16_out, void *out, float *scale_out, hipStream_t s);

// H = relu(diag(rowscale) X W^T + b) (optional store) and per-column-tile
// goodness partials gpart[tile][M].  X: [M][K], W: [N][K]; fp32 or bf16
// operands (dtype).  rowscale [M] or null (scale 1): the normalisation of raw
// input rows, applied to the product.
hipError_t launch_fwd(int dtype, const void *X, const void *W, const float *bias,
                      const float *rowscale, int M, int N, int K, float *H, float *gpart,
                      hipStream_t s);

// Shared-base layer-0 forward: X [M][K] normalised masked base rows, W [N][K],
// H [M * ex.n_classes][N] (optional) and gpart[tile][M * ex.n_classes] for the
// expanded rows (see LabelExpand); the number of goodness partials per row is
// fwd_expand_col_tiles(M, N, dtype) (tiles follow the base rows).
hipError_t launch_fwd_expand(int dtype, const void *X, const void *W, const float *bias,
                             const LabelExpand &ex, int M, int N, int K, float *H, float *gpart,
                             hipStream_t s);

// g_r = sum_t gpart[t][r] (into g unless null), c_r = 2 dL/dg_r, and loss
// partials lpart[loss_blocks(R)][2]; s_out (unless null) gets the
// normalisation 1/(sqrt(g_r) + norm_eps) of the activity rows as the next
// layer's input (g_r is their squared norm).  With s_in (the layer input's
// row scales, when its rows are raw), cs_r = c_r * s_in_r.
hipError_t launch_loss(const float *gpart, int ntiles, int R, int n_pos, float theta, float *g,
                       float *c, float *lpart, float *s_out, float norm_eps, const float *s_in,
                       float *cs, hipStream_t s);

// dW = (c . H)^T Xh contracted over the R rows, db = sum_r c_r H_r, then one
// Adam update of W (and its bf16 shadow when Wb != nullptr) and of b; also
// finishes the loss scalar described by lf.  cs [R] or null (fp32 only): Xh
// rows are raw, x_hat_r = s_r * Xh_r, and cs_r = c_r * s_r is the factor the
// product applies to H row r (db still uses c).
hipError_t launch_dw_adam(int dtype, const float *H, const float *c, const void *Xh,
                          const float *cs, int M, int N, int K, float *W, float *mW, float *vW,
                          uint16_t *Wb, float *b, float *mb, float *vb, const AdamArgs &a,
                          const LossFinish &lf, hipStream_t s);

// Rows of the transposed bf16 weight-gradient operands: R rounded up to a
// multiple of 64 (the extra columns are zeros).
int padded_rows(int rows);

// Loss rows as launch_loss (g, c into g_out, c_out when non-null, loss
// partials lpart[loss_blocks(R)][2]) for a bf16 layer, plus its weight-gradient
// operand dZ^T = bf16(c . H)^T [D][padded_rows(R)] (R3) and the fp32 column
// sums of c . H over each 64-row block, dbp[loss_blocks(R)][D] (for db).
// xn, xnT (both or neither): also the next layer's bf16 operand from H, rows
// xn [R][D] = bf16(h_r / (sqrt(g_r) + norm_eps)) and xnT [D][padded_rows(R)].
// x, xT (both or neither): also the transpose xT [dx][padded_rows(R)] of the
// layer's bf16 input rows x [R][dx] (dx a multiple of 8), in the same launch.
hipError_t launch_loss_t(const float *gpart, int ntiles, int R, int n_pos, float theta,
                         const float *H, int D, float *g_out, float *c_out, float *lpart,
                         uint16_t *dzT, float *dbp, float norm_eps, uint16_t *xn, uint16_t *xnT,
                         const uint16_t *x, int dx, uint16_t *xT, hipStream_t s);

// bf16 weight gradient dW = dZ^T (xT)^T over padded_rows(R) rows (operands from
// launch_loss_t; M = d_out, N = d_in), with the Adam
// update of W, its shadow Wb and b (db from dbp) fused, and the loss scalar of lf.
// G non-null: dW is stored into G [M][N] instead and W, b are left for
// launch_adam_dense (the loss scalar is still finished).
hipError_t launch_dw4(const uint16_t *dzT, const uint16_t *xT, int M, int N, int R, float *G,
                      float *W, float *mW, float *vW, uint16_t *Wb, const float *dbp, float *b,
                      float *mb, float *vb, const AdamArgs &a, const LossFinish &lf,
                      hipStream_t s);

// Whether a bf16 training step of a d_out x d_in layer runs its Adam update as
// a launch of its own: when the product takes one 192x192 tile per CU (every
// CU would run the fused update after its product at the same time, while
// launch_adam_dense streams it near the HBM rate; 3072 x 3072 over 4096 rows:
// 67.5 + 45.2 us against 121.7 us).
bool dw4_split_adam(int M, int N);

// The Adam update launch_dw4 fuses, from a stored gradient: W, mW, vW, Wb
// [M][N] from G [M][N] (N a multiple of 4), and b, mb, vb [M] from the db
// partials dbp [loss_blocks(R)][M] of the R-row step.
hipError_t launch_adam_dense(const float *G, int M, int N, float *W, float *mW, float *vW,
                             uint16_t *Wb, const float *dbp, int R, float *b, float *mb,
                             float *vb, const AdamArgs &a, hipStream_t s);

// g_r = sum_t gpart[t][r] into g (any of the outputs may be null);
// out[r] = g_r (accumulate == 0) or out[r] += g_r (accumulate == 1);
// s_out[r] = 1/(sqrt(g_r) + norm_eps), the next layer's input normalisation.
hipError_t launch_goodness(const float *gpart, int ntiles, int R, float *g, float *out,
                           int accumulate, float *s_out, float norm_eps, hipStream_t s);

// pred[n] = argmax_c scores[n][c], lowest c on ties; with `exclude` (C >= 2),
// c == exclude[n] is skipped.
hipError_t launch_argmax(const float *scores, int n, int C, const int32_t *exclude, int32_t *pred,
                         hipStream_t s);

// Wb[i] = bf16(W[i]).
hipError_t launch_bf16_shadow(const float *W, uint16_t *Wb, size_t count, hipStream_t s);

}  // namespace ffk
