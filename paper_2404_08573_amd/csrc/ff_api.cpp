// Host side of the C ABI declared in include/ff.h: argument validation,
// workspace carving, launch sequencing, and the one-stream-per-layer pipeline
// scheduler (Single-Layer PFF, Sec. 4.1 / Alg. 1, emulated on one GPU).
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <vector>

#include "../../include/ff.h"
#include "ff_internal.h"

static_assert(FF_MAX_WIDTH == ffk::kMaxWidth, "one width limit");

namespace {

thread_local char g_msg[512] = "";

ff_status fail(ff_status st, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_msg, sizeof g_msg, fmt, ap);
  va_end(ap);
  return st;
}

#define FF_HIP(expr)                                                                   \
  do {                                                                                 \
    hipError_t e_ = (expr);                                                            \
    if (e_ != hipSuccess)                                                              \
      return fail(FF_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));          \
  } while (0)

#define FF_TRY(expr)                 \
  do {                               \
    ff_status s_ = (expr);           \
    if (s_ != FF_OK) return s_;      \
  } while (0)

constexpr size_t kAlign = 256;

// Carves aligned regions out of a workspace; with base == nullptr it only
// measures, so size queries and real carving share one code path.
struct Carver {
  char *base;
  size_t off = 0;
  explicit Carver(void *b) : base(static_cast<char *>(b)) {}
  void *take(size_t bytes) {
    off = (off + kAlign - 1) / kAlign * kAlign;
    void *p = base ? base + off : nullptr;
    off += bytes;
    return p;
  }
};

inline size_t elem_bytes(int dtype) { return dtype == FF_BF16 ? 2 : 4; }

// ---------------------------------------------------------------------------
// Kernel timing: event pairs around launches while a profile is active.
// ---------------------------------------------------------------------------
// Sizes of a launch, recorded with its timing (ff_launch_record).
struct Sizes {
  int32_t m = 0, n = 0, k = 0, aux = 0;
};
struct ProfRec {
  int kind;
  Sizes sz;
  double flops, bytes;
  hipEvent_t a, b;
};
struct Profiler {
  std::mutex mu;
  bool on = false;
  uint32_t mask = ~0u;  // kinds timed while on
  std::vector<hipEvent_t> pool;
  size_t used = 0;
  std::vector<ProfRec> recs;
};
Profiler g_prof;

// Test aid (ff_fail_next_launch): kernel kind whose next launch fails, or -1.
std::atomic<int> g_fail_kind{-1};

// Launches `fn` (returning hipError_t), bracketed by timing events when a
// profile is active and events remain.
template <class F>
hipError_t launch(int kind, Sizes sz, double flops, double bytes, hipStream_t st, F fn) {
  int armed = kind;
  if (g_fail_kind.load(std::memory_order_relaxed) == kind &&
      g_fail_kind.compare_exchange_strong(armed, -1))
    return hipErrorLaunchFailure;  // nothing enqueued
  std::unique_lock<std::mutex> lk(g_prof.mu);
  if (!g_prof.on || !((g_prof.mask >> kind) & 1u) || g_prof.used + 2 > g_prof.pool.size()) {
    lk.unlock();
    return fn();
  }
  hipEvent_t a = g_prof.pool[g_prof.used++], b = g_prof.pool[g_prof.used++];
  hipError_t e = hipEventRecord(a, st);
  if (e != hipSuccess) return e;
  e = fn();
  if (e != hipSuccess) return e;
  e = hipEventRecord(b, st);
  if (e == hipSuccess) g_prof.recs.push_back(ProfRec{kind, sz, flops, bytes, a, b});
  return e;
}

// Algorithmic work of the launches (what the operation must move or compute).
inline double gemm_flops(long m, long n, long k) { return 2.0 * m * n * k; }

// Scratch of one layer step.  Pointers the caller supplied are not carved.
struct StepScratch {
  void *xhat = nullptr;   // [rows][d_in], fp32 or bf16
  float *h = nullptr;     // [rows][d_out]
  float *gpart = nullptr; // [col tiles][rows]
  float *g = nullptr;     // [rows]
  float *c = nullptr;     // [rows]
  float *cs = nullptr;    // [rows] c times the input row scale (raw fp32 input rows)
  float *lpart = nullptr; // [loss blocks][2]
  float *loss = nullptr;  // [1]
  // Performance-optimised steps (po_classes > 0): the classifier's logit
  // gradient, per-row loss and weight-gradient partials, and the layer's dZ
  float *G = nullptr;     // [rows][C]
  float *lrow = nullptr;  // [rows]
  float *part = nullptr;  // [head_grad_splits(rows)][C][d_out]
  float *dz = nullptr;    // [rows][d_out]
  // bf16 FF training steps: the weight-gradient product's operands, row-major
  // over the rows padded to Rp = padded_rows(rows), and the db partials
  uint16_t *xt = nullptr;   // [d_in][Rp] x_hat^T
  uint16_t *dzt = nullptr;  // [d_out][Rp] bf16(c . H)^T
  float *dbp = nullptr;     // [Rp / 64][d_out]
  // bf16 FF training steps of an epoch: the weight gradient, stored for an
  // Adam launch of its own (which other streams' products can run beside)
  float *dw = nullptr;      // [d_out][d_in]
};

// train: the scratch of a training step (the bf16 weight-gradient operands);
// false for forward passes only.  split_adam: a bf16 training step also gets
// the weight-gradient buffer, and runs its Adam update as a launch of its own;
// it always does at the sizes where that is faster on one stream
// (ffk::dw4_split_adam).
void carve_step(Carver &cv, StepScratch &s, int rows, int d_in, int d_out, int dtype, bool need_h,
                bool need_g, bool need_loss, int po_classes = 0, bool train = true,
                bool split_adam = false) {
  if (po_classes > 0) {
    s.G = static_cast<float *>(cv.take((size_t)rows * po_classes * 4));
    s.lrow = static_cast<float *>(cv.take((size_t)rows * 4));
    s.part = static_cast<float *>(
        cv.take((size_t)ffk::head_grad_splits(rows) * po_classes * d_out * 4));
    s.dz = static_cast<float *>(cv.take((size_t)rows * d_out * 4));
  }
  s.xhat = cv.take((size_t)rows * d_in * elem_bytes(dtype));
  if (need_h) s.h = static_cast<float *>(cv.take((size_t)rows * d_out * 4));
  s.gpart = static_cast<float *>(cv.take((size_t)ffk::fwd_col_tiles_max(d_out) * rows * 4));
  if (need_g) s.g = static_cast<float *>(cv.take((size_t)rows * 4));
  s.c = static_cast<float *>(cv.take((size_t)rows * 4));
  s.cs = static_cast<float *>(cv.take((size_t)rows * 4));
  s.lpart = static_cast<float *>(cv.take((size_t)ffk::loss_blocks(rows) * 2 * 4));
  if (need_loss) s.loss = static_cast<float *>(cv.take(4));
  if (train && dtype == FF_BF16 && po_classes == 0 && d_in > 0) {
    const size_t rp = (size_t)ffk::padded_rows(rows);
    s.xt = static_cast<uint16_t *>(cv.take(rp * d_in * 2));
    s.dzt = static_cast<uint16_t *>(cv.take(rp * d_out * 2));
    s.dbp = static_cast<float *>(cv.take((size_t)ffk::loss_blocks(rows) * d_out * 4));
    if (split_adam || ffk::dw4_split_adam(d_out, d_in))
      s.dw = static_cast<float *>(cv.take((size_t)d_out * d_in * 4));
  }
}

size_t step_ws_bytes(int rows, int d_in, int d_out, int dtype, bool need_h) {
  Carver cv(nullptr);
  StepScratch s;
  carve_step(cv, s, rows, d_in, d_out, dtype, need_h, true, true);
  return cv.off + kAlign;
}

ff_status check_hp(const ff_hparams *hp) {
  if (!hp) return fail(FF_ERR_INVALID_ARG, "hp is NULL");
  if (hp->dtype != FF_F32 && hp->dtype != FF_BF16)
    return fail(FF_ERR_INVALID_ARG, "dtype %d is not FF_F32 or FF_BF16", hp->dtype);
  if (!(hp->norm_eps >= 0.f) || !(hp->adam_eps >= 0.f) || !(hp->lr >= 0.f) ||
      !(hp->beta1 >= 0.f && hp->beta1 < 1.f) || !(hp->beta2 >= 0.f && hp->beta2 < 1.f) ||
      !isfinite(hp->theta))
    return fail(FF_ERR_INVALID_ARG, "hyper-parameter out of range");
  return FF_OK;
}

ff_status check_layer(const ff_layer *L, const ff_hparams *hp, bool for_update, int idx) {
  if (!L) return fail(FF_ERR_INVALID_ARG, "layer %d is NULL", idx);
  if (L->d_in <= 0 || L->d_out <= 0)
    return fail(FF_ERR_INVALID_ARG, "layer %d: d_in=%d d_out=%d must be positive", idx, L->d_in,
                L->d_out);
  if (L->d_in % 4 || L->d_out % 4)
    return fail(FF_ERR_UNSUPPORTED, "layer %d: d_in=%d d_out=%d must be multiples of 4", idx,
                L->d_in, L->d_out);
  if (L->d_in > FF_MAX_WIDTH || L->d_out > FF_MAX_WIDTH)
    return fail(FF_ERR_UNSUPPORTED, "layer %d: d_in=%d d_out=%d exceed %d", idx, L->d_in,
                L->d_out, FF_MAX_WIDTH);
  if (!L->W || !L->b) return fail(FF_ERR_INVALID_ARG, "layer %d: W or b is NULL", idx);
  if (for_update && (!L->mW || !L->vW || !L->mb || !L->vb))
    return fail(FF_ERR_INVALID_ARG, "layer %d: Adam moment buffer is NULL", idx);
  if (hp && hp->dtype == FF_BF16 && !L->W_bf16)
    return fail(FF_ERR_INVALID_ARG, "layer %d: FF_BF16 needs the W_bf16 shadow", idx);
  if (hp && hp->dtype == FF_BF16 && L->d_in % 8)
    return fail(FF_ERR_UNSUPPORTED, "layer %d: FF_BF16 needs d_in=%d to be a multiple of 8", idx,
                L->d_in);
  return FF_OK;
}

ff_status check_stack(const ff_layer *layers, int n_layers, const ff_hparams *hp,
                      bool for_update) {
  if (!layers || n_layers <= 0) return fail(FF_ERR_INVALID_ARG, "no layers");
  for (int l = 0; l < n_layers; ++l) {
    FF_TRY(check_layer(&layers[l], hp, for_update, l));
    if (l > 0 && layers[l].d_in != layers[l - 1].d_out)
      return fail(FF_ERR_INVALID_ARG, "layer %d: d_in=%d does not match d_out=%d of layer %d", l,
                  layers[l].d_in, layers[l - 1].d_out, l - 1);
  }
  return FF_OK;
}

inline const void *weight_operand(const ff_layer *L, int dtype) {
  return dtype == FF_BF16 ? static_cast<const void *>(L->W_bf16) : static_cast<const void *>(L->W);
}

// Normalised operand rows for a layer: fp32 rows may be used in place when
// already normalised; otherwise (and always for bf16) the embed/normalise
// kernel writes them into scratch.
hipError_t embed_norm(const ffk::RowMap &src, int rows, int d, float eps, bool normalise,
                      bool bf16, void *out, hipStream_t st, float *scale_out = nullptr) {
  // unique source rows: a chunk's positives and negatives share base rows, and
  // label expansion reads each base row once per label
  const double src_rows = src.mode == ffk::PAIRS    ? (double)src.n_pos
                          : src.mode == ffk::EXPAND ? (double)rows / src.n_classes
                                                    : (double)rows;
  const double bytes = src_rows * d * 4.0 + (double)rows * d * (bf16 ? 2 : 4) +
                       (scale_out ? rows * 4.0 : 0.0);
  return launch(FF_KERNEL_EMBED_NORM, Sizes{rows, d, 0, src.mode | (bf16 ? 16 : 0)}, 0.0,
                bytes, st, [&] {
    return ffk::launch_embed_norm(src, rows, d, eps, normalise, bf16, out, scale_out, st);
  });
}

hipError_t fwd(int dtype, const void *X, const void *W, const float *bias, const float *rowscale,
               int M, int N, int K, float *H, float *gpart, hipStream_t st) {
  const double eb = (double)elem_bytes(dtype);
  const double nt = ffk::fwd_col_tiles(M, N, dtype);
  const double bytes = (double)M * K * eb + (double)N * K * eb + N * 4.0 +
                       (rowscale ? M * 4.0 : 0.0) + (H ? (double)M * N * 4.0 : 0.0) +
                       nt * M * 4.0;
  return launch(FF_KERNEL_FORWARD, Sizes{M, N, K, 0}, gemm_flops(M, N, K), bytes, st, [&] {
    return ffk::launch_fwd(dtype, X, W, bias, rowscale, M, N, K, H, gpart, st);
  });
}

// Shared-base layer-0 forward over M base rows expanded by ex (bytes: the
// base rows, W, the expanded H and partials).
hipError_t fwd_expand(int dtype, const void *X, const void *W, const float *bias,
                      const ffk::LabelExpand &ex, int M, int N, int K, float *H, float *gpart,
                      hipStream_t st) {
  const double eb = (double)elem_bytes(dtype);
  const double rows_out = (double)M * ex.n_classes;
  const double nt = ffk::fwd_expand_col_tiles(M, N, dtype);
  const double bytes = (double)M * K * eb + (double)N * K * eb + N * 4.0 + M * 4.0 +
                       (H ? rows_out * N * 4.0 : 0.0) + nt * rows_out * 4.0;
  return launch(FF_KERNEL_FORWARD, Sizes{M, N, K, ex.n_classes}, gemm_flops(M, N, K), bytes, st,
                [&] {
    return ffk::launch_fwd_expand(dtype, X, W, bias, ex, M, N, K, H, gpart, st);
  });
}

hipError_t goodness_sum(const float *gpart, int nt, int R, float *g, float *out, int accumulate,
                        float *s_out, float norm_eps, hipStream_t st) {
  const double bytes = (double)nt * R * 4.0 + (g ? R * 4.0 : 0.0) +
                       (out ? R * 4.0 * (accumulate ? 2 : 1) : 0.0) + (s_out ? R * 4.0 : 0.0);
  return launch(FF_KERNEL_GOODNESS, Sizes{R, nt, 0, 0}, 0.0, bytes, st, [&] {
    return ffk::launch_goodness(gpart, nt, R, g, out, accumulate, s_out, norm_eps, st);
  });
}

// Normalised operand rows for a layer: fp32 rows may be used in place when
// already normalised; otherwise (and always for bf16) the embed/normalise
// kernel writes them into scratch.
ff_status stage_input(const ffk::RowMap &src, int rows, int d_in, bool normalised, int dtype,
                      float norm_eps, void *scratch, const void **operand, hipStream_t st) {
  const bool bf16 = dtype == FF_BF16;
  if (normalised && !bf16 && src.mode == ffk::ROWS) {
    *operand = src.base;
    return FF_OK;
  }
  FF_HIP(embed_norm(src, rows, d_in, norm_eps, !normalised, bf16, scratch, st));
  *operand = scratch;
  return FF_OK;
}

// Input rows of a layer.  `rowscale` (fp32 only) marks raw hidden-activity rows
// (src.mode == ROWS) whose normalisation 1/(||x_r|| + eps) is already known
// (from the producing layer's goodness, the squared norm of the row): the
// products then take the raw rows and apply the scale themselves (the
// forward to its accumulators, dW to the rows it stages), and no normalised
// copy is written.
struct LayerInput {
  ffk::RowMap src{};
  bool normalised = false;
  const float *rowscale = nullptr;
  // bf16 steps: src.base holds the normalised bf16 operand rows [rows][d_in]
  // and xt their transpose [d_in][padded_rows(rows)], written by the previous
  // layer's loss pass (NextBf16)
  const uint16_t *xt = nullptr;
};

// Where a bf16 training step's loss pass writes the next layer's operand:
// normalised bf16 rows [rows][d_out] and their transpose [d_out][padded rows].
struct NextBf16 {
  uint16_t *rows = nullptr;
  uint16_t *xt = nullptr;
};

LayerInput raw_rows(const float *x, const float *rowscale) {
  LayerInput in;
  in.src.base = x;
  in.src.mode = ffk::ROWS;
  in.rowscale = rowscale;
  return in;
}

// Forward of one layer; `s_next` (optional) receives the output rows'
// normalisation for the next layer.
ff_status forward_core(const ff_layer *L, const ff_hparams *hp, const LayerInput &in, int rows,
                       float *h_out, float *goodness, float *s_next, StepScratch &s,
                       hipStream_t st) {
  const void *xop = in.src.base;
  if (!in.rowscale)
    FF_TRY(stage_input(in.src, rows, L->d_in, in.normalised, hp->dtype, hp->norm_eps, s.xhat,
                       &xop, st));
  FF_HIP(fwd(hp->dtype, xop, weight_operand(L, hp->dtype), L->b, in.rowscale, rows, L->d_out,
             L->d_in, h_out, s.gpart, st));
  if (goodness || s_next)
    FF_HIP(goodness_sum(s.gpart, ffk::fwd_col_tiles(rows, L->d_out, hp->dtype), rows, goodness,
                        nullptr, 0, s_next, hp->norm_eps, st));
  return FF_OK;
}

// Adam arguments of update t.
ffk::AdamArgs adam_args(const ff_hparams *hp, int64_t t) {
  ffk::AdamArgs a;
  a.lr = hp->lr;
  a.beta1 = hp->beta1;
  a.beta2 = hp->beta2;
  a.eps = hp->adam_eps;
  a.lr_bc1 = (float)((double)hp->lr / (1.0 - pow((double)hp->beta1, (double)t)));
  a.inv_bc2 = (float)(1.0 / (1.0 - pow((double)hp->beta2, (double)t)));
  return a;
}

// One training step (n_pos positives first); `s_next` as in forward_core.
// out_ready (optional) is recorded on st once the step's outputs for the next
// layer (h_out, s_next or nx) are written, before the weight update.
ff_status step_core(ff_layer *L, const ff_hparams *hp, const LayerInput &in, int n_pos,
                    int n_neg, float *h_out, float *goodness, float *loss, float *s_next,
                    StepScratch &s, hipStream_t st, const NextBf16 *nx = nullptr,
                    hipEvent_t out_ready = nullptr) {
  const int R = n_pos + n_neg;
  const void *xop = in.src.base;
  if ((in.xt || nx) && !(hp->dtype == FF_BF16 && s.dzt && !in.rowscale))
    return fail(FF_ERR_INVALID_ARG, "bf16 operand handoff outside a bf16 training step");
  if (!in.rowscale && !in.xt)
    FF_TRY(stage_input(in.src, R, L->d_in, in.normalised, hp->dtype, hp->norm_eps, s.xhat, &xop,
                       st));
  float *H = h_out ? h_out : s.h;
  float *g = goodness ? goodness : s.g;
  float *lo = loss ? loss : s.loss;
  const int nt = ffk::fwd_col_tiles(R, L->d_out, hp->dtype);
  FF_HIP(fwd(hp->dtype, xop, weight_operand(L, hp->dtype), L->b, in.rowscale, R, L->d_out,
             L->d_in, H, s.gpart, st));
  if (hp->dtype == FF_BF16 && s.dzt) {
    // bf16: the weight gradient as an NT product over the rows.  The loss pass
    // also writes bf16(c . H)^T and the db partials; x_hat^T is transposed from
    // the normalised bf16 rows.
    const int Rp = ffk::padded_rows(R), nrb = ffk::loss_blocks(R);
    const uint16_t *xh = static_cast<const uint16_t *>(xop);
    // without a handed-off transpose the same launch transposes the input rows
    const bool tr = !in.xt;
    FF_HIP(launch(FF_KERNEL_LOSS, Sizes{R, L->d_out, nt, 1 | (nx ? 2 : 0) | (tr ? 4 : 0)}, 0.0,
                  (double)nt * R * 4.0 + (double)R * L->d_out * 4.0 + (g ? R * 4.0 : 0.0) +
                      (double)Rp * L->d_out * 2.0 + (double)nrb * L->d_out * 4.0 +
                      (nx ? ((double)R + Rp) * L->d_out * 2.0 : 0.0) +
                      (tr ? ((double)R + Rp) * L->d_in * 2.0 : 0.0),
                  st, [&] {
                    return ffk::launch_loss_t(s.gpart, nt, R, n_pos, hp->theta, H, L->d_out, g,
                                              nullptr, s.lpart, s.dzt, s.dbp, hp->norm_eps,
                                              nx ? nx->rows : nullptr, nx ? nx->xt : nullptr,
                                              tr ? xh : nullptr, L->d_in, tr ? s.xt : nullptr,
                                              st);
                  }));
    if (out_ready) FF_HIP(hipEventRecord(out_ready, st));
    const uint16_t *xT = in.xt ? in.xt : s.xt;
    ffk::LossFinish lf;
    lf.lpart = s.lpart;
    lf.nblk = nrb;
    lf.n_pos = n_pos;
    lf.n_neg = n_neg;
    lf.loss = lo;
    const int64_t t = L->step + 1;
    const ffk::AdamArgs a = adam_args(hp, t);
    const double params = (double)L->d_out * L->d_in;
    const double operands = (double)Rp * (L->d_out + L->d_in) * 2.0;
    const double adam = params * 24.0 + params * 2.0 + (double)nrb * L->d_out * 4.0 +
                        L->d_out * 24.0;  // W, m, v in and out, Wb out, b
    // split: the product stores dW, then the Adam launch reads it back
    const double bytes = s.dw ? operands + params * 4.0 : operands + adam;
    FF_HIP(launch(FF_KERNEL_DW_ADAM, Sizes{L->d_out, L->d_in, R, s.dw ? 1 : 0},
                  gemm_flops(L->d_out, L->d_in, R), bytes, st, [&] {
      return ffk::launch_dw4(s.dzt, xT, L->d_out, L->d_in, R, s.dw, L->W, L->mW, L->vW,
                             L->W_bf16, s.dbp, L->b, L->mb, L->vb, a, lf, st);
    }));
    if (s.dw)
      FF_HIP(launch(FF_KERNEL_ADAM, Sizes{L->d_out, L->d_in, R, 0}, 0.0, params * 4.0 + adam, st,
                    [&] {
                      return ffk::launch_adam_dense(s.dw, L->d_out, L->d_in, L->W, L->mW, L->vW,
                                                    L->W_bf16, s.dbp, R, L->b, L->mb, L->vb, a,
                                                    st);
                    }));
    L->step = t;
    return FF_OK;
  }
  float *cs = in.rowscale ? s.cs : nullptr;
  FF_HIP(launch(FF_KERNEL_LOSS, Sizes{R, L->d_out, nt, 0}, 0.0,
                (double)nt * R * 4.0 + R * (g ? 8.0 : 4.0) + (s_next ? R * 4.0 : 0.0) +
                    (cs ? R * 8.0 : 0.0),
                st, [&] {
                  return ffk::launch_loss(s.gpart, nt, R, n_pos, hp->theta, g, s.c, s.lpart,
                                          s_next, hp->norm_eps, in.rowscale, cs, st);
                }));
  if (out_ready) FF_HIP(hipEventRecord(out_ready, st));
  ffk::LossFinish lf;
  lf.lpart = s.lpart;
  lf.nblk = ffk::loss_blocks(R);
  lf.n_pos = n_pos;
  lf.n_neg = n_neg;
  lf.loss = lo;
  // the update is t = step + 1; the count moves only once its launch is enqueued
  const int64_t t = L->step + 1;
  const ffk::AdamArgs a = adam_args(hp, t);
  {
    const double eb = (double)elem_bytes(hp->dtype);
    const double params = (double)L->d_out * L->d_in;
    const double bytes = (double)R * L->d_out * 4.0 + (double)R * L->d_in * eb +
                         R * (in.rowscale ? 8.0 : 4.0) +
                         params * (24.0 + (hp->dtype == FF_BF16 ? 2.0 : 0.0)) + L->d_out * 24.0;
    FF_HIP(launch(FF_KERNEL_DW_ADAM, Sizes{L->d_out, L->d_in, R, 0},
                  gemm_flops(L->d_out, L->d_in, R), bytes, st, [&] {
      return ffk::launch_dw_adam(hp->dtype, H, s.c, xop, cs, L->d_out, L->d_in, R, L->W,
                                 L->mW, L->vW, hp->dtype == FF_BF16 ? L->W_bf16 : nullptr, L->b,
                                 L->mb, L->vb, a, lf, st);
    }));
  }
  L->step = t;
  return FF_OK;
}

// One performance-optimised step (R rows, labels): the layer and its softmax
// classifier trained together by backprop through the two, no negatives.
// out_ready (optional) is recorded on st once h_out and s_next are written,
// right after the forward: the rest of the step only reads them.
ff_status po_step_core(ff_layer *L, ff_head *head, const ff_hparams *hp, const ff_hparams *head_hp,
                       const LayerInput &in, int R, const int32_t *labels, float *h_out,
                       float *loss, float *s_next, StepScratch &s, hipStream_t st,
                       hipEvent_t out_ready = nullptr) {
  const int C = head->n_classes, D = L->d_out;
  const void *xop = in.src.base;
  if (!in.rowscale)
    FF_TRY(stage_input(in.src, R, L->d_in, in.normalised, hp->dtype, hp->norm_eps, s.xhat, &xop,
                       st));
  float *H = h_out ? h_out : s.h;
  FF_HIP(fwd(hp->dtype, xop, weight_operand(L, hp->dtype), L->b, in.rowscale, R, D, L->d_in, H,
             s.gpart, st));
  if (s_next)
    FF_HIP(goodness_sum(s.gpart, ffk::fwd_col_tiles(R, D, hp->dtype), R, nullptr, nullptr, 0,
                        s_next, hp->norm_eps, st));
  if (out_ready) FF_HIP(hipEventRecord(out_ready, st));
  ffk::HeadFeatures f{};
  f.n_blocks = 1;
  f.h[0] = H;
  f.d[0] = D;
  f.w[0] = head->W;
  f.ldw[0] = D;
  f.n_bias = 1;
  f.bias[0] = head->b;
  const int splits = ffk::head_grad_splits(R);
  const double hbytes = (double)R * D * 4.0;
  FF_HIP(launch(FF_KERNEL_HEAD, Sizes{R, C, D, 1}, 2.0 * R * C * D,
                hbytes + (double)C * D * 4.0 + R * C * 8.0, st,
                [&] {
                  return ffk::launch_head_logits(f, R, C, labels, nullptr, nullptr, s.G, s.lrow,
                                                 st);
                }));
  FF_HIP(launch(FF_KERNEL_HEAD, Sizes{R, C, D, 2}, 2.0 * R * C * D,
                2.0 * hbytes + (double)C * D * 4.0, st, [&] {
    return ffk::launch_po_dz(H, s.G, head->W, R, D, C, s.dz, s.c, st);
  }));
  FF_HIP(launch(FF_KERNEL_HEAD, Sizes{R, C, D, 3}, 2.0 * R * C * D,
                hbytes + (double)splits * C * D * 4.0, st, [&] {
    return ffk::launch_head_grad(f, s.G, R, C, D, splits, s.part, st);
  }));
  const ffk::AdamArgs ah = adam_args(head_hp, head->step + 1);
  FF_HIP(launch(FF_KERNEL_HEAD, Sizes{R, C, D, 4}, 0.0,
                (double)splits * C * D * 4.0 + (double)C * D * 24.0, st, [&] {
                  return ffk::launch_head_adam(s.part, splits, s.G, s.lrow, R, C, D, head->W,
                                               head->mW, head->vW, head->b, head->mb, head->vb,
                                               ah, loss ? loss : s.loss, st);
                }));
  ++head->step;
  // dW = dZ^T x_hat, db = sum dZ: the weight-gradient product with row scale
  // c = 1, so with raw input rows the product's factor c * s is the input row
  // scale s itself
  const ffk::AdamArgs a = adam_args(hp, L->step + 1);
  ffk::LossFinish lf{};
  const double eb = (double)elem_bytes(hp->dtype);
  const double params = (double)D * L->d_in;
  const double bytes = hbytes + (double)R * L->d_in * eb + R * (in.rowscale ? 8.0 : 4.0) +
                       params * (24.0 + (hp->dtype == FF_BF16 ? 2.0 : 0.0)) + D * 24.0;
  FF_HIP(launch(FF_KERNEL_DW_ADAM, Sizes{D, L->d_in, R, 0}, gemm_flops(D, L->d_in, R), bytes,
                st, [&] {
    return ffk::launch_dw_adam(hp->dtype, s.dz, s.c, xop, in.rowscale, D, L->d_in, R, L->W,
                               L->mW, L->vW, hp->dtype == FF_BF16 ? L->W_bf16 : nullptr, L->b,
                               L->mb, L->vb, a, lf, st);
  }));
  ++L->step;
  return FF_OK;
}

ff_status check_ws(void *ws, size_t ws_bytes, size_t need) {
  if (!ws) return fail(FF_ERR_WORKSPACE, "workspace is NULL (needs %zu bytes)", need);
  if ((reinterpret_cast<uintptr_t>(ws) % kAlign) != 0)
    return fail(FF_ERR_WORKSPACE, "workspace must be %zu-byte aligned", kAlign);
  if (ws_bytes < need)
    return fail(FF_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  return FF_OK;
}

ffk::RowMap rows_of(const float *x) {
  ffk::RowMap m{};
  m.base = x;
  m.mode = ffk::ROWS;
  return m;
}

constexpr int kScoreBlockImages = 8192;  // images per scoring pass (rows = images * classes)

}  // namespace

extern "C" {

const char *ff_status_string(int32_t status) {
  switch (status) {
    case FF_OK: return "FF_OK";
    case FF_ERR_INVALID_ARG: return "FF_ERR_INVALID_ARG";
    case FF_ERR_UNSUPPORTED: return "FF_ERR_UNSUPPORTED";
    case FF_ERR_WORKSPACE: return "FF_ERR_WORKSPACE";
    case FF_ERR_HIP: return "FF_ERR_HIP";
    default: return "FF_UNKNOWN_STATUS";
  }
}

const char *ff_last_error(void) { return g_msg; }

ff_status ff_embed_labels(const float *x_base, const int32_t *labels, int32_t rows, int32_t d,
                          int32_t n_classes, float *out, void *stream) {
  if (rows < 0 || d <= 0 || n_classes <= 0) return fail(FF_ERR_INVALID_ARG, "bad sizes");
  if (d % 4) return fail(FF_ERR_UNSUPPORTED, "d=%d must be a multiple of 4", d);
  if (n_classes > d) return fail(FF_ERR_INVALID_ARG, "n_classes=%d exceeds d=%d", n_classes, d);
  if (rows == 0) return FF_OK;
  if (!x_base || !labels || !out) return fail(FF_ERR_INVALID_ARG, "NULL pointer");
  ffk::RowMap m{};
  m.base = x_base;
  m.lab_a = labels;
  m.lab_b = labels;
  m.mode = ffk::PAIRS;
  m.n_pos = rows;
  m.base_off = 0;
  m.n_classes = n_classes;
  FF_HIP(embed_norm(m, rows, d, 0.f, false, false, out, static_cast<hipStream_t>(stream)));
  return FF_OK;
}

size_t ff_step_workspace_size(int32_t rows, int32_t d_in, int32_t d_out, int32_t dtype) {
  if (rows <= 0 || d_in <= 0 || d_out <= 0) return 0;
  return step_ws_bytes(rows, d_in, d_out, dtype, true);
}

ff_status ff_layer_forward(const ff_layer *L, const ff_hparams *hp, const float *x, int32_t rows,
                           int32_t x_normalised, float *h_out, float *goodness, void *ws,
                           size_t ws_bytes, void *stream) {
  FF_TRY(check_hp(hp));
  FF_TRY(check_layer(L, hp, false, 0));
  if (rows < 0) return fail(FF_ERR_INVALID_ARG, "rows=%d", rows);
  if (rows == 0) return FF_OK;
  if (!x) return fail(FF_ERR_INVALID_ARG, "x is NULL");
  FF_TRY(check_ws(ws, ws_bytes, step_ws_bytes(rows, L->d_in, L->d_out, hp->dtype, true)));
  Carver cv(ws);
  StepScratch s;
  carve_step(cv, s, rows, L->d_in, L->d_out, hp->dtype, true, true, true);
  LayerInput in;
  in.src = rows_of(x);
  in.normalised = x_normalised != 0;
  return forward_core(L, hp, in, rows, h_out, goodness, nullptr, s,
                      static_cast<hipStream_t>(stream));
}

ff_status ff_layer_step(ff_layer *L, const ff_hparams *hp, const float *x, int32_t n_pos,
                        int32_t n_neg, int32_t x_normalised, float *h_out, float *goodness,
                        float *loss, void *ws, size_t ws_bytes, void *stream) {
  FF_TRY(check_hp(hp));
  FF_TRY(check_layer(L, hp, true, 0));
  if (n_pos < 1 || n_neg < 1)
    return fail(FF_ERR_INVALID_ARG, "n_pos=%d n_neg=%d: both halves need at least one row",
                n_pos, n_neg);
  if (!x) return fail(FF_ERR_INVALID_ARG, "x is NULL");
  const int R = n_pos + n_neg;
  FF_TRY(check_ws(ws, ws_bytes, step_ws_bytes(R, L->d_in, L->d_out, hp->dtype, true)));
  Carver cv(ws);
  StepScratch s;
  carve_step(cv, s, R, L->d_in, L->d_out, hp->dtype, true, true, true);
  LayerInput in;
  in.src = rows_of(x);
  in.normalised = x_normalised != 0;
  return step_core(L, hp, in, n_pos, n_neg, h_out, goodness, loss, nullptr, s,
                   static_cast<hipStream_t>(stream));
}

}  // extern "C"

// ---------------------------------------------------------------------------
// The no-allocation step: its scratch is this file-scope device array (each
// GPU holds its own copy).  In host code `scratch` only names the symbol; its
// device address, per device, comes from hipGetSymbolAddress.
// ---------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[FF_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device, looked up on the first
// call made with that device current and kept.
ff_status scratch_of_current_device(void **out) {
  int dev = -1;
  FF_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(FF_ERR_UNSUPPORTED, "device %d: the no-allocation scratch table holds %d devices",
                dev, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    FF_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(FF_ERR_HIP, "hipGetSymbolAddress gave no address for the scratch");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return FF_OK;
}
}  // namespace

extern "C" {

ff_status ff_layer_step_noalloc(ff_layer *L, const ff_hparams *hp, const float *x, int32_t n_pos,
                                int32_t n_neg, int32_t x_normalised, float *h_out,
                                float *goodness, float *loss, void *stream) {
  FF_TRY(check_hp(hp));
  FF_TRY(check_layer(L, hp, true, 0));
  if (n_pos < 1 || n_neg < 1)
    return fail(FF_ERR_INVALID_ARG, "n_pos=%d n_neg=%d: both halves need at least one row",
                n_pos, n_neg);
  if (!x) return fail(FF_ERR_INVALID_ARG, "x is NULL");
  const int R = n_pos + n_neg;
  // scratch for what the caller does not receive: the activities only when
  // h_out is NULL, the goodness and loss only when not passed
  Carver size_cv(nullptr);
  StepScratch tmp;
  carve_step(size_cv, tmp, R, L->d_in, L->d_out, hp->dtype, !h_out, !goodness, !loss);
  const size_t need = size_cv.off;
  if (need > (size_t)FF_NOALLOC_SCRATCH_BYTES)
    return fail(FF_ERR_UNSUPPORTED,
                "%d rows of %d -> %d need %zu bytes of scratch; the no-allocation step holds %zu "
                "(pass h_out, or use ff_layer_step with a workspace)",
                R, L->d_in, L->d_out, need, (size_t)FF_NOALLOC_SCRATCH_BYTES);
  void *base = nullptr;
  FF_TRY(scratch_of_current_device(&base));
  Carver cv(base);
  StepScratch s;
  carve_step(cv, s, R, L->d_in, L->d_out, hp->dtype, !h_out, !goodness, !loss);
  LayerInput in;
  in.src = rows_of(x);
  in.normalised = x_normalised != 0;
  return step_core(L, hp, in, n_pos, n_neg, h_out, goodness, loss, nullptr, s,
                   static_cast<hipStream_t>(stream));
}

ff_status ff_refresh_bf16_shadow(const ff_layer *L, void *stream) {
  FF_TRY(check_layer(L, nullptr, false, 0));
  if (!L->W_bf16) return fail(FF_ERR_INVALID_ARG, "W_bf16 is NULL");
  const size_t count = (size_t)L->d_out * L->d_in;
  hipStream_t st = static_cast<hipStream_t>(stream);
  FF_HIP(launch(FF_KERNEL_SHADOW, Sizes{L->d_out, L->d_in, 0, 0}, 0.0, count * 6.0, st,
                [&] { return ffk::launch_bf16_shadow(L->W, L->W_bf16, count, st); }));
  return FF_OK;
}

// ---------------------------------------------------------------------------
// Goodness prediction
// ---------------------------------------------------------------------------
namespace {
// fp32: layer 0 takes normalised rows from x; layer l > 0 takes the raw rows
// h[(l-1) % 2] with their normalisation rs (written by layer l-1's goodness
// pass).  bf16: every layer's input is normalised into x (bf16), and h[0]
// holds each layer's output.
// With the shared-base layer 0 (n_classes <= kMaxExpand), x first holds the
// normalised masked base rows [images][d_in of layer 0] and ls their scale.
struct ScoreScratch {
  void *x = nullptr;              // [rows][d_in of layer 0] fp32, or [rows][max d_in] bf16
  float *ls = nullptr;            // [images] shared-base scale
  float *h[2] = {nullptr, nullptr};  // [rows][max d_out]; h[1] for fp32 stacks of 3+ layers
  float *rs = nullptr;            // [rows] fp32
  float *gpart = nullptr;         // [max col tiles][rows]
  float *scores = nullptr;        // [n][C] when the caller passes none
};

void carve_score(Carver &cv, ScoreScratch &s, const ff_layer *layers, int n_layers, int n, int C,
                 int dtype, bool need_scores) {
  const int nb = std::min(n, kScoreBlockImages);
  const size_t rows = (size_t)nb * C;
  int max_in = 0, max_out = 0, max_nt = 0;
  for (int l = 0; l < n_layers; ++l) {
    max_in = std::max(max_in, layers[l].d_in);
    max_out = std::max(max_out, layers[l].d_out);
    max_nt = std::max(max_nt, ffk::fwd_col_tiles_max(layers[l].d_out));
  }
  const bool bf16 = dtype == FF_BF16;
  const bool shared = C <= ffk::kMaxExpand;
  const size_t x_rows = bf16 && n_layers > 1 ? rows : (shared ? (size_t)nb : rows);
  s.x = cv.take(x_rows * (bf16 ? max_in : layers[0].d_in) * elem_bytes(dtype));
  if (shared) s.ls = static_cast<float *>(cv.take((size_t)nb * 4));
  if (n_layers > 1) s.h[0] = static_cast<float *>(cv.take(rows * max_out * 4));
  if (n_layers > 2 && !bf16) s.h[1] = static_cast<float *>(cv.take(rows * max_out * 4));
  if (n_layers > 1 && !bf16) s.rs = static_cast<float *>(cv.take(rows * 4));
  s.gpart = static_cast<float *>(cv.take((size_t)max_nt * rows * 4));
  if (need_scores) s.scores = static_cast<float *>(cv.take((size_t)n * C * 4));
}
}  // namespace

size_t ff_score_workspace_size(const ff_layer *layers, int32_t n_layers, int32_t n,
                               int32_t n_classes, int32_t dtype) {
  if (!layers || n_layers <= 0 || n <= 0 || n_classes <= 0) return 0;
  Carver cv(nullptr);
  ScoreScratch s;
  carve_score(cv, s, layers, n_layers, n, n_classes, dtype, true);
  return cv.off + kAlign;
}

namespace {
ff_status check_score_args(const ff_layer *layers, int32_t n_layers, int32_t first_scored_layer,
                           const ff_hparams *hp, int32_t n, int32_t n_classes) {
  FF_TRY(check_hp(hp));
  FF_TRY(check_stack(layers, n_layers, hp, false));
  if (first_scored_layer < 0 || first_scored_layer >= n_layers)
    return fail(FF_ERR_INVALID_ARG, "first_scored_layer=%d outside [0, %d)", first_scored_layer,
                n_layers);
  if (n < 0 || n_classes <= 0) return fail(FF_ERR_INVALID_ARG, "n=%d n_classes=%d", n, n_classes);
  if (n_classes > layers[0].d_in)
    return fail(FF_ERR_INVALID_ARG, "n_classes=%d exceeds d_in=%d", n_classes, layers[0].d_in);
  if ((int64_t)n * n_classes > INT32_MAX) return fail(FF_ERR_UNSUPPORTED, "n too large");
  return FF_OK;
}

// Scores every input under every label into S, then takes the argmax
// (skipping exclude[i] when exclude is given); arguments already checked.
ff_status score_run(const ff_layer *layers, int32_t n_layers, int32_t first_scored_layer,
                    const ff_hparams *hp, const float *x_base, int32_t n, int32_t n_classes,
                    const int32_t *exclude, float *S, int32_t *pred, ScoreScratch &s,
                    hipStream_t st) {
  const bool bf16 = hp->dtype == FF_BF16;
  for (int n0 = 0; n0 < n; n0 += kScoreBlockImages) {
    const int nb = std::min(kScoreBlockImages, n - n0);
    const int rows = nb * n_classes;
    const bool shared = n_classes <= ffk::kMaxExpand;
    ffk::RowMap m{};
    m.base = x_base;
    m.mode = shared ? ffk::MASKED : ffk::EXPAND;
    m.base_off = n0;
    m.n_classes = n_classes;
    FF_HIP(embed_norm(m, shared ? nb : rows, layers[0].d_in, hp->norm_eps, true, bf16, s.x, st,
                      shared ? s.ls : nullptr));
    for (int l = 0; l < n_layers; ++l) {
      const ff_layer *L = &layers[l];
      const bool last = l + 1 == n_layers;
      const bool raw = l > 0 && !bf16;
      const void *X = raw ? s.h[(l - 1) & 1] : s.x;
      float *H = last ? nullptr : s.h[bf16 ? 0 : (l & 1)];
      int nt = ffk::fwd_col_tiles(rows, L->d_out, hp->dtype);
      if (l == 0 && shared) {
        ffk::LabelExpand ex{};
        ex.n_classes = n_classes;
        ex.scale = s.ls;
        FF_HIP(fwd_expand(hp->dtype, X, weight_operand(L, hp->dtype), L->b, ex, nb, L->d_out,
                          L->d_in, H, s.gpart, st));
        nt = ffk::fwd_expand_col_tiles(nb, L->d_out, hp->dtype);
      } else {
        FF_HIP(fwd(hp->dtype, X, weight_operand(L, hp->dtype), L->b, raw ? s.rs : nullptr, rows,
                   L->d_out, L->d_in, H, s.gpart, st));
      }
      const bool scored = l >= first_scored_layer;
      float *s_next = !last && !bf16 ? s.rs : nullptr;
      if (scored || s_next)
        FF_HIP(goodness_sum(s.gpart, nt, rows, nullptr,
                            scored ? S + (size_t)n0 * n_classes : nullptr,
                            l > first_scored_layer ? 1 : 0, s_next, hp->norm_eps, st));
      if (!last && bf16)
        FF_HIP(embed_norm(rows_of(H), rows, L->d_out, hp->norm_eps, true, true, s.x, st));
    }
  }
  FF_HIP(launch(FF_KERNEL_ARGMAX, Sizes{n, n_classes, 0, 0}, 0.0,
                (double)n * n_classes * 4.0 + n * 4.0, st,
                [&] { return ffk::launch_argmax(S, n, n_classes, exclude, pred, st); }));
  return FF_OK;
}

ff_status score_core(const ff_layer *layers, int32_t n_layers, int32_t first_scored_layer,
                     const ff_hparams *hp, const float *x_base, int32_t n, int32_t n_classes,
                     const int32_t *exclude, float *scores, int32_t *pred, void *ws,
                     size_t ws_bytes, void *stream) {
  FF_TRY(check_score_args(layers, n_layers, first_scored_layer, hp, n, n_classes));
  if (n == 0) return FF_OK;
  if (!x_base || !pred) return fail(FF_ERR_INVALID_ARG, "x_base or the output labels are NULL");
  Carver size_cv(nullptr);
  ScoreScratch tmp;
  carve_score(size_cv, tmp, layers, n_layers, n, n_classes, hp->dtype, scores == nullptr);
  FF_TRY(check_ws(ws, ws_bytes, size_cv.off + kAlign));
  Carver cv(ws);
  ScoreScratch s;
  carve_score(cv, s, layers, n_layers, n, n_classes, hp->dtype, scores == nullptr);
  return score_run(layers, n_layers, first_scored_layer, hp, x_base, n, n_classes, exclude,
                   scores ? scores : s.scores, pred, s, static_cast<hipStream_t>(stream));
}
}  // namespace

ff_status ff_score_labels(const ff_layer *layers, int32_t n_layers, int32_t first_scored_layer,
                          const ff_hparams *hp, const float *x_base, int32_t n, int32_t n_classes,
                          float *scores, int32_t *pred, void *ws, size_t ws_bytes, void *stream) {
  return score_core(layers, n_layers, first_scored_layer, hp, x_base, n, n_classes, nullptr,
                    scores, pred, ws, ws_bytes, stream);
}

ff_status ff_adaptive_negatives(const ff_layer *layers, int32_t n_layers,
                                int32_t first_scored_layer, const ff_hparams *hp,
                                const float *x_base, const int32_t *labels, int32_t n,
                                int32_t n_classes, float *scores, int32_t *y_neg, void *ws,
                                size_t ws_bytes, void *stream) {
  if (n > 0 && !labels) return fail(FF_ERR_INVALID_ARG, "labels is NULL");
  if (n_classes < 2) return fail(FF_ERR_INVALID_ARG, "n_classes=%d: no wrong label", n_classes);
  return score_core(layers, n_layers, first_scored_layer, hp, x_base, n, n_classes, labels,
                    scores, y_neg, ws, ws_bytes, stream);
}

// ---------------------------------------------------------------------------
// Softmax prediction layer
// ---------------------------------------------------------------------------
namespace {
// Every layer's activities for the n inputs and their row normalisation (the
// normalisation of layer l's output is both layer l+1's input scale, in fp32,
// and the scale of the head's feature block l).
struct HeadScratch {
  void *x0 = nullptr;           // [n][d_in of layer 0] normalised neutral rows
  void *xb = nullptr;           // bf16: [n][max hidden d_in] normalised bf16 rows
  std::vector<float *> h, s;    // [l]: [n][d_out_l], [n]
  float *gpart = nullptr;       // [max col tiles][n]
  float *G = nullptr;           // [n][C]
  float *lrow = nullptr;        // [n]
  float *part = nullptr;        // [splits][C][d_feat]
  float *loss = nullptr;        // [1]
};

int head_feat_width(const ff_layer *layers, int n_layers, int first) {
  int d = 0;
  for (int l = first; l < n_layers; ++l) d += layers[l].d_out;
  return d;
}

void carve_head(Carver &cv, HeadScratch &hs, const ff_layer *layers, int L, int first, int n,
                int C, int dtype) {
  const bool bf16 = dtype == FF_BF16;
  hs.x0 = cv.take((size_t)n * layers[0].d_in * elem_bytes(dtype));
  int max_hidden_in = 0, max_nt = 0;
  for (int l = 0; l < L; ++l) {
    if (l > 0) max_hidden_in = std::max(max_hidden_in, layers[l].d_in);
    max_nt = std::max(max_nt, ffk::fwd_col_tiles_max(layers[l].d_out));
  }
  if (bf16 && L > 1) hs.xb = cv.take((size_t)n * max_hidden_in * 2);
  hs.h.assign(L, nullptr);
  hs.s.assign(L, nullptr);
  for (int l = 0; l < L; ++l) {
    hs.h[l] = static_cast<float *>(cv.take((size_t)n * layers[l].d_out * 4));
    hs.s[l] = static_cast<float *>(cv.take((size_t)n * 4));
  }
  hs.gpart = static_cast<float *>(cv.take((size_t)max_nt * n * 4));
  hs.G = static_cast<float *>(cv.take((size_t)n * C * 4));
  hs.lrow = static_cast<float *>(cv.take((size_t)n * 4));
  hs.part = static_cast<float *>(cv.take((size_t)ffk::head_grad_splits(n) * C *
                                         head_feat_width(layers, L, first) * 4));
  hs.loss = static_cast<float *>(cv.take(4));
}

ff_status check_head(const ff_layer *layers, int n_layers, int first, const ff_hparams *hp,
                     const ff_head *head, bool for_update) {
  FF_TRY(check_hp(hp));
  FF_TRY(check_stack(layers, n_layers, hp, false));
  if (first < 0 || first >= n_layers)
    return fail(FF_ERR_INVALID_ARG, "first_layer=%d outside [0, %d)", first, n_layers);
  if (n_layers - first > ffk::kHeadMaxBlocks)
    return fail(FF_ERR_UNSUPPORTED, "%d layers feed the softmax layer (at most %d)",
                n_layers - first, ffk::kHeadMaxBlocks);
  if (!head) return fail(FF_ERR_INVALID_ARG, "head is NULL");
  if (head->d_feat != head_feat_width(layers, n_layers, first))
    return fail(FF_ERR_INVALID_ARG, "head d_feat=%d, but layers %d.. give %d features",
                head->d_feat, first, head_feat_width(layers, n_layers, first));
  if (head->n_classes < 2 || head->n_classes > ffk::kHeadMaxClasses ||
      head->n_classes > layers[0].d_in)
    return fail(FF_ERR_INVALID_ARG, "head n_classes=%d outside [2, %d] or above d_in",
                head->n_classes, ffk::kHeadMaxClasses);
  if (!head->W || !head->b) return fail(FF_ERR_INVALID_ARG, "head W or b is NULL");
  if (for_update && (!head->mW || !head->vW || !head->mb || !head->vb))
    return fail(FF_ERR_INVALID_ARG, "head Adam moment buffer is NULL");
  return FF_OK;
}

// The neutral pass through the FF layers; returns the head's feature blocks.
ff_status head_features(const ff_layer *layers, int L, int first, const ff_hparams *hp,
                        const float *x_base, int n, int C, HeadScratch &hs, hipStream_t st,
                        ffk::HeadFeatures &f) {
  const bool bf16 = hp->dtype == FF_BF16;
  ffk::RowMap m{};
  m.base = x_base;
  m.mode = ffk::NEUTRAL;
  m.n_classes = C;
  FF_HIP(embed_norm(m, n, layers[0].d_in, hp->norm_eps, true, bf16, hs.x0, st));
  for (int l = 0; l < L; ++l) {
    const ff_layer *Ly = &layers[l];
    const void *X = hs.x0;
    const float *rs = nullptr;
    if (l > 0 && bf16) {
      FF_HIP(embed_norm(rows_of(hs.h[l - 1]), n, Ly->d_in, hp->norm_eps, true, true, hs.xb, st));
      X = hs.xb;
    } else if (l > 0) {
      X = hs.h[l - 1];
      rs = hs.s[l - 1];
    }
    FF_HIP(fwd(hp->dtype, X, weight_operand(Ly, hp->dtype), Ly->b, rs, n, Ly->d_out, Ly->d_in,
               hs.h[l], hs.gpart, st));
    FF_HIP(goodness_sum(hs.gpart, ffk::fwd_col_tiles(n, Ly->d_out, hp->dtype), n, nullptr,
                        nullptr, 0, hs.s[l], hp->norm_eps, st));
  }
  f = ffk::HeadFeatures{};
  f.n_blocks = L - first;
  for (int l = first; l < L; ++l) {
    f.h[l - first] = hs.h[l];
    f.s[l - first] = hs.s[l];
    f.d[l - first] = layers[l].d_out;
  }
  return FF_OK;
}

// The head's weights as per-block views of W [C][D] (row stride D), one bias.
void head_weights(ffk::HeadFeatures &f, const float *W, const float *b, int D) {
  int off = 0;
  for (int i = 0; i < f.n_blocks; ++i) {
    f.w[i] = W + off;
    f.ldw[i] = D;
    off += f.d[i];
  }
  f.n_bias = 1;
  f.bias[0] = b;
}

ff_status head_prepare(const ff_layer *layers, int L, int first, const ff_hparams *hp,
                       const ff_head *head, int n, void *ws, size_t ws_bytes, HeadScratch &hs) {
  Carver size_cv(nullptr);
  HeadScratch tmp;
  carve_head(size_cv, tmp, layers, L, first, n, head->n_classes, hp->dtype);
  FF_TRY(check_ws(ws, ws_bytes, size_cv.off + kAlign));
  Carver cv(ws);
  carve_head(cv, hs, layers, L, first, n, head->n_classes, hp->dtype);
  return FF_OK;
}
}  // namespace

size_t ff_head_workspace_size(const ff_layer *layers, int32_t n_layers, int32_t first_layer,
                              int32_t n, int32_t n_classes, int32_t dtype) {
  if (!layers || n_layers <= 0 || first_layer < 0 || first_layer >= n_layers || n <= 0 ||
      n_classes <= 0)
    return 0;
  Carver cv(nullptr);
  HeadScratch hs;
  carve_head(cv, hs, layers, n_layers, first_layer, n, n_classes, dtype);
  return cv.off + kAlign;
}

ff_status ff_head_step(const ff_layer *layers, int32_t n_layers, int32_t first_layer,
                       const ff_hparams *hp, ff_head *head, const ff_hparams *head_hp,
                       const float *x_base, const int32_t *labels, int32_t n, float *loss,
                       void *ws, size_t ws_bytes, void *stream) {
  FF_TRY(check_head(layers, n_layers, first_layer, hp, head, true));
  FF_TRY(check_hp(head_hp));
  if (n < 0) return fail(FF_ERR_INVALID_ARG, "n=%d", n);
  if (n == 0) return FF_OK;
  if (!x_base || !labels) return fail(FF_ERR_INVALID_ARG, "x_base or labels is NULL");
  HeadScratch hs;
  FF_TRY(head_prepare(layers, n_layers, first_layer, hp, head, n, ws, ws_bytes, hs));
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int C = head->n_classes, D = head->d_feat;
  ffk::HeadFeatures f;
  FF_TRY(head_features(layers, n_layers, first_layer, hp, x_base, n, C, hs, st, f));
  head_weights(f, head->W, head->b, D);
  const int splits = ffk::head_grad_splits(n);
  const ffk::AdamArgs a = adam_args(head_hp, head->step + 1);
  const double feat_bytes = (double)n * D * 4.0 + (double)n * f.n_blocks * 4.0;
  FF_HIP(launch(FF_KERNEL_HEAD, Sizes{n, C, D, 1}, 2.0 * n * C * D,
                feat_bytes + (double)C * D * 4.0 + n * C * 4.0, st, [&] {
                  return ffk::launch_head_logits(f, n, C, labels, nullptr, nullptr, hs.G,
                                                 hs.lrow, st);
                }));
  FF_HIP(launch(FF_KERNEL_HEAD, Sizes{n, C, D, 3}, 2.0 * n * C * D,
                feat_bytes + n * C * 4.0 + (double)splits * C * D * 4.0, st, [&] {
                  return ffk::launch_head_grad(f, hs.G, n, C, D, splits, hs.part, st);
                }));
  FF_HIP(launch(FF_KERNEL_HEAD, Sizes{n, C, D, 4}, 0.0,
                (double)splits * C * D * 4.0 + (double)C * D * 24.0, st, [&] {
                  return ffk::launch_head_adam(hs.part, splits, hs.G, hs.lrow, n, C, D,
                                               head->W, head->mW, head->vW, head->b, head->mb,
                                               head->vb, a, loss ? loss : hs.loss, st);
                }));
  ++head->step;
  return FF_OK;
}

ff_status ff_head_predict(const ff_layer *layers, int32_t n_layers, int32_t first_layer,
                          const ff_hparams *hp, const ff_head *head, const float *x_base,
                          int32_t n, float *logits, int32_t *pred, void *ws, size_t ws_bytes,
                          void *stream) {
  FF_TRY(check_head(layers, n_layers, first_layer, hp, head, false));
  if (n < 0) return fail(FF_ERR_INVALID_ARG, "n=%d", n);
  if (n == 0) return FF_OK;
  if (!x_base || !pred) return fail(FF_ERR_INVALID_ARG, "x_base or pred is NULL");
  HeadScratch hs;
  FF_TRY(head_prepare(layers, n_layers, first_layer, hp, head, n, ws, ws_bytes, hs));
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int C = head->n_classes, D = head->d_feat;
  ffk::HeadFeatures f;
  FF_TRY(head_features(layers, n_layers, first_layer, hp, x_base, n, C, hs, st, f));
  head_weights(f, head->W, head->b, D);
  FF_HIP(launch(FF_KERNEL_HEAD, Sizes{n, C, D, 1}, 2.0 * n * C * D,
                (double)n * D * 4.0 + (double)C * D * 4.0 + n * (C + 1) * 4.0, st, [&] {
                  return ffk::launch_head_logits(f, n, C, nullptr, logits, pred, nullptr,
                                                 nullptr, st);
                }));
  return FF_OK;
}

// ---------------------------------------------------------------------------
// Training over chunks: sequential or one stream per layer
// ---------------------------------------------------------------------------
namespace {
// fp32 hidden inputs travel raw, with their row normalisation beside them
// (slot_s, act_s); bf16 layers normalise their input into their own scratch.
// Input slots per layer boundary of the pipelined schedule: layer l may run
// this many chunks ahead of layer l+1.
constexpr int kPipeSlots = 3;
struct PipeScratch {
  std::vector<StepScratch> step;    // per layer (pipelined); sequential: steps, re-forward
  std::vector<float *> slot[kPipeSlots];    // pipelined: [l] input slots of layer l (l >= 1)
  std::vector<float *> slot_s[kPipeSlots];  // pipelined, fp32: row normalisation of slot[.][l]
  // pipelined bf16 FF epochs: layer l's input slots hold its normalised bf16
  // operand rows and their transpose, written by layer l-1's loss pass
  bool bf16_handoff = false;
  std::vector<uint16_t *> slot_b[kPipeSlots], slot_t[kPipeSlots];
  float *act[2] = {nullptr, nullptr};    // sequential: whole-set activations, ping-pong
  float *act_s[2] = {nullptr, nullptr};  // sequential, fp32: their row normalisation
};

// Whether the bf16 steps of an epoch run Adam as a launch of its own (see
// StepScratch::dw), by schedule.
constexpr bool kSplitAdamPipelined = true;
constexpr bool kSplitAdamSequential = false;
// Whether pipelined bf16 FF epochs hand the next layer its operand from the
// loss pass (PipeScratch::bf16_handoff) instead of the activities.
constexpr bool kBf16Handoff = true;

// rpp: rows per sample in a chunk (2 for FF: a positive and a negative row;
// 1 for the performance-optimised variant); po_classes > 0 adds its scratch.
void carve_pipe(Carver &cv, PipeScratch &p, const ff_layer *layers, int L, int n, int chunk,
                int sched, int dtype, int rpp = 2, int po_classes = 0) {
  const int rows = rpp * std::min(chunk, n);
  if (sched == FF_PIPELINED) {
    p.bf16_handoff = kBf16Handoff && dtype == FF_BF16 && po_classes == 0;
    p.step.assign(L, StepScratch());
    for (int k = 0; k < kPipeSlots; ++k) {
      p.slot[k].assign(L, nullptr);
      p.slot_s[k].assign(L, nullptr);
      p.slot_b[k].assign(L, nullptr);
      p.slot_t[k].assign(L, nullptr);
    }
    for (int l = 0; l < L; ++l)
      carve_step(cv, p.step[l], rows, l == 0 || dtype == FF_BF16 ? layers[l].d_in : 0,
                 layers[l].d_out, dtype, l + 1 == L || p.bf16_handoff, false, false, po_classes,
                 true, kSplitAdamPipelined);
    const size_t rp = (size_t)ffk::padded_rows(rows);
    for (int l = 1; l < L; ++l)
      for (int k = 0; k < kPipeSlots; ++k) {
        const size_t d = (size_t)layers[l].d_in;
        if (p.bf16_handoff) {
          p.slot_b[k][l] = static_cast<uint16_t *>(cv.take((size_t)rows * d * 2));
          p.slot_t[k][l] = static_cast<uint16_t *>(cv.take(rp * d * 2));
          continue;
        }
        p.slot[k][l] = static_cast<float *>(cv.take((size_t)rows * d * 4));
        if (dtype == FF_F32) p.slot_s[k][l] = static_cast<float *>(cv.take((size_t)rows * 4));
      }
  } else {
    int max_in = 0, max_out = 0;
    for (int l = 0; l < L; ++l) {
      max_in = std::max(max_in, layers[l].d_in);
      max_out = std::max(max_out, layers[l].d_out);
    }
    p.step.assign(2, StepScratch());
    carve_step(cv, p.step[0], rows, max_in, max_out, dtype, true, false, false, po_classes, true,
               kSplitAdamSequential);
    // the forward pass with the final weights, run beside the next layer's steps
    carve_step(cv, p.step[1], rows, max_in, max_out, dtype, false, false, false, 0, false);
    int max_hidden = 0;
    for (int l = 0; l + 1 < L; ++l) max_hidden = std::max(max_hidden, layers[l].d_out);
    if (L > 1)
      for (int k = 0; k < 2; ++k) {
        p.act[k] = static_cast<float *>(cv.take((size_t)rpp * n * max_hidden * 4));
        if (dtype == FF_F32) p.act_s[k] = static_cast<float *>(cv.take((size_t)rpp * n * 4));
      }
  }
}

struct EventRing {
  std::vector<hipEvent_t> ev;
  ~EventRing() {
    for (hipEvent_t e : ev)
      if (e) (void)hipEventDestroy(e);
  }
};
}  // namespace

size_t ff_pipeline_workspace_size(const ff_layer *layers, int32_t n_layers, int32_t n,
                                  int32_t chunk_pairs, int32_t schedule, int32_t dtype) {
  if (!layers || n_layers <= 0 || n <= 0 || chunk_pairs <= 0) return 0;
  Carver cv(nullptr);
  PipeScratch p;
  carve_pipe(cv, p, layers, n_layers, n, chunk_pairs, schedule, dtype);
  return cv.off + kAlign;
}

}  // extern "C"

namespace {
// Chunk-by-chunk training over `epochs` passes, sequential or one stream per
// layer (see ff_pipeline_epoch).  input0(start, b) describes layer 0's rows of
// the chunk of b samples at `start` (rpp rows per sample); step(l, in, start,
// b, h_out, loss, s_next, scratch, stream) runs one training step of layer l.
template <class Input0, class Step>
ff_status epoch_core(ff_layer *layers, int n_layers, const ff_hparams *hp, int n, int chunk_pairs,
                     int epochs, int schedule, void *const *streams, float *loss_trace,
                     PipeScratch &p, int rpp, Input0 input0, Step step) {
  const int nc = (n + chunk_pairs - 1) / chunk_pairs;
  const int steps = nc * epochs;
  auto chunk_map = [&](int c, int &start, int &b) {
    start = c * chunk_pairs;
    b = std::min(chunk_pairs, n - start);
  };

  if (schedule == FF_SEQUENTIAL) {
    // Layer l's steps run on streams[0].  The forward pass with layer l-1's
    // final weights, which gives layer l its input, runs chunk by chunk on
    // streams[1] (when there is one) beside layer l's steps: step q waits only
    // for the chunk it reads, and the pass starts once layer l-1's last step
    // is done.  The same kernels on the same data as on one stream.
    hipStream_t st = static_cast<hipStream_t>(streams[0]);
    hipStream_t fs = n_layers > 1 && streams[1] ? static_cast<hipStream_t>(streams[1]) : st;
    EventRing evs;  // [0]: layer l-1's steps done; [1]: a chunk of its forward pass done
    if (fs != st) {
      evs.ev.assign(2, nullptr);
      for (auto &e : evs.ev) FF_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    }
    auto input_of = [&](int l, int start, int b) {
      if (l == 0) return input0(start, b);
      const float *in_s = p.act_s[(l - 1) & 1];
      return raw_rows(p.act[(l - 1) & 1] + (size_t)rpp * start * layers[l].d_in,
                      in_s ? in_s + (size_t)rpp * start : nullptr);
    };
    // forward pass of layer l over chunk c into layer l+1's input
    auto reforward = [&](int l, int c, hipStream_t s) -> ff_status {
      int start, b;
      chunk_map(c, start, b);
      float *out_s = p.act_s[l & 1];
      return forward_core(&layers[l], hp, input_of(l, start, b), rpp * b,
                          p.act[l & 1] + (size_t)rpp * start * layers[l].d_out, nullptr,
                          out_s ? out_s + (size_t)rpp * start : nullptr, p.step[1], s);
    };
    for (int l = 0; l < n_layers; ++l) {
      const bool overlap = l > 0 && fs != st;
      if (overlap) {
        FF_HIP(hipEventRecord(evs.ev[0], st));  // layer l-1's last step
        FF_HIP(hipStreamWaitEvent(fs, evs.ev[0], 0));
      }
      for (int q = 0; q < steps; ++q) {
        int start, b;
        chunk_map(q % nc, start, b);
        if (overlap && q < nc) {
          FF_TRY(reforward(l - 1, q, fs));
          FF_HIP(hipEventRecord(evs.ev[1], fs));
          FF_HIP(hipStreamWaitEvent(st, evs.ev[1], 0));
        }
        FF_TRY(step(l, input_of(l, start, b), start, b, nullptr,
                    loss_trace ? loss_trace + (size_t)l * steps + q : nullptr, nullptr, p.step[0],
                    st, nullptr, nullptr));
      }
      if (l + 1 < n_layers && fs == st)
        for (int c = 0; c < nc; ++c) FF_TRY(reforward(l, c, st));
    }
    return FF_OK;
  }

  // Pipelined: out[l][q % kRing] marks layer l's step q's output for layer l+1
  // written (recorded before its weight update), done[l][q % kRing] the whole
  // step complete.  Layer l's step q waits for out[l-1][q] (its input slot is
  // filled) and, before it overwrites layer l+1's slot q % kPipeSlots, for
  // done[l+1][q - kPipeSlots] (the slot's previous reader).  Both waits are
  // enqueued before the event they name is recorded again (kRing >= kPipeSlots
  // steps later, and layer l+1's record of a step follows layer l's in host
  // order).
  constexpr int kRing = 4;
  static_assert(kRing >= kPipeSlots, "event ring");
  EventRing ring, out;
  ring.ev.assign((size_t)n_layers * kRing, nullptr);
  out.ev.assign((size_t)n_layers * kRing, nullptr);
  for (auto &e : ring.ev) FF_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  for (auto &e : out.ev) FF_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  for (int q = 0; q < steps; ++q) {
    int start, b;
    chunk_map(q % nc, start, b);
    for (int l = 0; l < n_layers; ++l) {
      ff_layer *L = &layers[l];
      hipStream_t st = static_cast<hipStream_t>(streams[l]);
      if (l > 0) FF_HIP(hipStreamWaitEvent(st, out.ev[(size_t)(l - 1) * kRing + q % kRing], 0));
      if (l + 1 < n_layers && q >= kPipeSlots)
        FF_HIP(hipStreamWaitEvent(
            st, ring.ev[(size_t)(l + 1) * kRing + (q - kPipeSlots) % kRing], 0));
      const int k = q % kPipeSlots;
      const bool next = l + 1 < n_layers, hand = p.bf16_handoff;
      LayerInput in;
      if (l == 0) {
        in = input0(start, b);
      } else if (hand) {
        in.src.base = reinterpret_cast<const float *>(p.slot_b[k][l]);  // bf16 rows
        in.src.mode = ffk::ROWS;
        in.normalised = true;
        in.xt = p.slot_t[k][l];
      } else {
        in = raw_rows(p.slot[k][l], p.slot_s[k][l]);
      }
      NextBf16 nx;
      if (next && hand) {
        nx.rows = p.slot_b[k][l + 1];
        nx.xt = p.slot_t[k][l + 1];
      }
      FF_TRY(step(l, in, start, b, next && !hand ? p.slot[k][l + 1] : nullptr,
                  loss_trace ? loss_trace + (size_t)l * steps + q : nullptr,
                  next && !hand ? p.slot_s[k][l + 1] : nullptr, p.step[l], st,
                  next && hand ? &nx : nullptr, out.ev[(size_t)l * kRing + q % kRing]));
      FF_HIP(hipEventRecord(ring.ev[(size_t)l * kRing + q % kRing], st));
    }
  }
  return FF_OK;
}
}  // namespace

extern "C" {

ff_status ff_pipeline_epoch(ff_layer *layers, int32_t n_layers, const ff_hparams *hp,
                            const float *x_base, const int32_t *y_pos, const int32_t *y_neg,
                            int32_t n, int32_t n_classes, int32_t chunk_pairs, int32_t epochs,
                            int32_t schedule, void *const *streams, float *loss_trace, void *ws,
                            size_t ws_bytes) {
  FF_TRY(check_hp(hp));
  FF_TRY(check_stack(layers, n_layers, hp, true));
  if (schedule != FF_SEQUENTIAL && schedule != FF_PIPELINED)
    return fail(FF_ERR_INVALID_ARG, "schedule=%d", schedule);
  if (n <= 0 || chunk_pairs <= 0 || epochs <= 0 || n_classes <= 0)
    return fail(FF_ERR_INVALID_ARG, "n=%d chunk_pairs=%d epochs=%d n_classes=%d", n, chunk_pairs,
                epochs, n_classes);
  if (n_classes > layers[0].d_in)
    return fail(FF_ERR_INVALID_ARG, "n_classes=%d exceeds d_in=%d", n_classes, layers[0].d_in);
  if ((int64_t)2 * n > INT32_MAX) return fail(FF_ERR_UNSUPPORTED, "n too large");
  if (!x_base || !y_pos || !y_neg || !streams)
    return fail(FF_ERR_INVALID_ARG, "NULL pointer argument");
  Carver size_cv(nullptr);
  PipeScratch tmp;
  carve_pipe(size_cv, tmp, layers, n_layers, n, chunk_pairs, schedule, hp->dtype);
  FF_TRY(check_ws(ws, ws_bytes, size_cv.off + kAlign));
  Carver cv(ws);
  PipeScratch p;
  carve_pipe(cv, p, layers, n_layers, n, chunk_pairs, schedule, hp->dtype);

  auto pairs_map = [&](int start, int b) {
    ffk::RowMap m{};
    m.base = x_base;
    m.lab_a = y_pos;
    m.lab_b = y_neg;
    m.mode = ffk::PAIRS;
    m.n_pos = b;
    m.base_off = start;
    m.n_classes = n_classes;
    return m;
  };
  auto input0 = [&](int start, int b) {
    LayerInput li;
    li.src = pairs_map(start, b);
    return li;
  };
  auto step = [&](int l, const LayerInput &in, int, int b, float *h_out, float *loss,
                  float *s_next, StepScratch &sc, hipStream_t st, const NextBf16 *nx,
                  hipEvent_t out_ready) {
    return step_core(&layers[l], hp, in, b, b, h_out, nullptr, loss, s_next, sc, st, nx,
                     out_ready);
  };
  return epoch_core(layers, n_layers, hp, n, chunk_pairs, epochs, schedule, streams, loss_trace,
                    p, 2, input0, step);
}
// ---------------------------------------------------------------------------
// Chapter schedules (Single-Layer / All-Layers PFF)
// ---------------------------------------------------------------------------
namespace {
constexpr int kPubSlots = 2;  // published weight versions in flight per layer

struct ChapterScratch {
  std::vector<StepScratch> step;           // per stream
  std::vector<float *> act[2], act_s[2];   // per stream: whole-set activities, ping-pong
  std::vector<float *> pub_w, pub_b;       // [l * kPubSlots + slot]
  std::vector<uint16_t *> pub_wb;          // bf16 shadows of the published weights
  ScoreScratch score;                      // AdaptiveNEG: scoring of the whole set
};

// score_classes > 0: the AdaptiveNEG variant, which also scores the n samples
// under that many labels.
void carve_chapter(Carver &cv, ChapterScratch &c, const ff_layer *layers, int L, int n,
                   int chunk, int n_streams, int dtype, int score_classes = 0) {
  if (score_classes > 0) carve_score(cv, c.score, layers, L, n, score_classes, dtype, true);
  const int rows = 2 * std::min(chunk, n);
  int max_in = 0, max_out = 0, max_hidden = 0;
  for (int l = 0; l < L; ++l) {
    max_in = std::max(max_in, layers[l].d_in);
    max_out = std::max(max_out, layers[l].d_out);
    if (l + 1 < L) max_hidden = std::max(max_hidden, layers[l].d_out);
  }
  c.step.assign(n_streams, StepScratch());
  for (int k = 0; k < 2; ++k) {
    c.act[k].assign(n_streams, nullptr);
    c.act_s[k].assign(n_streams, nullptr);
  }
  for (int s = 0; s < n_streams; ++s) {
    carve_step(cv, c.step[s], rows, max_in, max_out, dtype, true, false, false);
    if (L > 1)
      for (int k = 0; k < 2; ++k) {
        c.act[k][s] = static_cast<float *>(cv.take((size_t)2 * n * max_hidden * 4));
        if (dtype == FF_F32) c.act_s[k][s] = static_cast<float *>(cv.take((size_t)2 * n * 4));
      }
  }
  c.pub_w.assign((size_t)L * kPubSlots, nullptr);
  c.pub_b.assign((size_t)L * kPubSlots, nullptr);
  c.pub_wb.assign((size_t)L * kPubSlots, nullptr);
  for (int l = 0; l + 1 < L; ++l)  // the last layer's versions are never read
    for (int k = 0; k < kPubSlots; ++k) {
      const size_t i = (size_t)l * kPubSlots + k;
      c.pub_w[i] = static_cast<float *>(cv.take((size_t)layers[l].d_out * layers[l].d_in * 4));
      c.pub_b[i] = static_cast<float *>(cv.take((size_t)layers[l].d_out * 4));
      if (dtype == FF_BF16)
        c.pub_wb[i] = static_cast<uint16_t *>(
            cv.take((size_t)layers[l].d_out * layers[l].d_in * 2));
    }
}

float cooldown(float lr0, int epoch, int epochs, int start) {
  if (epoch < start || start >= epochs) return lr0;
  return (float)((double)lr0 * (epochs - epoch) / (epochs - start));
}
}  // namespace

size_t ff_chapter_workspace_size(const ff_layer *layers, int32_t n_layers, int32_t n,
                                 int32_t chunk_pairs, int32_t n_streams, int32_t dtype) {
  if (!layers || n_layers <= 0 || n <= 0 || chunk_pairs <= 0 || n_streams <= 0) return 0;
  Carver cv(nullptr);
  ChapterScratch c;
  carve_chapter(cv, c, layers, n_layers, n, chunk_pairs, n_streams, dtype);
  return cv.off + kAlign;
}

size_t ff_chapter_adaptive_workspace_size(const ff_layer *layers, int32_t n_layers, int32_t n,
                                          int32_t n_classes, int32_t chunk_pairs,
                                          int32_t n_streams, int32_t dtype) {
  if (!layers || n_layers <= 0 || n <= 0 || n_classes <= 0 || chunk_pairs <= 0 || n_streams <= 0)
    return 0;
  Carver cv(nullptr);
  ChapterScratch c;
  carve_chapter(cv, c, layers, n_layers, n, chunk_pairs, n_streams, dtype, n_classes);
  return cv.off + kAlign;
}
}  // extern "C"

namespace {
// Both chapter entry points.  adaptive: chapter c's wrong labels are computed
// on the device when the chapter starts, from the network as every layer left
// it after chapter c-1 (AdaptiveNEG), and written to y_neg_chapters[c];
// otherwise they are read from it.
ff_status chapter_core(ff_layer *layers, int32_t n_layers, const ff_hparams *hp,
                       const float *x_base, const int32_t *y_pos, int32_t *y_neg_chapters,
                       int32_t n, int32_t n_classes, int32_t chunk_pairs, int32_t epochs,
                       int32_t splits, int32_t cooldown_start, int32_t assignment,
                       int32_t n_streams, void *const *streams, float *loss_trace, void *ws,
                       size_t ws_bytes, bool adaptive, int32_t first_scored_layer) {
  FF_TRY(check_hp(hp));
  FF_TRY(check_stack(layers, n_layers, hp, true));
  if (n <= 0 || chunk_pairs <= 0 || splits <= 0 || epochs <= 0 || epochs % splits)
    return fail(FF_ERR_INVALID_ARG, "n=%d chunk_pairs=%d epochs=%d splits=%d (epochs must be a "
                "multiple of splits)", n, chunk_pairs, epochs, splits);
  if (n_classes <= 0 || n_classes > layers[0].d_in)
    return fail(FF_ERR_INVALID_ARG, "n_classes=%d", n_classes);
  if (assignment != FF_SINGLE_LAYER && assignment != FF_ALL_LAYERS)
    return fail(FF_ERR_INVALID_ARG, "assignment=%d", assignment);
  if (assignment == FF_SINGLE_LAYER && n_streams != n_layers)
    return fail(FF_ERR_INVALID_ARG, "FF_SINGLE_LAYER needs one stream per layer (%d, not %d)",
                n_layers, n_streams);
  if (n_streams <= 0) return fail(FF_ERR_INVALID_ARG, "n_streams=%d", n_streams);
  if ((int64_t)2 * n > INT32_MAX) return fail(FF_ERR_UNSUPPORTED, "n too large");
  if (!x_base || !y_pos || !y_neg_chapters || !streams)
    return fail(FF_ERR_INVALID_ARG, "NULL pointer argument");
  if (adaptive) {
    if (n_classes < 2) return fail(FF_ERR_INVALID_ARG, "n_classes=%d: no wrong label", n_classes);
    FF_TRY(check_score_args(layers, n_layers, first_scored_layer, hp, n, n_classes));
  }
  const int score_classes = adaptive ? n_classes : 0;
  Carver size_cv(nullptr);
  ChapterScratch tmp;
  carve_chapter(size_cv, tmp, layers, n_layers, n, chunk_pairs, n_streams, hp->dtype,
                score_classes);
  FF_TRY(check_ws(ws, ws_bytes, size_cv.off + kAlign));
  Carver cv(ws);
  ChapterScratch cs;
  carve_chapter(cv, cs, layers, n_layers, n, chunk_pairs, n_streams, hp->dtype, score_classes);

  const int L = n_layers, S = splits, per = epochs / splits;
  const int nc = (n + chunk_pairs - 1) / chunk_pairs;
  const bool bf16 = hp->dtype == FF_BF16;
  // pub[l][slot]: layer l's version of a chapter is published (its training
  // done); fwd[l][slot]: layer l's input pass of a chapter is done (its reads
  // of the published versions of the layers below are over).
  EventRing pub, fwd;
  pub.ev.assign((size_t)L * kPubSlots, nullptr);
  fwd.ev.assign((size_t)L * kPubSlots, nullptr);
  for (auto &e : pub.ev) FF_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  for (auto &e : fwd.ev) FF_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  auto ev = [&](EventRing &r, int l, int c) { return r.ev[(size_t)l * kPubSlots + c % kPubSlots]; };
  auto pairs = [&](int c, int start, int b) {
    ffk::RowMap m{};
    m.base = x_base;
    m.lab_a = y_pos;
    m.lab_b = y_neg_chapters + (size_t)c * n;
    m.mode = ffk::PAIRS;
    m.n_pos = b;
    m.base_off = start;
    m.n_classes = n_classes;
    LayerInput in;
    in.src = m;
    return in;
  };

  for (int c = 0; c < S; ++c) {
    if (adaptive) {
      // UpdateXNEG: on the worker that trains layer 0 in this chapter, once
      // every layer has finished chapter c-1 (no layer starts chapter c before
      // layer 0, which follows this on the same stream), score the whole set
      // with the live weights and take the best wrong label of each sample.
      const int si = assignment == FF_SINGLE_LAYER ? 0 : c % n_streams;
      hipStream_t st = static_cast<hipStream_t>(streams[si]);
      if (c > 0)
        for (int l = 0; l < L; ++l) FF_HIP(hipStreamWaitEvent(st, ev(pub, l, c - 1), 0));
      FF_TRY(score_run(layers, L, first_scored_layer, hp, x_base, n, n_classes, y_pos,
                       cs.score.scores, y_neg_chapters + (size_t)c * n, cs.score, st));
    }
    for (int l = 0; l < L; ++l) {
      const int si = assignment == FF_SINGLE_LAYER ? l : c % n_streams;
      hipStream_t st = static_cast<hipStream_t>(streams[si]);
      StepScratch &sc = cs.step[si];
      if (l > 0) FF_HIP(hipStreamWaitEvent(st, ev(pub, l - 1, c), 0));
      if (c > 0 && assignment == FF_ALL_LAYERS)  // the layer's chapter c-1 ran elsewhere
        FF_HIP(hipStreamWaitEvent(st, ev(pub, l, c - 1), 0));
      if (c >= kPubSlots && L > 1)  // the version slot of chapter c-2 has no reader left
        FF_HIP(hipStreamWaitEvent(st, ev(fwd, L - 1, c - kPubSlots), 0));
      // input pass: the chapter's pairs through the published layers 0..l-1
      for (int k = 0; k < l; ++k) {
        ff_layer P = layers[k];
        const size_t slot = (size_t)k * kPubSlots + c % kPubSlots;
        P.W = cs.pub_w[slot];
        P.b = cs.pub_b[slot];
        P.W_bf16 = cs.pub_wb[slot];
        float *out = cs.act[k & 1][si];
        float *out_s = cs.act_s[k & 1][si];
        for (int q = 0; q < nc; ++q) {
          const int start = q * chunk_pairs, b = std::min(chunk_pairs, n - start);
          const LayerInput in =
              k == 0 ? pairs(c, start, b)
                     : raw_rows(cs.act[(k - 1) & 1][si] + (size_t)2 * start * P.d_in,
                                bf16 ? nullptr : cs.act_s[(k - 1) & 1][si] + (size_t)2 * start);
          FF_TRY(forward_core(&P, hp, in, 2 * b, out + (size_t)2 * start * P.d_out, nullptr,
                              bf16 ? nullptr : out_s + (size_t)2 * start, sc, st));
        }
      }
      FF_HIP(hipEventRecord(ev(fwd, l, c), st));
      // E/S epochs of layer l over the chunks, with the cooled-down rate
      ff_layer *Ly = &layers[l];
      for (int m = 0; m < per; ++m) {
        const int e = c * per + m;
        ff_hparams hpe = *hp;
        hpe.lr = cooldown(hp->lr, e, epochs, cooldown_start);
        for (int q = 0; q < nc; ++q) {
          const int start = q * chunk_pairs, b = std::min(chunk_pairs, n - start);
          const LayerInput in =
              l == 0 ? pairs(c, start, b)
                     : raw_rows(cs.act[(l - 1) & 1][si] + (size_t)2 * start * Ly->d_in,
                                bf16 ? nullptr : cs.act_s[(l - 1) & 1][si] + (size_t)2 * start);
          float *lt = loss_trace ? loss_trace + (size_t)l * epochs * nc + (size_t)e * nc + q
                                 : nullptr;
          FF_TRY(step_core(Ly, &hpe, in, b, b, nullptr, nullptr, lt, nullptr, sc, st));
        }
      }
      // publish this chapter's version (read by the layers above)
      if (l + 1 < L) {
        const size_t slot = (size_t)l * kPubSlots + c % kPubSlots;
        const size_t wbytes = (size_t)Ly->d_out * Ly->d_in;
        FF_HIP(hipMemcpyAsync(cs.pub_w[slot], Ly->W, wbytes * 4, hipMemcpyDeviceToDevice, st));
        FF_HIP(hipMemcpyAsync(cs.pub_b[slot], Ly->b, (size_t)Ly->d_out * 4,
                              hipMemcpyDeviceToDevice, st));
        if (bf16)
          FF_HIP(hipMemcpyAsync(cs.pub_wb[slot], Ly->W_bf16, wbytes * 2, hipMemcpyDeviceToDevice,
                                st));
      }
      FF_HIP(hipEventRecord(ev(pub, l, c), st));
    }
  }
  return FF_OK;
}
}  // namespace

extern "C" {

ff_status ff_chapter_train(ff_layer *layers, int32_t n_layers, const ff_hparams *hp,
                           const float *x_base, const int32_t *y_pos,
                           const int32_t *y_neg_chapters, int32_t n, int32_t n_classes,
                           int32_t chunk_pairs, int32_t epochs, int32_t splits,
                           int32_t cooldown_start, int32_t assignment, int32_t n_streams,
                           void *const *streams, float *loss_trace, void *ws, size_t ws_bytes) {
  // given negatives are only read
  return chapter_core(layers, n_layers, hp, x_base, y_pos, const_cast<int32_t *>(y_neg_chapters),
                      n, n_classes, chunk_pairs, epochs, splits, cooldown_start, assignment,
                      n_streams, streams, loss_trace, ws, ws_bytes, false, 0);
}

ff_status ff_chapter_train_adaptive(ff_layer *layers, int32_t n_layers, const ff_hparams *hp,
                                    const float *x_base, const int32_t *y_pos,
                                    int32_t *y_neg_chapters, int32_t n, int32_t n_classes,
                                    int32_t chunk_pairs, int32_t epochs, int32_t splits,
                                    int32_t cooldown_start, int32_t assignment,
                                    int32_t first_scored_layer, int32_t n_streams,
                                    void *const *streams, float *loss_trace, void *ws,
                                    size_t ws_bytes) {
  return chapter_core(layers, n_layers, hp, x_base, y_pos, y_neg_chapters, n, n_classes,
                      chunk_pairs, epochs, splits, cooldown_start, assignment, n_streams, streams,
                      loss_trace, ws, ws_bytes, true, first_scored_layer);
}


// ---------------------------------------------------------------------------
// Performance-optimised PFF
// ---------------------------------------------------------------------------
namespace {
ff_status check_po_head(const ff_head *h, int d_out, int l) {
  if (!h) return fail(FF_ERR_INVALID_ARG, "head %d is NULL", l);
  if (h->d_feat != d_out)
    return fail(FF_ERR_INVALID_ARG, "head %d: d_feat=%d, layer d_out=%d", l, h->d_feat, d_out);
  if (h->n_classes < 2 || h->n_classes > ffk::kHeadMaxClasses)
    return fail(FF_ERR_INVALID_ARG, "head %d: n_classes=%d outside [2, %d]", l, h->n_classes,
                ffk::kHeadMaxClasses);
  if (!h->W || !h->b || !h->mW || !h->vW || !h->mb || !h->vb)
    return fail(FF_ERR_INVALID_ARG, "head %d: a buffer is NULL", l);
  return FF_OK;
}
}  // namespace

size_t ff_po_step_workspace_size(int32_t rows, int32_t d_in, int32_t d_out, int32_t n_classes,
                                 int32_t dtype) {
  if (rows <= 0 || d_in <= 0 || d_out <= 0 || n_classes <= 0) return 0;
  Carver cv(nullptr);
  StepScratch s;
  carve_step(cv, s, rows, d_in, d_out, dtype, true, false, true, n_classes);
  return cv.off + kAlign;
}

ff_status ff_po_layer_step(ff_layer *L, ff_head *head, const ff_hparams *hp,
                           const ff_hparams *head_hp, const float *x, const int32_t *labels,
                           int32_t rows, int32_t x_normalised, float *h_out, float *loss, void *ws,
                           size_t ws_bytes, void *stream) {
  FF_TRY(check_hp(hp));
  FF_TRY(check_hp(head_hp));
  FF_TRY(check_layer(L, hp, true, 0));
  FF_TRY(check_po_head(head, L->d_out, 0));
  if (rows < 1) return fail(FF_ERR_INVALID_ARG, "rows=%d", rows);
  if (!x || !labels) return fail(FF_ERR_INVALID_ARG, "x or labels is NULL");
  const int C = head->n_classes;
  Carver size_cv(nullptr);
  StepScratch tmp;
  carve_step(size_cv, tmp, rows, L->d_in, L->d_out, hp->dtype, true, false, true, C);
  FF_TRY(check_ws(ws, ws_bytes, size_cv.off + kAlign));
  Carver cv(ws);
  StepScratch s;
  carve_step(cv, s, rows, L->d_in, L->d_out, hp->dtype, true, false, true, C);
  LayerInput in;
  in.src = rows_of(x);
  in.normalised = x_normalised != 0;
  return po_step_core(L, head, hp, head_hp, in, rows, labels, h_out, loss, nullptr, s,
                      static_cast<hipStream_t>(stream));
}

size_t ff_po_epoch_workspace_size(const ff_layer *layers, int32_t n_layers, int32_t n,
                                  int32_t n_classes, int32_t chunk, int32_t schedule,
                                  int32_t dtype) {
  if (!layers || n_layers <= 0 || n <= 0 || chunk <= 0 || n_classes <= 0) return 0;
  Carver cv(nullptr);
  PipeScratch p;
  carve_pipe(cv, p, layers, n_layers, n, chunk, schedule, dtype, 1, n_classes);
  return cv.off + kAlign;
}

ff_status ff_po_epoch(ff_layer *layers, ff_head *heads, int32_t n_layers, const ff_hparams *hp,
                      const ff_hparams *head_hp, const float *x_base, const int32_t *labels,
                      int32_t n, int32_t n_classes, int32_t chunk, int32_t epochs,
                      int32_t schedule, void *const *streams, float *loss_trace, void *ws,
                      size_t ws_bytes) {
  FF_TRY(check_hp(hp));
  FF_TRY(check_hp(head_hp));
  FF_TRY(check_stack(layers, n_layers, hp, true));
  if (!heads) return fail(FF_ERR_INVALID_ARG, "heads is NULL");
  for (int l = 0; l < n_layers; ++l) {
    FF_TRY(check_po_head(&heads[l], layers[l].d_out, l));
    if (heads[l].n_classes != n_classes)
      return fail(FF_ERR_INVALID_ARG, "head %d: n_classes=%d, expected %d", l,
                  heads[l].n_classes, n_classes);
  }
  if (schedule != FF_SEQUENTIAL && schedule != FF_PIPELINED)
    return fail(FF_ERR_INVALID_ARG, "schedule=%d", schedule);
  if (n <= 0 || chunk <= 0 || epochs <= 0)
    return fail(FF_ERR_INVALID_ARG, "n=%d chunk=%d epochs=%d", n, chunk, epochs);
  if (n_classes > layers[0].d_in)
    return fail(FF_ERR_INVALID_ARG, "n_classes=%d exceeds d_in=%d", n_classes, layers[0].d_in);
  if (!x_base || !labels || !streams) return fail(FF_ERR_INVALID_ARG, "NULL pointer argument");
  Carver size_cv(nullptr);
  PipeScratch tmp;
  carve_pipe(size_cv, tmp, layers, n_layers, n, chunk, schedule, hp->dtype, 1, n_classes);
  FF_TRY(check_ws(ws, ws_bytes, size_cv.off + kAlign));
  Carver cv(ws);
  PipeScratch p;
  carve_pipe(cv, p, layers, n_layers, n, chunk, schedule, hp->dtype, 1, n_classes);
  auto input0 = [&](int start, int) {
    LayerInput li;
    li.src.base = x_base;
    li.src.mode = ffk::NEUTRAL;
    li.src.base_off = start;
    li.src.n_classes = n_classes;
    return li;
  };
  auto step = [&](int l, const LayerInput &in, int start, int b, float *h_out, float *loss,
                  float *s_next, StepScratch &sc, hipStream_t st, const NextBf16 *,
                  hipEvent_t out_ready) -> ff_status {
    return po_step_core(&layers[l], &heads[l], hp, head_hp, in, b, labels + start, h_out, loss,
                        s_next, sc, st, out_ready);
  };
  return epoch_core(layers, n_layers, hp, n, chunk, epochs, schedule, streams, loss_trace, p, 1,
                    input0, step);
}

size_t ff_po_predict_workspace_size(const ff_layer *layers, int32_t n_layers, int32_t n,
                                    int32_t n_classes, int32_t dtype) {
  return ff_head_workspace_size(layers, n_layers, 0, n, n_classes, dtype);
}

ff_status ff_po_predict(const ff_layer *layers, const ff_head *heads, int32_t n_layers,
                        const ff_hparams *hp, const float *x_base, int32_t n, int32_t all_layers,
                        float *logits, int32_t *pred, void *ws, size_t ws_bytes, void *stream) {
  FF_TRY(check_hp(hp));
  FF_TRY(check_stack(layers, n_layers, hp, false));
  if (!heads) return fail(FF_ERR_INVALID_ARG, "heads is NULL");
  if (n_layers > ffk::kHeadMaxBlocks)
    return fail(FF_ERR_UNSUPPORTED, "%d layers (at most %d)", n_layers, ffk::kHeadMaxBlocks);
  const int C = heads[0].n_classes;
  for (int l = 0; l < n_layers; ++l) {
    if (!heads[l].W || !heads[l].b) return fail(FF_ERR_INVALID_ARG, "head %d: W or b is NULL", l);
    if (heads[l].d_feat != layers[l].d_out || heads[l].n_classes != C || C < 2 ||
        C > ffk::kHeadMaxClasses || C > layers[0].d_in)
      return fail(FF_ERR_INVALID_ARG, "head %d: shape does not match", l);
  }
  if (n < 0) return fail(FF_ERR_INVALID_ARG, "n=%d", n);
  if (n == 0) return FF_OK;
  if (!x_base || !pred) return fail(FF_ERR_INVALID_ARG, "x_base or pred is NULL");
  Carver size_cv(nullptr);
  HeadScratch tmp;
  carve_head(size_cv, tmp, layers, n_layers, 0, n, C, hp->dtype);
  FF_TRY(check_ws(ws, ws_bytes, size_cv.off + kAlign));
  Carver cv(ws);
  HeadScratch hs;
  carve_head(cv, hs, layers, n_layers, 0, n, C, hp->dtype);
  hipStream_t st = static_cast<hipStream_t>(stream);
  ffk::HeadFeatures all;
  FF_TRY(head_features(layers, n_layers, 0, hp, x_base, n, C, hs, st, all));
  // raw activities of every layer (or the last) against their own classifiers
  ffk::HeadFeatures f{};
  const int l0 = all_layers ? 0 : n_layers - 1;
  for (int l = l0; l < n_layers; ++l) {
    const int i = f.n_blocks++;
    f.h[i] = all.h[l];
    f.s[i] = nullptr;
    f.d[i] = layers[l].d_out;
    f.w[i] = heads[l].W;
    f.ldw[i] = layers[l].d_out;
    f.bias[f.n_bias++] = heads[l].b;
  }
  double D = 0;
  for (int l = l0; l < n_layers; ++l) D += layers[l].d_out;
  FF_HIP(launch(FF_KERNEL_HEAD, Sizes{n, C, (int32_t)D, 1}, 2.0 * n * C * D,
                (double)n * D * 4.0 + C * D * 4.0, st, [&] {
    return ffk::launch_head_logits(f, n, C, nullptr, logits, pred, nullptr, nullptr, st);
  }));
  return FF_OK;
}

ff_status ff_fail_next_launch(int32_t kind) {
  if (kind < -1 || kind >= FF_KERNEL_KINDS)
    return fail(FF_ERR_INVALID_ARG, "kind=%d outside [-1, %d)", kind, (int)FF_KERNEL_KINDS);
  g_fail_kind.store(kind);
  return FF_OK;
}

// ---------------------------------------------------------------------------
// Kernel timing
// ---------------------------------------------------------------------------
ff_status ff_profile_start(int32_t max_launches, uint32_t kind_mask) {
  if (max_launches <= 0) return fail(FF_ERR_INVALID_ARG, "max_launches=%d", max_launches);
  std::lock_guard<std::mutex> lk(g_prof.mu);
  if (g_prof.on) return fail(FF_ERR_INVALID_ARG, "a profile is already active");
  g_prof.pool.assign((size_t)2 * max_launches, nullptr);
  for (auto &e : g_prof.pool) {
    hipError_t err = hipEventCreate(&e);
    if (err != hipSuccess) {
      for (auto &f : g_prof.pool)
        if (f) (void)hipEventDestroy(f);
      g_prof.pool.clear();
      return fail(FF_ERR_HIP, "hipEventCreate failed: %s", hipGetErrorString(err));
    }
  }
  g_prof.used = 0;
  g_prof.recs.clear();
  g_prof.mask = kind_mask ? kind_mask : ~0u;
  g_prof.on = true;
  return FF_OK;
}

ff_status ff_profile_stop_launches(ff_kernel_stats *stats, ff_launch_record *launches,
                                   int32_t max_launches, int32_t *n_launches) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  if (!g_prof.on) return fail(FF_ERR_INVALID_ARG, "no active profile");
  g_prof.on = false;
  ff_status st = FF_OK;
  if (n_launches) *n_launches = 0;
  if (stats)
    for (int k = 0; k < FF_KERNEL_KINDS; ++k) stats[k] = ff_kernel_stats{0, 0.0, 0.0, 0.0};
  for (const ProfRec &r : g_prof.recs) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(r.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e != hipSuccess) {
      st = fail(FF_ERR_HIP, "reading kernel timing events: %s", hipGetErrorString(e));
      continue;
    }
    if (launches && n_launches && *n_launches < max_launches)
      launches[(*n_launches)++] =
          ff_launch_record{r.kind, r.sz.m, r.sz.n, r.sz.k, r.sz.aux, ms, r.flops, r.bytes};
    if (stats) {
      ff_kernel_stats &k = stats[r.kind];
      k.launches += 1;
      k.total_ms += ms;
      k.flops += r.flops;
      k.bytes += r.bytes;
    }
  }
  for (auto &e : g_prof.pool) (void)hipEventDestroy(e);
  g_prof.pool.clear();
  g_prof.recs.clear();
  g_prof.used = 0;
  return st;
}

ff_status ff_profile_stop(ff_kernel_stats *stats) {
  return ff_profile_stop_launches(stats, nullptr, 0, nullptr);
}

}  // extern "C"
