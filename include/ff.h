/*
 * ff.h -- C ABI of the MI355X (gfx950) Forward-Forward library, libff.so.
 *
 * The library computes the layer-local Forward-Forward (FF) training step and
 * goodness label scoring of "Going Forward-Forward in Distributed Deep
 * Learning" (Aktemur et al., arXiv 2404.08573), and the one-GPU emulation of
 * its Single-Layer pipeline (one HIP stream per layer).
 *
 * Conventions shared by every entry point:
 *  - Pointers marked (device) are HIP device pointers, (host) are host memory.
 *    Matrices are row-major with no padding: a [rows][cols] float matrix has
 *    its element (r, c) at offset r*cols + c.  Device buffers must be 16-byte
 *    aligned (any hipMalloc/PyTorch allocation is).
 *  - The caller allocates and owns every buffer, including the workspace
 *    (`ws`, device, 256-byte aligned, size from the matching *_workspace_size
 *    call) and the Adam state.  The library allocates no device memory.
 *  - `stream` arguments are hipStream_t values passed as void* (NULL is the
 *    default stream).  Calls enqueue asynchronously and return without
 *    synchronising; device-side faults surface at the caller's next sync.
 *  - Errors are returned as ff_status; argument errors are detected on the
 *    host before anything is enqueued, so no state changes (in particular
 *    ff_layer.step is not incremented).  ff_last_error() gives the reason.
 *  - Feature counts (d_in, d_out, d) must be multiples of 4 (16-byte rows).
 *  - Reentrant across distinct layers and streams; one ff_layer must not be
 *    stepped on two streams at once.
 */
#ifndef FF_H
#define FF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FF_OK = 0,
  FF_ERR_INVALID_ARG = -1,   /* bad pointer, size or shape                    */
  FF_ERR_UNSUPPORTED = -2,   /* valid request outside what the kernels handle */
  FF_ERR_WORKSPACE = -3,     /* ws NULL or smaller than required              */
  FF_ERR_HIP = -4            /* a HIP runtime call or kernel launch failed    */
} ff_status;

/* Operand type of the matrix products; accumulation is always fp32.  In
 * FF_BF16 mode three values are rounded to bfloat16 (round to nearest even)
 * before they enter a product: R1 the normalised layer input, R2 the weight
 * shadow W_bf16, R3 the gradient rows dZ = 2 dL/dg * h.  Everything else
 * (activities, goodness, loss, master weights, Adam moments) stays fp32. */
typedef enum { FF_F32 = 0, FF_BF16 = 1 } ff_dtype;

/* Training schedule of ff_pipeline_epoch. */
typedef enum { FF_SEQUENTIAL = 0, FF_PIPELINED = 1 } ff_schedule;

/* Who trains what in ff_chapter_train: one layer per worker stream for every
 * chapter (Single-Layer PFF, Alg. 1), or every layer of chapter c on worker
 * c mod n_streams (All-Layers PFF, Alg. 2). */
typedef enum { FF_SINGLE_LAYER = 0, FF_ALL_LAYERS = 1 } ff_assignment;

/* Largest layer width (d_in, d_out) the kernels take: a 256-row operand tile
 * of that width stays within a 32-bit buffer range.  Wider layers are
 * rejected with FF_ERR_UNSUPPORTED. */
#define FF_MAX_WIDTH (1 << 20)

/* One dense ReLU FF layer, h = max(x_hat W^T + b, 0) (Sec. 3, Sec. 5.1).
 * d_in and d_out are multiples of 4 (of 8 for d_in in FF_BF16 mode), at most
 * FF_MAX_WIDTH.  All buffers are caller-owned device memory. */
typedef struct {
  int32_t d_in, d_out;
  float *W;          /* (device) [d_out][d_in] fp32 master weights           */
  float *b;          /* (device) [d_out]                                      */
  float *mW, *vW;    /* (device) [d_out][d_in] Adam moments, zero at start    */
  float *mb, *vb;    /* (device) [d_out]       Adam moments, zero at start    */
  uint16_t *W_bf16;  /* (device) [d_out][d_in] bf16 shadow of W; required when
                        dtype == FF_BF16 (kept in sync by every update, see
                        ff_refresh_bf16_shadow), ignored otherwise            */
  int64_t step;      /* (host) Adam step count: an update runs with
                        t = step + 1 (the first with t = 1) and stores t in
                        step once its launch is enqueued; a failed launch
                        leaves it unchanged                                   */
} ff_layer;

/* Hyper-parameters.  theta: goodness threshold of Eq. 1.  lr, beta1, beta2,
 * adam_eps: Adam (Sec. 5.1) with bias correction, eps added to sqrt(v_hat),
 * no weight decay.  norm_eps: each layer input row is scaled by
 * 1/(||x||_2 + norm_eps).  dtype: an ff_dtype. */
typedef struct {
  float theta, lr, beta1, beta2, adam_eps, norm_eps;
  int32_t dtype;
} ff_hparams;

/* Human-readable name of a status code (static string). */
const char *ff_status_string(int32_t status);

/* Reason for the last error returned on the calling thread (static buffer). */
const char *ff_last_error(void);

/* Label embedding (Sec. 3, "Negative Data"): out[r] = x_base[r] with features
 * 0..n_classes-1 replaced by the one-hot code of labels[r].
 *   x_base (device) [rows][d] fp32; labels (device) [rows] int32 in
 *   [0, n_classes); out (device) [rows][d] fp32, may alias x_base.
 *   Requires n_classes <= d.  rows == 0 is a no-op. */
ff_status ff_embed_labels(const float *x_base, const int32_t *labels, int32_t rows, int32_t d,
                          int32_t n_classes, float *out, void *stream);

/* Workspace bytes for ff_layer_forward / ff_layer_step on up to `rows` rows. */
size_t ff_step_workspace_size(int32_t rows, int32_t d_in, int32_t d_out, int32_t dtype);

/* Forward pass of one layer without update (Sec. 3, Eq. 1):
 *   x_hat = x / (||x|| + norm_eps) (skipped when x_normalised != 0),
 *   h = max(x_hat W^T + b, 0), g_r = sum_j h_rj^2.
 *   x (device) [rows][d_in]; h_out (device) [rows][d_out] or NULL;
 *   goodness (device) [rows] or NULL.  rows == 0 is a no-op. */
ff_status ff_layer_forward(const ff_layer *L, const ff_hparams *hp, const float *x, int32_t rows,
                           int32_t x_normalised, float *h_out, float *goodness, void *ws,
                           size_t ws_bytes, void *stream);

/* One FF training step of one layer, trainLayer(idx, batch) of Alg. 1/2,
 * on R = n_pos + n_neg concatenated rows (positives first, as the
 * concatenated dataset x of Sec. 4):
 *   forward as ff_layer_forward;
 *   loss = mean_{pos} softplus(theta - g) + mean_{neg} softplus(g - theta)
 *          (negative log-likelihood of Eq. 1, each half averaged over its rows);
 *   dZ_rj = 2 dL/dg_r h_rj;  dW = dZ^T x_hat;  db = sum_r dZ_r
 *          (local gradient only: FF needs no input gradient);
 *   one Adam update of W and b with t = L->step + 1 (then L->step = t).
 *   x (device) [R][d_in]; h_out (device) [R][d_out] or NULL: the activities,
 *   computed with the weights before the update; goodness (device) [R] or
 *   NULL; loss (device) [1] or NULL.  Requires n_pos >= 1 and n_neg >= 1. */
ff_status ff_layer_step(ff_layer *L, const ff_hparams *hp, const float *x, int32_t n_pos,
                        int32_t n_neg, int32_t x_normalised, float *h_out, float *goodness,
                        float *loss, void *ws, size_t ws_bytes, void *stream);

/* ---- No-allocation step ------------------------------------------------------
 * For callers that cannot allocate device memory or take a workspace (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): ff_layer_step with its scratch in a fixed device array of
 * FF_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on
 * until the process ends.  No hipMalloc, hipFree or allocating library call.
 * Arguments and results as ff_layer_step (the same kernels).  The scratch
 * holds the normalised input, the goodness partials and, in bf16, the
 * weight-gradient operands (and the weight gradient itself where the Adam
 * update runs as a launch of its own: layers of 3072 x 3072 and up), plus the
 * activities when h_out is NULL and the
 * goodness and loss when those are NULL; a request that needs more returns
 * FF_ERR_UNSUPPORTED before anything is enqueued (784 -> 2000 and
 * 2000 -> 2000 layers on 2048 rows, and 3072 -> 3072 bf16 layers on 4096 rows
 * with h_out, fit).  The scratch is
 * found for the calling thread's current device, which must be the device
 * of `stream`.  Every call on a GPU shares that GPU's one scratch: calls
 * that overlap on one GPU (different streams or threads) race, so the
 * caller must order them. */
#define FF_NOALLOC_SCRATCH_BYTES (128u << 20)
ff_status ff_layer_step_noalloc(ff_layer *L, const ff_hparams *hp, const float *x, int32_t n_pos,
                                int32_t n_neg, int32_t x_normalised, float *h_out,
                                float *goodness, float *loss, void *stream);

/* Rewrite W_bf16 = bf16(W) (round to nearest even).  Call once after
 * initialising W in FF_BF16 mode; updates keep the shadow in sync after that. */
ff_status ff_refresh_bf16_shadow(const ff_layer *L, void *stream);

/* Workspace bytes for ff_score_labels. */
size_t ff_score_workspace_size(const ff_layer *layers, int32_t n_layers, int32_t n,
                               int32_t n_classes, int32_t dtype);

/* Goodness prediction (Sec. 3 "Prediction"): every input n is run under each
 * label c, embedded as in ff_embed_labels, through all layers;
 *   S[n][c] = sum_{l >= first_scored_layer} g_l(n, c),  pred[n] = argmax_c S[n][c]
 * with the lowest c winning exact ties.  The paper sums "all but the first
 * hidden layer" (first_scored_layer = 1); 0 sums every layer.
 *   layers (host) [n_layers], chained (d_in of l+1 == d_out of l);
 *   x_base (device) [n][layers[0].d_in]; scores (device) [n][n_classes] or
 *   NULL; pred (device) [n] int32.  n == 0 is a no-op. */
ff_status ff_score_labels(const ff_layer *layers, int32_t n_layers, int32_t first_scored_layer,
                          const ff_hparams *hp, const float *x_base, int32_t n, int32_t n_classes,
                          float *scores, int32_t *pred, void *ws, size_t ws_bytes, void *stream);

/* AdaptiveNEG negative labels (Sec. 5, after Hinton's FF paper): the wrong
 * label the network currently scores highest,
 *   y_neg[n] = argmax_{c != labels[n]} S[n][c]   (lowest c on exact ties),
 * with S as in ff_score_labels (same first_scored_layer reading), so the
 * caller can redraw the negatives of the training set between chapters.
 *   labels (device) [n] int32, the true labels: a value outside
 *   [0, n_classes) excludes nothing (not checked on the device);
 *   scores (device) [n][n_classes] or NULL (the unmasked S);
 *   y_neg (device) [n] int32, may not alias labels.
 * n_classes >= 2.  Workspace: ff_score_workspace_size.  n == 0 is a no-op. */
ff_status ff_adaptive_negatives(const ff_layer *layers, int32_t n_layers,
                                int32_t first_scored_layer, const ff_hparams *hp,
                                const float *x_base, const int32_t *labels, int32_t n,
                                int32_t n_classes, float *scores, int32_t *y_neg, void *ws,
                                size_t ws_bytes, void *stream);

/* ---- Chapter schedules (Sec. 4.1 Alg. 1 Single-Layer, Sec. 4.2 Alg. 2 All-Layers)
 * The `epochs` of training are split into `splits` chapters of epochs/splits
 * epochs.  In chapter c, layer l takes the training set (positives with
 * y_pos, negatives with this chapter's wrong labels y_neg_chapters[c]: the
 * RandomNEG redraw, or AdaptiveNEG labels from ff_adaptive_negatives) passed
 * through layers 0..l-1 as published at the end of their chapter c; then it
 * trains epochs/splits epochs over the chunks of chunk_pairs pairs, starting
 * from its own weights after chapter c-1; then its weights are published.
 * The learning rate of (0-based) epoch e is hp->lr until cooldown_start, then
 * hp->lr * (epochs - e) / (epochs - cooldown_start) (the paper's cooldown
 * after epoch 50; its shape is a reading); cooldown_start >= epochs disables it.
 * Both assignments compute the same result: they differ only in which worker
 * stream runs which (layer, chapter), as the nodes of Alg. 1 and Alg. 2 do.
 *   y_neg_chapters (device) [splits][n]; streams (host) [n_streams]
 *   (FF_SINGLE_LAYER: n_streams == n_layers); loss_trace (device)
 *   [n_layers][epochs * n_chunks] or NULL.  epochs must be a multiple of
 *   splits.  The caller must not touch the layers or ws until all streams
 *   have drained. */
size_t ff_chapter_workspace_size(const ff_layer *layers, int32_t n_layers, int32_t n,
                                 int32_t chunk_pairs, int32_t n_streams, int32_t dtype);

ff_status ff_chapter_train(ff_layer *layers, int32_t n_layers, const ff_hparams *hp,
                           const float *x_base, const int32_t *y_pos,
                           const int32_t *y_neg_chapters, int32_t n, int32_t n_classes,
                           int32_t chunk_pairs, int32_t epochs, int32_t splits,
                           int32_t cooldown_start, int32_t assignment, int32_t n_streams,
                           void *const *streams, float *loss_trace, void *ws, size_t ws_bytes);

/* AdaptiveNEG chapters (Sec. 5 negative selection; the UpdateXNEG step of
 * Alg. 1 / Alg. 2): as ff_chapter_train, but chapter c's wrong labels are
 * computed on the device as the chapter begins,
 *   y_neg_chapters[c][i] = argmax_{k != y_pos[i]} S[i][k]   (lowest k on ties),
 * S as in ff_score_labels (first_scored_layer as there) over the whole set,
 * with every layer's weights as they stand after chapter c-1 (the initial
 * weights for c = 0): the last network all layers agree on (a reading; the
 * paper does not say which layer versions regenerate the negatives).  The
 * scoring runs on the worker stream that trains layer 0 in chapter c, after
 * every layer has published chapter c-1, so chapter c of any layer starts
 * after it.
 *   y_neg_chapters (device) [splits][n] int32: output; n_classes >= 2.
 *   Workspace: ff_chapter_adaptive_workspace_size.  Other arguments, errors
 *   and asynchrony as for ff_chapter_train. */
size_t ff_chapter_adaptive_workspace_size(const ff_layer *layers, int32_t n_layers, int32_t n,
                                          int32_t n_classes, int32_t chunk_pairs,
                                          int32_t n_streams, int32_t dtype);

ff_status ff_chapter_train_adaptive(ff_layer *layers, int32_t n_layers, const ff_hparams *hp,
                                    const float *x_base, const int32_t *y_pos,
                                    int32_t *y_neg_chapters, int32_t n, int32_t n_classes,
                                    int32_t chunk_pairs, int32_t epochs, int32_t splits,
                                    int32_t cooldown_start, int32_t assignment,
                                    int32_t first_scored_layer, int32_t n_streams,
                                    void *const *streams, float *loss_trace, void *ws,
                                    size_t ws_bytes);

/* ---- Softmax prediction layer (Sec. 3 "Prediction": Softmax; Sec. 5.1) ------
 * An input is labelled with the neutral label (0.1 in every label feature) and
 * run once through the FF layers without updates.  The activity vectors of
 * layers first_layer..n_layers-1 (the paper: all but the first hidden layer,
 * first_layer = 1), each length-normalised h / (||h|| + norm_eps) as the next
 * layer receives it, are concatenated into A[n][d_feat] and fed to a softmax
 * layer: logits = A W^T + b.  The softmax layer is trained by backpropagation
 * that stops at it (mean cross-entropy, Adam); the FF layers are not changed.
 * Its arithmetic is fp32 in both dtypes (hp->dtype selects the FF layers'
 * operand type only).  At most 8 layers feed it. */
typedef struct {
  int32_t d_feat;     /* sum of d_out over layers first_layer..n_layers-1      */
  int32_t n_classes;  /* C, 2..16, at most layers[0].d_in                      */
  float *W;           /* (device) [n_classes][d_feat]                          */
  float *b;           /* (device) [n_classes]                                  */
  float *mW, *vW;     /* (device) [n_classes][d_feat] Adam moments, zero at start */
  float *mb, *vb;     /* (device) [n_classes]                                  */
  int64_t step;       /* (host) Adam step count, incremented by ff_head_step   */
} ff_head;

/* Workspace bytes for ff_head_step / ff_head_predict on n inputs (it grows
 * with n: every layer's activities for the n inputs are held). */
size_t ff_head_workspace_size(const ff_layer *layers, int32_t n_layers, int32_t first_layer,
                              int32_t n, int32_t n_classes, int32_t dtype);

/* One training step of the softmax layer on a batch of n inputs: logits,
 * mean cross-entropy against labels, its gradient, one Adam update of W and
 * b (head_hp: lr, beta1, beta2, adam_eps; the paper's lr is 1e-4).
 *   layers (host) [n_layers] chained; hp: norm_eps and dtype of the FF layers;
 *   x_base (device) [n][layers[0].d_in]; labels (device) [n] int32 in
 *   [0, n_classes) (others give unspecified results, no stray accesses);
 *   loss (device) [1] or NULL.  n == 0 is a no-op. */
ff_status ff_head_step(const ff_layer *layers, int32_t n_layers, int32_t first_layer,
                       const ff_hparams *hp, ff_head *head, const ff_hparams *head_hp,
                       const float *x_base, const int32_t *labels, int32_t n, float *loss,
                       void *ws, size_t ws_bytes, void *stream);

/* Softmax prediction: one pass, logits (device) [n][n_classes] or NULL and
 * pred (device) [n] int32 = argmax of the logits (lowest class on ties). */
ff_status ff_head_predict(const ff_layer *layers, int32_t n_layers, int32_t first_layer,
                          const ff_hparams *hp, const ff_head *head, const float *x_base,
                          int32_t n, float *logits, int32_t *pred, void *ws, size_t ws_bytes,
                          void *stream);

/* Workspace bytes for ff_pipeline_epoch. */
size_t ff_pipeline_workspace_size(const ff_layer *layers, int32_t n_layers, int32_t n,
                                  int32_t chunk_pairs, int32_t schedule, int32_t dtype);

/* Layer-local FF training of a layer stack over the chunks
 * [c*chunk_pairs, min((c+1)*chunk_pairs, n)) of x_base, in order, `epochs`
 * times.  Chunk c's rows are its positives (labels y_pos) then its negatives
 * (labels y_neg), embedded as in ff_embed_labels.
 *   FF_SEQUENTIAL (Sec. 3 sequential training): layer l takes all its steps,
 *     then one forward pass with its final weights gives layer l+1's input
 *     (the "x <- layer(x)" step of Alg. 2).  The steps run on streams[0]; that
 *     forward pass runs chunk by chunk on streams[1] (when n_layers > 1 and
 *     streams[1] is not NULL; else on streams[0]), beside layer l+1's steps,
 *     each of which waits only for the chunk it reads.  Work on streams[1]
 *     always ends before the last step on streams[0], and the result is the
 *     same either way.
 *   FF_PIPELINED (Single-Layer PFF, Sec. 4.1 / Alg. 1, at the per-batch
 *     exchange granularity proposed in Sec. 6): layer l runs on streams[l];
 *     its step on chunk c starts once layer l-1 has emitted the activities of
 *     chunk c (computed with its weights before that step's update) and
 *     layer l has finished chunk c-1.  The result depends only on these
 *     dependencies, not on how the streams interleave.
 *   layers (host) [n_layers] chained; x_base (device) [n][layers[0].d_in];
 *   y_pos, y_neg (device) [n] int32 in [0, n_classes) (other values give
 *   unspecified results, without out-of-bounds accesses); streams (host)
 *   [n_layers] (only [0] and [1] are read for FF_SEQUENTIAL); loss_trace (device) [n_layers][epochs*n_chunks]
 *   or NULL.  The caller must not touch the layers or ws until all streams
 *   have drained. */
ff_status ff_pipeline_epoch(ff_layer *layers, int32_t n_layers, const ff_hparams *hp,
                            const float *x_base, const int32_t *y_pos, const int32_t *y_neg,
                            int32_t n, int32_t n_classes, int32_t chunk_pairs, int32_t epochs,
                            int32_t schedule, void *const *streams, float *loss_trace, void *ws,
                            size_t ws_bytes);

/* ---- Performance-Optimised PFF (Sec. 4, "PFF with a new goodness function") -
 * Each layer l carries its own softmax classifier heads[l] (d_feat = d_out of
 * layer l).  The layer and its classifier are trained together by
 * backpropagation through those two layers only, on the mean cross-entropy of
 * the labels; there is no negative data.  Readings: the classifier takes the
 * layer's activities h as they are; layer 0 sees the neutrally labelled input
 * (0.1 in every label feature); each layer input is normalised as for FF.
 * Both the layer (hp: lr, betas, adam_eps) and the classifier (head_hp) take
 * one Adam update per step.  In FF_BF16 mode the layer's products use bf16
 * operands at R1/R2/R3 (R3: the gradient rows dZ); the classifier is fp32. */

/* Workspace bytes for ff_po_layer_step on up to `rows` rows. */
size_t ff_po_step_workspace_size(int32_t rows, int32_t d_in, int32_t d_out, int32_t n_classes,
                                 int32_t dtype);

/* One step on `rows` input rows x (device) [rows][d_in] with labels (device)
 * [rows] int32 in [0, n_classes): h = relu(x_hat W^T + b), logits = h Wc^T +
 * bc, loss = mean cross-entropy; dWc = G^T h, dZ = (G Wc) * [h > 0],
 * dW = dZ^T x_hat (G = dloss/dlogits); Adam on W, b, Wc, bc.
 *   h_out (device) [rows][d_out] or NULL: the activities before the update
 *   (the next layer's input); loss (device) [1] or NULL. */
ff_status ff_po_layer_step(ff_layer *L, ff_head *head, const ff_hparams *hp,
                           const ff_hparams *head_hp, const float *x, const int32_t *labels,
                           int32_t rows, int32_t x_normalised, float *h_out, float *loss, void *ws,
                           size_t ws_bytes, void *stream);

/* Workspace bytes for ff_po_epoch. */
size_t ff_po_epoch_workspace_size(const ff_layer *layers, int32_t n_layers, int32_t n,
                                  int32_t n_classes, int32_t chunk, int32_t schedule,
                                  int32_t dtype);

/* Performance-optimised training over the chunks [c*chunk, min((c+1)*chunk, n))
 * of x_base, `epochs` times, with the schedules of ff_pipeline_epoch
 * (sequential, or one stream per layer handing each chunk's activities on).
 *   heads (host) [n_layers], all with n_classes classes; labels (device) [n];
 *   loss_trace (device) [n_layers][epochs*n_chunks] or NULL. */
ff_status ff_po_epoch(ff_layer *layers, ff_head *heads, int32_t n_layers, const ff_hparams *hp,
                      const ff_hparams *head_hp, const float *x_base, const int32_t *labels,
                      int32_t n, int32_t n_classes, int32_t chunk, int32_t epochs,
                      int32_t schedule, void *const *streams, float *loss_trace, void *ws,
                      size_t ws_bytes);

/* Workspace bytes for ff_po_predict on n inputs. */
size_t ff_po_predict_workspace_size(const ff_layer *layers, int32_t n_layers, int32_t n,
                                    int32_t n_classes, int32_t dtype);

/* Prediction of a performance-optimised network: one neutral-label pass; the
 * logits of the last layer's classifier (all_layers == 0) or the sum of every
 * layer's classifier logits (all_layers != 0, a reading of "all layers").
 *   logits (device) [n][n_classes] or NULL; pred (device) [n] int32 (argmax,
 *   lowest class on ties).  At most 8 layers. */
ff_status ff_po_predict(const ff_layer *layers, const ff_head *heads, int32_t n_layers,
                        const ff_hparams *hp, const float *x_base, int32_t n, int32_t all_layers,
                        float *logits, int32_t *pred, void *ws, size_t ws_bytes, void *stream);

/* ---- Kernel timing (tracing aid) -------------------------------------------
 * Between ff_profile_start and ff_profile_stop every kernel the library
 * launches (up to max_launches) is bracketed by a pair of hipEvents recorded on
 * the stream it is launched on, and the algorithmic work of the launch is
 * counted: flops of the matrix products (2*M*N*K) and the bytes that the
 * operation must read and write at minimum.  ff_profile_stop waits for the
 * recorded events, fills stats[FF_KERNEL_KINDS] and releases the events.
 * Process-wide state; not reentrant with itself. */
typedef enum {
  FF_KERNEL_EMBED_NORM = 0,  /* label embedding + row normalisation          */
  FF_KERNEL_FORWARD = 1,     /* fused forward product + bias/ReLU/goodness    */
  FF_KERNEL_LOSS = 2,        /* goodness reduction, loss, row coefficients    */
  FF_KERNEL_DW_ADAM = 3,     /* weight-gradient product + fused Adam          */
  FF_KERNEL_GOODNESS = 4,    /* goodness reduction / score accumulation       */
  FF_KERNEL_ARGMAX = 5,      /* label argmax                                  */
  FF_KERNEL_SHADOW = 6,      /* bf16 weight shadow refresh                    */
  FF_KERNEL_HEAD = 7,        /* softmax layer: logits, gradient, Adam         */
  FF_KERNEL_TRANSPOSE = 8,   /* reserved: the bf16 loss pass writes the transposes */
  FF_KERNEL_ADAM = 9,        /* Adam update from a stored weight gradient     */
  FF_KERNEL_KINDS = 10
} ff_kernel_kind;

typedef struct {
  int64_t launches;   /* launches timed                                      */
  double total_ms;    /* sum of event-measured durations                     */
  double flops;       /* algorithmic flops of those launches                 */
  double bytes;       /* algorithmic HBM bytes of those launches             */
} ff_kernel_stats;

/* One timed launch.  Sizes by kind:
 *   FORWARD      m rows, n output features, k input features; aux = label
 *                count of the label-expanding scoring product (m base rows),
 *                else 0;
 *   DW_ADAM      m = d_out, n = d_in, k = rows contracted; aux = 1 when the
 *                product stores the gradient for a separate ADAM launch;
 *   ADAM         m = d_out, n = d_in, k = rows of the step;
 *   EMBED_NORM   m rows, n features; aux = the row source mode, plus 16
 *                for bf16 output rows;
 *   LOSS         m rows, n = d_out, k = goodness partials per row; aux bit 0:
 *                the pass also writes the bf16 weight-gradient operand, bit 1:
 *                the next layer's normalised bf16 operand, bit 2: the
 *                transpose of the layer's bf16 input rows;
 *   GOODNESS     m rows, n = partials per row;
 *   ARGMAX       m rows, n labels;
 *   SHADOW       m x n weights;
 *   HEAD         m rows, n classes, k features; aux = 1 logits, 2 layer dZ,
 *                3 weight-gradient partials, 4 Adam. */
typedef struct {
  int32_t kind;       /* ff_kernel_kind                                      */
  int32_t m, n, k, aux;
  float ms;           /* event-measured duration                             */
  double flops;       /* algorithmic flops                                   */
  double bytes;       /* algorithmic HBM bytes                               */
} ff_launch_record;

/* kind_mask: bit k selects kernel kind k (0 selects every kind); launches of
 * other kinds run without events. */
ff_status ff_profile_start(int32_t max_launches, uint32_t kind_mask);
ff_status ff_profile_stop(ff_kernel_stats *stats /* (host) [FF_KERNEL_KINDS] */);
/* As ff_profile_stop, and also the timed launches one by one in the order the
 * host enqueued them: the first min(max_launches, timed) into launches
 * (host, may be NULL), their number into *n_launches (host, may be NULL). */
ff_status ff_profile_stop_launches(ff_kernel_stats *stats /* (host) [FF_KERNEL_KINDS] or NULL */,
                                   ff_launch_record *launches, int32_t max_launches,
                                   int32_t *n_launches);

/* ---- Failure injection (testing aid) ---------------------------------------
 * The next launch of kernel kind `kind` (an ff_kernel_kind) that any entry
 * point makes enqueues nothing and fails, so the entry point returns
 * FF_ERR_HIP as for a failed launch; -1 disarms.  Lets tests check that a
 * failed launch leaves host state (the Adam step counts) as it was.
 * Process-wide; FF_ERR_INVALID_ARG for a kind outside [-1, FF_KERNEL_KINDS). */
ff_status ff_fail_next_launch(int32_t kind);

#ifdef __cplusplus
}
#endif

#endif /* FF_H */
