"""CPU oracle for the Forward-Forward (FF) training step and goodness label scoring.

TEST INFRASTRUCTURE ONLY.  This is a plain, slow, deliberately unfused fp64
NumPy statement of what the paper defines.  Only the test suite, the smoke
check and the benchmark's CPU-baseline leg may import it; the HIP library and
its Python binding never do, and it imports nothing from them.

Every function cites the passage of "Going Forward-Forward in Distributed
Deep Learning" (Aktemur et al., arXiv 2404.08573) it follows.  Where the paper
is silent the reading taken is stated in the docstring; the same readings are
documented for the HIP path.

Precision: contractions and all elementwise work run in float64 from the
float32 inputs.  In ``bf16`` mode the values that the HIP path feeds to its
bf16 matrix instructions are rounded to bfloat16 (round to nearest even) at
exactly three points -- R1 the normalised layer input, R2 the weight shadow,
R3 the gradient rows ``dZ`` -- and everything else stays float64.

Parity status: every function below is pinned by the CPU tests in
``tests/test_oracle.py`` (closed forms, hand-built layers, finite differences,
a PyTorch-CPU autograd/Adam cross-check, brute force, invariances), except the
paper-level accuracy and timing tables, which need MNIST/CIFAR-10 and the
paper's cluster: parity unpinned for those (not computed here at all).
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence, Tuple

import numpy as np

F64 = np.float64


# ----------------------------------------------------------------------------
# bfloat16 rounding (the GPU path's bf16 operand format)
# ----------------------------------------------------------------------------
def bf16_round(x) -> np.ndarray:
    """Round to bfloat16 (round to nearest, ties to even) and return float64.

    The value is first rounded to float32 (the GPU holds it in float32 before
    conversion), then the low 16 mantissa bits are rounded away.
    """
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    u = (u + 0x7FFF + lsb) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(F64)


# ----------------------------------------------------------------------------
# Inputs: label embedding and per-layer normalisation
# ----------------------------------------------------------------------------
def embed_labels(x_base: np.ndarray, labels: np.ndarray, n_classes: int) -> np.ndarray:
    """Write a 1-of-C label into the first ``n_classes`` features (Sec. 3, "Negative Data").

    The paper places the label in a 10-pixel border area of the MNIST image;
    the workloads here use features 0..C-1 as that area.  A positive sample
    carries the true label, a negative one a wrong label.
    """
    x = np.array(x_base, dtype=F64, copy=True)
    x[:, :n_classes] = 0.0
    x[np.arange(x.shape[0]), np.asarray(labels, dtype=np.int64)] = 1.0
    return x


def l2_normalise(x: np.ndarray, eps: float) -> np.ndarray:
    """Scale each row to unit length: ``x / (||x||_2 + eps)``.

    The paper does not mention input normalisation; the workloads require it
    for every layer input (eps 1e-8).  Reading: eps is added to the norm, not
    to the squared norm; an all-zero row stays zero.
    """
    x = np.asarray(x, dtype=F64)
    nrm = np.sqrt(np.sum(x * x, axis=1, keepdims=True))
    return x / (nrm + eps)


# ----------------------------------------------------------------------------
# One FF layer: forward, goodness, loss, local gradient (Sec. 3, Eq. 1)
# ----------------------------------------------------------------------------
def goodness(h: np.ndarray) -> np.ndarray:
    """Goodness of each row: the sum of squared ReLU activities (Sec. 3, Eq. 1)."""
    return np.sum(h * h, axis=1)


def layer_forward(W, b, x, norm_eps: float, normalised: bool = False, bf16: bool = False):
    """Dense ReLU layer on normalised input; returns (x_hat, z, h, g).

    ``z = x_hat W^T + b``, ``h = max(z, 0)``, ``g = sum_j h_j^2`` (Sec. 3, Eq. 1;
    the layer shapes of Sec. 5.1).  In bf16 mode x_hat (R1) and W (R2) are
    rounded to bfloat16 before the contraction.
    """
    xh = np.asarray(x, dtype=F64) if normalised else l2_normalise(x, norm_eps)
    Wm = np.asarray(W, dtype=F64)
    if bf16:
        xh = bf16_round(xh)
        Wm = bf16_round(Wm)
    z = xh @ Wm.T + np.asarray(b, dtype=F64)
    h = np.maximum(z, 0.0)
    return xh, z, h, goodness(h)


def softplus(x):
    """``log(1 + e^x)`` in the overflow-free form ``max(x, 0) + log1p(e^-|x|)``."""
    x = np.asarray(x, dtype=F64)
    return np.maximum(x, 0.0) + np.log1p(np.exp(-np.abs(x)))


def sigmoid(x):
    """Logistic function, evaluated without overflow on either side."""
    x = np.asarray(x, dtype=F64)
    e = np.exp(-np.abs(x))
    return np.where(x >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def ff_loss(g: np.ndarray, n_pos: int, theta: float) -> Tuple[float, np.ndarray]:
    """Threshold loss of Eq. 1 and its derivative with respect to each row's goodness.

    Eq. 1 gives ``p(real) = sigma(g - theta)``.  Its negative log-likelihood is
    ``softplus(theta - g)`` for a positive row and ``softplus(g - theta)`` for a
    negative row.  Reading of the normalisation: the loss is the mean over the
    positive rows plus the mean over the negative rows (rows ``0..n_pos-1`` are
    positive, the rest negative, as in the concatenated dataset of Sec. 4).
    Returns ``(loss, dL/dg)``.
    """
    g = np.asarray(g, dtype=F64)
    n_neg = g.shape[0] - n_pos
    pos, neg = g[:n_pos], g[n_pos:]
    loss = np.sum(softplus(theta - pos)) / n_pos + np.sum(softplus(neg - theta)) / n_neg
    dg = np.concatenate([-sigmoid(theta - pos) / n_pos, sigmoid(neg - theta) / n_neg])
    return float(loss), dg


def layer_grads(xh: np.ndarray, h: np.ndarray, dLdg: np.ndarray, bf16: bool = False):
    """Local weight gradient of one FF layer; there is no input gradient.

    FF trains each layer from its own objective (Sec. 1, Sec. 3), so only
    dL/dW and dL/db of this layer are needed.  By the chain rule through
    ``g = sum_j h_j^2`` and ``h = max(z, 0)``: ``dZ_rj = 2 (dL/dg_r) h_rj``
    (``h = 0`` wherever the ReLU is off, so the mask is implicit),
    ``dW = dZ^T x_hat`` and ``db = sum_r dZ_r``.  In bf16 mode dZ is rounded to
    bfloat16 (R3) before the contraction; x_hat arrives already rounded (R1).
    """
    dZ = 2.0 * dLdg[:, None] * h
    dZc = bf16_round(dZ) if bf16 else dZ
    dW = dZc.T @ xh
    db = np.sum(dZ, axis=0)
    return dW, db


def adam(p, m, v, grad, t: int, lr: float, beta1: float, beta2: float, eps: float):
    """One Adam update with bias correction (the optimiser of Sec. 5.1).

    The paper names Adam and its learning rate only.  Reading: the standard
    form with bias-corrected moments, eps added to the root of the second
    moment, no weight decay, ``t`` counting from 1 for each layer.
    """
    m = beta1 * m + (1.0 - beta1) * grad
    v = beta2 * v + (1.0 - beta2) * grad * grad
    m_hat = m / (1.0 - beta1 ** t)
    v_hat = v / (1.0 - beta2 ** t)
    p = p - lr * m_hat / (np.sqrt(v_hat) + eps)
    return p, m, v


# ----------------------------------------------------------------------------
# Layer state and one training step
# ----------------------------------------------------------------------------
@dataclasses.dataclass
class HParams:
    theta: float = 2.0
    lr: float = 0.03
    beta1: float = 0.9
    beta2: float = 0.999
    adam_eps: float = 1e-8
    norm_eps: float = 1e-8
    bf16: bool = False


@dataclasses.dataclass
class Layer:
    """Parameters and Adam moments of one FF layer, in float64."""
    W: np.ndarray
    b: np.ndarray
    mW: np.ndarray
    vW: np.ndarray
    mb: np.ndarray
    vb: np.ndarray
    t: int = 0

    @staticmethod
    def from_params(W, b) -> "Layer":
        W = np.array(W, dtype=F64)
        b = np.array(b, dtype=F64)
        return Layer(W, b, np.zeros_like(W), np.zeros_like(W), np.zeros_like(b), np.zeros_like(b))

    def copy(self) -> "Layer":
        return Layer(self.W.copy(), self.b.copy(), self.mW.copy(), self.vW.copy(),
                     self.mb.copy(), self.vb.copy(), self.t)


@dataclasses.dataclass
class StepResult:
    h: np.ndarray        # [R, d_out] activities, computed with the weights before the update
    g: np.ndarray        # [R] goodness
    loss: float
    dW: np.ndarray       # gradient applied by the update
    db: np.ndarray
    xh: np.ndarray       # [R, d_in] normalised input (bf16-rounded in bf16 mode)
    dLdg: np.ndarray     # [R] derivative of the loss with respect to each goodness


def layer_step(L: Layer, x: np.ndarray, n_pos: int, hp: HParams,
               normalised: bool = False) -> StepResult:
    """One FF training step of a layer on concatenated positive+negative rows.

    ``trainLayer(idx, batch)`` of Alg. 1/2 for one mini-batch: the positive
    pass raises and the negative pass lowers the goodness (Sec. 3), both via
    the loss of Eq. 1, followed by one Adam update (Sec. 5.1).  Mutates ``L``.
    """
    xh, _, h, g = layer_forward(L.W, L.b, x, hp.norm_eps, normalised, hp.bf16)
    loss, dg = ff_loss(g, n_pos, hp.theta)
    dW, db = layer_grads(xh, h, dg, hp.bf16)
    L.t += 1
    L.W, L.mW, L.vW = adam(L.W, L.mW, L.vW, dW, L.t, hp.lr, hp.beta1, hp.beta2, hp.adam_eps)
    L.b, L.mb, L.vb = adam(L.b, L.mb, L.vb, db, L.t, hp.lr, hp.beta1, hp.beta2, hp.adam_eps)
    return StepResult(h, g, loss, dW, db, xh, dg)


# ----------------------------------------------------------------------------
# Goodness label scoring (Sec. 3 "Prediction", Sec. 5)
# ----------------------------------------------------------------------------
def score_labels(layers: Sequence[Layer], x_base: np.ndarray, n_classes: int,
                 hp: HParams, first_scored_layer: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    """Goodness prediction: run every input under each label, sum goodness, take the argmax.

    Sec. 3 runs the input with each of the C one-hot labels and accumulates
    the goodness of the hidden layers; the label with the largest total wins.
    The paper counts "all but the first hidden layer" (``first_scored_layer=1``);
    the workloads count every layer (``first_scored_layer=0``).  Ties go to the
    lowest label index.  Returns ``(S[n, C], pred[n])``.
    """
    n = x_base.shape[0]
    S = np.zeros((n, n_classes), dtype=F64)
    for c in range(n_classes):
        a = embed_labels(x_base, np.full(n, c), n_classes)
        for li, L in enumerate(layers):
            _, _, a, g = layer_forward(L.W, L.b, a, hp.norm_eps, False, hp.bf16)
            if li >= first_scored_layer:
                S[:, c] += g
    return S, np.argmax(S, axis=1).astype(np.int32)


def adaptive_negatives(layers: Sequence[Layer], x_base: np.ndarray, labels: np.ndarray,
                       n_classes: int, hp: HParams,
                       first_scored_layer: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    """AdaptiveNEG (Sec. 5, the negative selection of Hinton's FF paper).

    Each sample's negative label is the wrong label that the current network
    predicts most strongly: the goodness prediction above is computed for every
    label, the true label is set aside, and the best of the remaining labels is
    taken (lowest index on ties).  Returns ``(S[n, C], y_neg[n])``.
    """
    S, _ = score_labels(layers, x_base, n_classes, hp, first_scored_layer)
    y_neg = np.empty(S.shape[0], dtype=np.int32)
    for i in range(S.shape[0]):
        best = -1
        for c in range(n_classes):
            if c != labels[i] and (best < 0 or S[i, c] > S[i, best]):
                best = c
        y_neg[i] = best
    return S, y_neg


# ----------------------------------------------------------------------------
# Chapter schedules of Single-Layer / All-Layers PFF (Sec. 4.1, Alg. 1; Sec. 4.2, Alg. 2)
# ----------------------------------------------------------------------------
def cooldown_lr(lr0: float, epoch: int, epochs: int, cooldown_start: int) -> float:
    """Learning rate of (0-based) global epoch ``epoch``.  The paper cools the rate
    down after the 50th of 100 epochs without giving the shape; reading: constant
    until ``cooldown_start``, then a linear decay that would reach 0 at ``epochs``."""
    if epoch < cooldown_start or cooldown_start >= epochs:
        return lr0
    return lr0 * (epochs - epoch) / (epochs - cooldown_start)


def chapter_train(layers: List[Layer], x_base, y, y_neg_chapters, n_classes: int,
                  chunk_pairs: int, epochs: int, splits: int, cooldown_start: int,
                  hp: HParams, on_step=None) -> np.ndarray:
    """Chapter-granularity PFF training (Alg. 1 Single-Layer; Alg. 2 All-Layers).

    The E epochs are split into S chapters of E/S epochs.  In chapter c, layer l
    first takes as input the training set (positives with labels y, negatives
    with this chapter's wrong labels) passed through layers 0..l-1 as published
    at the end of their chapter c ("x <- layer(x)" with getLayer(k, chapter));
    then it trains for E/S epochs over the chunks, starting from its own
    weights after chapter c-1, with the cooled-down learning rate of each
    epoch; then it is published.  Single-Layer (one layer per node) and
    All-Layers (each node trains the whole net for a chapter, handing each layer
    on) compute this same dependency graph; they differ in which node does
    which (layer, chapter).

    ``y_neg_chapters`` is either the chapters' wrong labels (``[S][n]``: the
    RandomNEG redraw of every chapter, random numbers being inputs here) or a
    function ``negatives(c, layers)`` called when chapter c begins, while every
    layer still holds its weights after chapter c-1 (the initial weights for
    c = 0), which returns that chapter's wrong labels (AdaptiveNEG:
    ``adaptive_chapter_negatives``).  Returns the loss trace ``[L, E * n_chunks]``.
    ``on_step(l, result)``, if given, sees every step's StepResult (test
    bookkeeping; no effect on results).
    """
    E, S = epochs, splits
    assert E % S == 0
    per = E // S
    chunks = chunk_bounds(x_base.shape[0], chunk_pairs)
    L = len(layers)
    trace = np.zeros((L, E * len(chunks)))
    for c in range(S):
        y_neg = y_neg_chapters(c, layers) if callable(y_neg_chapters) else y_neg_chapters[c]
        published = []
        for li, Ly in enumerate(layers):
            # the chapter's input of this layer: every chunk through the published layers
            inputs = []
            for (s, b) in chunks:
                a = chunk_input(x_base, y, y_neg, s, b, n_classes)
                for P in published:
                    a = layer_forward(P[0], P[1], a, hp.norm_eps, False, hp.bf16)[2]
                inputs.append(a)
            for m in range(per):
                e = c * per + m
                hp_e = dataclasses.replace(hp, lr=cooldown_lr(hp.lr, e, E, cooldown_start))
                for q, (s, b) in enumerate(chunks):
                    r = layer_step(Ly, inputs[q], b, hp_e)
                    trace[li, e * len(chunks) + q] = r.loss
                    if on_step:
                        on_step(li, r)
            published.append((Ly.W.copy(), Ly.b.copy()))
    return trace


def adaptive_chapter_negatives(x_base, y, n_classes: int, hp: HParams,
                               first_scored_layer: int = 0, record: Optional[list] = None):
    """AdaptiveNEG negatives for the chapter schedules (Sec. 5 negative selection,
    the UpdateXNEG step of Alg. 1 / Alg. 2): the function ``negatives(c, layers)``
    that ``chapter_train`` calls as chapter c begins.  It returns the wrong label
    the network scores highest for every training sample (``adaptive_negatives``
    over the whole set), evaluated with every layer's weights after chapter c-1.
    Reading: the paper regenerates the adaptive negatives between chapters
    without saying from which layer versions; here they come from the network as
    it stands when the chapter starts, the last network all layers agree on.
    ``record``, if given, collects each chapter's labels."""
    def negatives(c, layers):
        y_neg = adaptive_negatives(layers, x_base, y, n_classes, hp, first_scored_layer)[1]
        if record is not None:
            record.append(y_neg)
        return y_neg
    return negatives


# ----------------------------------------------------------------------------
# Softmax prediction head (Sec. 3 "Prediction", Sec. 5, Sec. 5.1)
# ----------------------------------------------------------------------------
NEUTRAL_LABEL = 0.1


def embed_neutral(x_base: np.ndarray, n_classes: int) -> np.ndarray:
    """Neutral label for Softmax prediction (Sec. 3): every label feature is 0.1."""
    x = np.array(x_base, dtype=F64, copy=True)
    x[:, :n_classes] = NEUTRAL_LABEL
    return x


@dataclasses.dataclass
class Head:
    """The softmax layer: ``W[C][D]``, ``b[C]`` and their Adam moments, float64."""
    W: np.ndarray
    b: np.ndarray
    mW: np.ndarray
    vW: np.ndarray
    mb: np.ndarray
    vb: np.ndarray
    t: int = 0

    @staticmethod
    def from_params(W, b) -> "Head":
        W = np.array(W, dtype=F64)
        b = np.array(b, dtype=F64)
        return Head(W, b, np.zeros_like(W), np.zeros_like(W), np.zeros_like(b),
                    np.zeros_like(b))

    def copy(self) -> "Head":
        return Head(self.W.copy(), self.b.copy(), self.mW.copy(), self.vW.copy(),
                    self.mb.copy(), self.vb.copy(), self.t)


def head_features(layers: Sequence[Layer], x_base: np.ndarray, n_classes: int, hp: HParams,
                  first_layer: int = 1) -> np.ndarray:
    """Input of the softmax layer: one pass of the neutrally labelled input through
    the FF layers (no update), keeping the activity vectors of the hidden layers
    from ``first_layer`` on ("all but the first hidden layer": 1).  Reading: each
    activity vector enters length-normalised, ``h / (||h|| + norm_eps)``, the form in
    which the next layer receives it.  Returns ``A[n, sum of their widths]``.
    """
    a = embed_neutral(x_base, n_classes)
    feats = []
    for li, L in enumerate(layers):
        _, _, a, _ = layer_forward(L.W, L.b, a, hp.norm_eps, False, hp.bf16)
        if li >= first_layer:
            feats.append(l2_normalise(a, hp.norm_eps))
    return np.concatenate(feats, axis=1)


def softmax_xent(logits: np.ndarray, y: np.ndarray) -> Tuple[float, np.ndarray, np.ndarray]:
    """Mean cross-entropy of softmax(logits) against labels y, its gradient with
    respect to the logits, and the probabilities.  Softmax is taken after
    subtracting each row's maximum (the same value in exact arithmetic)."""
    z = np.asarray(logits, dtype=F64)
    z = z - z.max(axis=1, keepdims=True)
    e = np.exp(z)
    p = e / e.sum(axis=1, keepdims=True)
    n = z.shape[0]
    loss = float(np.mean(np.log(e.sum(axis=1)) - z[np.arange(n), y]))
    d = p.copy()
    d[np.arange(n), y] -= 1.0
    return loss, d / n, p


def head_step(head: Head, layers: Sequence[Layer], x_base: np.ndarray, y: np.ndarray,
              n_classes: int, hp: HParams, head_hp: HParams, first_layer: int = 1):
    """One training step of the softmax layer on a batch (Sec. 3: trained by
    backpropagation, which stops at the softmax layer; Sec. 5.1: Adam).  The FF
    layers are not changed.  Returns ``(loss, logits, dW, db)``; mutates ``head``."""
    A = head_features(layers, x_base, n_classes, hp, first_layer)
    logits = A @ head.W.T + head.b
    loss, d, _ = softmax_xent(logits, np.asarray(y, dtype=np.int64))
    dW = d.T @ A
    db = d.sum(axis=0)
    head.t += 1
    head.W, head.mW, head.vW = adam(head.W, head.mW, head.vW, dW, head.t, head_hp.lr,
                                    head_hp.beta1, head_hp.beta2, head_hp.adam_eps)
    head.b, head.mb, head.vb = adam(head.b, head.mb, head.vb, db, head.t, head_hp.lr,
                                    head_hp.beta1, head_hp.beta2, head_hp.adam_eps)
    return loss, logits, dW, db


def head_predict(head: Head, layers: Sequence[Layer], x_base: np.ndarray, n_classes: int,
                 hp: HParams, first_layer: int = 1) -> Tuple[np.ndarray, np.ndarray]:
    """Softmax prediction: a single pass, then the most probable class (the largest
    logit; lowest class on ties).  Returns ``(logits[n, C], pred[n])``."""
    A = head_features(layers, x_base, n_classes, hp, first_layer)
    logits = A @ head.W.T + head.b
    return logits, np.argmax(logits, axis=1).astype(np.int32)


# ----------------------------------------------------------------------------
# Performance-Optimised PFF (the PFF variant with a classification goodness)
# ----------------------------------------------------------------------------
def po_layer_step(L: Layer, head: Head, x: np.ndarray, y: np.ndarray, hp: HParams,
                  head_hp: HParams, normalised: bool = False):
    """One step of Performance-Optimised PFF on one layer (Sec. 4 "PFF with a new
    goodness function"): a softmax classifier is attached to the layer, and both
    are trained by backpropagation through those two layers only, on the mean
    cross-entropy of the labels (no negative data).  Readings: the classifier
    takes the layer's activities h as they are; the layer input is normalised
    as for FF.  Returns ``(loss, h, logits, dW, db, dWc, dbc)``, where h (the
    next layer's input) uses the weights before the update; mutates L and head.
    """
    xh, z, h, _ = layer_forward(L.W, L.b, x, hp.norm_eps, normalised, hp.bf16)
    logits = h @ head.W.T + head.b
    loss, d, _ = softmax_xent(logits, np.asarray(y, dtype=np.int64))
    dWc = d.T @ h
    dbc = d.sum(axis=0)
    dh = d @ head.W
    dz = dh * (z > 0)
    dzc = bf16_round(dz) if hp.bf16 else dz
    dW = dzc.T @ xh
    db = dz.sum(axis=0)
    L.t += 1
    L.W, L.mW, L.vW = adam(L.W, L.mW, L.vW, dW, L.t, hp.lr, hp.beta1, hp.beta2, hp.adam_eps)
    L.b, L.mb, L.vb = adam(L.b, L.mb, L.vb, db, L.t, hp.lr, hp.beta1, hp.beta2, hp.adam_eps)
    head.t += 1
    head.W, head.mW, head.vW = adam(head.W, head.mW, head.vW, dWc, head.t, head_hp.lr,
                                    head_hp.beta1, head_hp.beta2, head_hp.adam_eps)
    head.b, head.mb, head.vb = adam(head.b, head.mb, head.vb, dbc, head.t, head_hp.lr,
                                    head_hp.beta1, head_hp.beta2, head_hp.adam_eps)
    return loss, h, logits, dW, db, dWc, dbc


def po_train_pipelined(layers: List[Layer], heads: List[Head], x_base, y, n_classes: int,
                       chunk_pairs: int, epochs: int, hp: HParams, head_hp: HParams,
                       on_step=None) -> np.ndarray:
    """Performance-Optimised PFF over chunks in the layer-per-stage pipeline: layer
    l trains chunk c on layer l-1's activities of chunk c (computed before that
    step's update), as the FF pipeline does.  Layer 0 sees the neutrally
    labelled input (a reading: no label is given to a network that predicts it).
    Returns the loss trace ``[L, epochs * n_chunks]``.  ``on_step(l, layer,
    head, x, y, result)``, if given, sees copies of the layer and its classifier
    before each step, the step's input and labels, and what po_layer_step
    returned (test bookkeeping; no effect on results)."""
    chunks = chunk_bounds(x_base.shape[0], chunk_pairs)
    trace = np.zeros((len(layers), epochs * len(chunks)))
    for e in range(epochs):
        for ci, (s, b) in enumerate(chunks):
            a = embed_neutral(x_base[s:s + b], n_classes)
            for li, (L, Hd) in enumerate(zip(layers, heads)):
                pre = (L.copy(), Hd.copy(), a) if on_step else None
                res = po_layer_step(L, Hd, a, y[s:s + b], hp, head_hp)
                if on_step:
                    on_step(li, pre[0], pre[1], pre[2], y[s:s + b], res)
                loss, a = res[0], res[1]
                trace[li, e * len(chunks) + ci] = loss
    return trace


def po_train_sequential(layers: List[Layer], heads: List[Head], x_base, y, n_classes: int,
                        chunk_pairs: int, epochs: int, hp: HParams,
                        head_hp: HParams, on_step=None) -> np.ndarray:
    """Performance-Optimised training one layer after another (the sequential FF
    schedule of Sec. 3): layer l takes all its steps over the chunks, then its
    output with its final weights is the next layer's input.  Returns the loss
    trace ``[L, epochs * n_chunks]``.  ``on_step`` as for po_train_pipelined."""
    chunks = chunk_bounds(x_base.shape[0], chunk_pairs)
    trace = np.zeros((len(layers), epochs * len(chunks)))
    a_all = embed_neutral(x_base, n_classes)
    for li, (L, Hd) in enumerate(zip(layers, heads)):
        for e in range(epochs):
            for ci, (s, b) in enumerate(chunks):
                pre = (L.copy(), Hd.copy()) if on_step else None
                res = po_layer_step(L, Hd, a_all[s:s + b], y[s:s + b], hp, head_hp)
                if on_step:
                    on_step(li, pre[0], pre[1], a_all[s:s + b], y[s:s + b], res)
                trace[li, e * len(chunks) + ci] = res[0]
        a_all = layer_forward(L.W, L.b, a_all, hp.norm_eps, False, hp.bf16)[2]
    return trace


def po_predict(layers: Sequence[Layer], heads: Sequence[Head], x_base: np.ndarray,
               n_classes: int, hp: HParams, all_layers: bool = True):
    """Prediction of a Performance-Optimised network: one neutral-label pass; the
    last layer's classifier logits, or (reading for "all layers") the sum of every
    layer's classifier logits.  Returns ``(logits[n, C], pred[n])``, lowest class
    on ties."""
    a = embed_neutral(x_base, n_classes)
    total = np.zeros((x_base.shape[0], heads[0].W.shape[0]))
    for li, (L, Hd) in enumerate(zip(layers, heads)):
        _, _, a, _ = layer_forward(L.W, L.b, a, hp.norm_eps, False, hp.bf16)
        z = a @ Hd.W.T + Hd.b
        total = total + z if all_layers else z
    return total, np.argmax(total, axis=1).astype(np.int32)


# ----------------------------------------------------------------------------
# Training schedules over chunks (Sec. 3 sequential FF, Sec. 4.1 Alg. 1)
# ----------------------------------------------------------------------------
def chunk_bounds(n: int, chunk_pairs: int) -> List[Tuple[int, int]]:
    """Chunks of ``chunk_pairs`` samples in order; the last one is ragged."""
    return [(s, min(chunk_pairs, n - s)) for s in range(0, n, chunk_pairs)]


def chunk_input(x_base, y, y_neg, s: int, b: int, n_classes: int) -> np.ndarray:
    """Concatenated rows of one chunk: b positive rows, then the b negative rows."""
    xs = x_base[s:s + b]
    return np.concatenate([embed_labels(xs, y[s:s + b], n_classes),
                           embed_labels(xs, y_neg[s:s + b], n_classes)])


def train_sequential(layers: List[Layer], x_base, y, y_neg, n_classes: int, chunk_pairs: int,
                     epochs: int, hp: HParams, on_step=None) -> np.ndarray:
    """Train the layers one after another ("Sequential Training", Sec. 3).

    Layer l runs ``epochs`` passes over all chunks, then its output on the
    whole set -- one forward pass with its final weights, as the ``x <- layer(x)``
    step of Alg. 2 -- becomes layer l+1's input.  Returns the loss trace
    ``[n_layers, epochs * n_chunks]``.  Mutates ``layers``.  ``on_step(l, result)``,
    if given, sees every step's StepResult (test bookkeeping; no effect on results).
    """
    chunks = chunk_bounds(x_base.shape[0], chunk_pairs)
    trace = np.zeros((len(layers), epochs * len(chunks)))
    acts = [chunk_input(x_base, y, y_neg, s, b, n_classes) for s, b in chunks]
    for li, L in enumerate(layers):
        for e in range(epochs):
            for ci, (s, b) in enumerate(chunks):
                r = layer_step(L, acts[ci], b, hp)
                trace[li, e * len(chunks) + ci] = r.loss
                if on_step:
                    on_step(li, r)
        if li + 1 < len(layers):
            acts = [layer_forward(L.W, L.b, a, hp.norm_eps, False, hp.bf16)[2] for a in acts]
    return trace


def train_pipelined(layers: List[Layer], x_base, y, y_neg, n_classes: int, chunk_pairs: int,
                    epochs: int, hp: HParams, order: str = "chunk_major",
                    on_step=None) -> np.ndarray:
    """Layer-per-stage pipeline at chunk granularity (Single-Layer PFF, Sec. 4.1, Alg. 1).

    Each layer trains on the chunks in order; layer l+1 trains on chunk c once
    layer l has emitted its activities for chunk c.  Reading of the handoff
    (the paper exchanges layers per chapter; Sec. 6 proposes per-batch
    exchange): layer l+1's input for chunk c is the activity ``h`` of layer l's
    step on chunk c, computed with layer l's weights before that step's
    update.  The result depends only on the dependencies (l-1, c) -> (l, c)
    and (l, c-1) -> (l, c); ``order`` picks one topological order
    ("chunk_major", "layer_major" or "wavefront") to demonstrate that.  With
    ``epochs > 1`` the chunk stream is the chunk list repeated.  Returns the
    loss trace ``[n_layers, epochs * n_chunks]``.  Mutates ``layers``.
    ``on_step(l, result)``, if given, sees every step's StepResult (test
    bookkeeping; no effect on results).
    """
    chunks = chunk_bounds(x_base.shape[0], chunk_pairs) * epochs
    nl, nc = len(layers), len(chunks)
    if order == "chunk_major":
        seq = [(l, c) for c in range(nc) for l in range(nl)]
    elif order == "layer_major":
        seq = [(l, c) for l in range(nl) for c in range(nc)]
    elif order == "wavefront":
        seq = [(l, d - l) for d in range(nl + nc - 1) for l in range(nl) if 0 <= d - l < nc]
    else:
        raise ValueError(order)
    trace = np.zeros((nl, nc))
    inputs = {}
    for l, c in seq:
        s, b = chunks[c]
        x = chunk_input(x_base, y, y_neg, s, b, n_classes) if l == 0 else inputs.pop((l, c))
        r = layer_step(layers[l], x, b, hp)
        trace[l, c] = r.loss
        if on_step:
            on_step(l, r)
        if l + 1 < nl:
            inputs[(l + 1, c)] = r.h
    return trace
