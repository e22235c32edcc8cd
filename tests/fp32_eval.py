"""A plain float32 evaluation of the FF step, for calibrating parity bars.

Test infrastructure: the same method as the oracle's layer step, evaluated in
NumPy float32 (BLAS summation order) instead of float64, with the same three
bf16 rounding points (R1 x_hat, R2 W, R3 dZ) in bf16 mode.  It shares no code
with the HIP path.  ``fp32_evaluation()`` swaps it for the oracle's step and
forward while a schedule of the oracle (train_pipelined, train_sequential,
chapter_train) runs, so the same schedule code drives it.

Why: in bf16 mode a hidden layer's input and dZ come from float32 products,
and every evaluation in a precision other than the oracle's float64 rounds
some of those operands to the other bf16 neighbour (they lie within its
evaluation error of a rounding boundary); after a few Adam steps the layers'
weights then differ from the oracle's by more than any per-element bar
derived for one step.  This evaluation measures how far a correct float32
implementation lands, which bounds what the device may do.
"""
import contextlib

import numpy as np

import oracle.ff_oracle as OF

F32 = np.float32

# Knobs for the tolerance tests only: SPLIT sums every product over its
# contraction in two halves (another float32 summation order); MISTAKE plants a
# named error in the step ("neg_sign": the negatives' gradient sign flipped,
# "no_bias_corr": Adam without bias correction).
SPLIT = False
MISTAKE = None


def _mm(a, b):
    if not SPLIT or a.shape[1] < 2:
        return a @ b
    k = a.shape[1] // 2
    return a[:, :k] @ b[:k] + a[:, k:] @ b[k:]


def _bf16(a):
    """Round float32 values to bfloat16 (nearest, ties to even), kept as float32."""
    u = np.ascontiguousarray(a, F32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000).astype(np.uint32).view(F32)


def forward32(W, b, x, norm_eps, normalised=False, bf16=False):
    x = np.asarray(x, F32)
    xh = x if normalised else x / (np.sqrt((x * x).sum(axis=1, keepdims=True)) + F32(norm_eps))
    Wm = np.asarray(W, F32)
    if bf16:
        xh, Wm = _bf16(xh), _bf16(Wm)
    z = _mm(xh, Wm.T) + np.asarray(b, F32)
    h = np.maximum(z, F32(0))
    return xh, z, h, (h * h).sum(axis=1)


def _softplus(t):
    return np.maximum(t, F32(0)) + np.log1p(np.exp(-np.abs(t)))


def _sigmoid(t):
    e = np.exp(-np.abs(t))
    return np.where(t >= 0, F32(1) / (F32(1) + e), e / (F32(1) + e))


def step32(L, x, n_pos, hp, normalised=False):
    """One FF step of layer L (float32 arrays) in float32; mutates L."""
    xh, _, h, g = forward32(L.W, L.b, x, hp.norm_eps, normalised, hp.bf16)
    n_neg = g.shape[0] - n_pos
    th = F32(hp.theta)
    loss = _softplus(th - g[:n_pos]).sum() / F32(n_pos) + _softplus(g[n_pos:] - th).sum() / F32(n_neg)
    dg = np.concatenate([-_sigmoid(th - g[:n_pos]) / F32(n_pos), _sigmoid(g[n_pos:] - th) / F32(n_neg)])
    dz = (F32(2) * dg)[:, None] * h
    if MISTAKE == "neg_sign":
        dg[n_pos:] = -dg[n_pos:]
        dz = (F32(2) * dg)[:, None] * h
    dW = _mm((_bf16(dz) if hp.bf16 else dz).T, xh)
    db = dz.sum(axis=0)
    L.t += 1
    t = L.t
    b1, b2 = F32(hp.beta1), F32(hp.beta2)
    for name, gr in (("W", dW), ("b", db)):
        p, m, v = getattr(L, name), getattr(L, "m" + name), getattr(L, "v" + name)
        m = b1 * m + (F32(1) - b1) * gr
        v = b2 * v + (F32(1) - b2) * gr * gr
        tc = 1 if MISTAKE == "no_bias_corr" else t
        p = p - F32(hp.lr) * (m / F32(1 - hp.beta1 ** tc)) / (np.sqrt(v / F32(1 - hp.beta2 ** tc))
                                                              + F32(hp.adam_eps))
        setattr(L, name, p)
        setattr(L, "m" + name, m)
        setattr(L, "v" + name, v)
    return OF.StepResult(h, g, float(loss), dW, db, xh, dg)


def layers32(params):
    """Oracle Layer objects holding float32 arrays, for the float32 evaluation."""
    out = []
    for W, b in params:
        W, b = np.array(W, F32), np.array(b, F32)
        out.append(OF.Layer(W, b, np.zeros_like(W), np.zeros_like(W), np.zeros_like(b),
                            np.zeros_like(b)))
    return out


@contextlib.contextmanager
def fp32_evaluation():
    """The oracle's schedules run float32 steps inside this block."""
    saved = OF.layer_step, OF.layer_forward
    OF.layer_step, OF.layer_forward = step32, forward32
    try:
        yield
    finally:
        OF.layer_step, OF.layer_forward = saved
