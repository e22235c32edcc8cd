"""Tolerances of the GPU-vs-oracle comparisons (shared by the GPU tests and the bench).

fp32 path:
  goodness, scores: |dg| <= 1e-4 |g_ref| + 1e-7 max|g_ref|
  loss:             |dL| <= 1e-4 |L_ref|
  activities h:     |dh| <= 1e-4 |h_ref| + 1e-5 max|h_ref| (fp32 contraction over
                    d_in terms of unit-norm rows)
  weights after k Adam steps: |dW| <= 1e-3 |W_ref| + 1e-6 outside the
                    ill-conditioned set, i.e. elements whose oracle gradient had
                    0 < |g| < 1e-5 sum|terms| at some step (Adam's first steps move
                    by about lr*sign(g), so a gradient whose sum cancels down to
                    rounding-noise level can flip its update in any fp32
                    implementation); that set must be at most 1e-3 of the tensor.
  labels:           bit-exact where the oracle's top-two gap is >= 1e-4 relative.
bf16 path (compared with the bf16-emulating oracle, which rounds the same three
  operands): goodness, scores and loss within 1e-3 relative (plus, for the
  forward, the slack of r1_goodness_slack on rows whose normalised input has an
  element the two sides may round either way); activities 1e-3
  relative + 1e-3 max|h| (an operand within fp32 rounding of a bf16 rounding
  boundary may round differently on the two sides); weights as fp32 with 2e-3;
  and against the fp32 oracle ||dW||_F <= 5e-2 ||W_ref||_F (the workload's bar).
"""
import numpy as np

from oracle import bf16_round


def assert_goodness(g, ref, rel=1e-4, what="goodness", slack=None):
    g = np.asarray(g, np.float64)
    ref = np.asarray(ref, np.float64)
    tol = rel * np.abs(ref) + 1e-7 * max(np.abs(ref).max(), 1e-30)
    if slack is not None:
        tol = tol + slack
    bad = np.abs(g - ref) > tol
    assert not bad.any(), f"{what}: {bad.sum()} of {bad.size} off, worst rel " \
                          f"{np.max(np.abs(g - ref) / (np.abs(ref) + 1e-30)):.3g}"


def bf16_ulp(x):
    """Spacing of bfloat16 values at |x| (8 significant bits): 2^(e - 8) for |x| in [2^(e-1), 2^e)."""
    _, e = np.frexp(np.abs(np.asarray(x, np.float64)))
    return np.ldexp(1.0, e - 8)


def r1_goodness_slack(Wb, xh, h, band=2.0 ** -18):
    """Per-row goodness allowance for R1 rounding decisions that fp32 leaves open.

    bf16 mode rounds the normalised layer input to bf16 (R1).  The device
    normalises in fp32, the oracle in fp64; an element whose exact value lies
    within ``band`` (relative) of a point where bf16 rounding changes may round
    to either neighbour, and both are results of the method in fp32 arithmetic
    (an fp32 norm over up to 2^12 terms and the scaling stay well inside 2^-18).
    Such an element moves each z_j by at most |W_ji| u_i (u_i its bf16 spacing),
    and for any shift d, |relu(z+d)^2 - relu(z)^2| <= 2 relu(z) |d| + d^2, so a
    row's goodness moves by at most sum_j (2 h_j D_j + D_j^2) with
    D_j = sum over its open elements i of |W_ji| u_i.

    Wb: [d_out, d_in] bf16-rounded weights; xh: [R, d_in] fp64 normalised input
    before rounding; h: [R, d_out] oracle activities.  Rows without an open
    element get 0."""
    xh = np.asarray(xh, np.float64)
    Wa = np.abs(np.asarray(Wb, np.float64))
    lo = bf16_round(xh * (1.0 - band))
    hi = bf16_round(xh * (1.0 + band))
    open_ = lo != hi
    slack = np.zeros(xh.shape[0])
    rows = np.nonzero(open_.any(axis=1))[0]
    if rows.size:
        U = np.where(open_[rows], bf16_ulp(hi[rows]), 0.0)  # [r, d_in]
        D = U @ Wa.T  # [r, d_out]
        slack[rows] = (2.0 * np.asarray(h, np.float64)[rows] * D + D * D).sum(axis=1)
    return slack


def r1_activity_slack(Wb, xh, band=2.0 ** -18):
    """Per-element activity allowance for open R1 roundings (see
    r1_goodness_slack): |dh_rj| <= D_rj = sum over row r's open elements i of
    |W_ji| u_i, since relu moves by at most the shift of z.  Returns [R, d_out]
    (zero on rows without an open element)."""
    xh = np.asarray(xh, np.float64)
    Wa = np.abs(np.asarray(Wb, np.float64))
    lo = bf16_round(xh * (1.0 - band))
    hi = bf16_round(xh * (1.0 + band))
    open_ = lo != hi
    D = np.zeros((xh.shape[0], Wa.shape[0]))
    rows = np.nonzero(open_.any(axis=1))[0]
    if rows.size:
        D[rows] = np.where(open_[rows], bf16_ulp(hi[rows]), 0.0) @ Wa.T
    return D


def assert_loss(l, ref, rel=1e-4):
    assert abs(float(l) - float(ref)) <= rel * abs(float(ref)), f"loss {l} vs {ref}"


def assert_acts(h, ref, rel=1e-4, floor=1e-5, slack=None):
    """|dh| <= rel |h_ref| + floor max|h_ref|.

    bf16 operands: a value that lies within fp32 rounding of a bf16 rounding
    boundary can round to neighbouring bf16 values on the two sides (the device
    computes it in fp32, the oracle in fp64); one such operand moves z by one bf16
    ulp (2^-8 relative) of one product term, about 1e-4 of max|h| at these
    shapes.  `slack` (bf16): r1_activity_slack, the per-element bound of that
    effect, added to the fp32 bar."""
    h = np.asarray(h, np.float64)
    tol = rel * np.abs(ref) + floor * max(np.abs(ref).max(), 1e-30)
    if slack is not None:
        tol = tol + slack
    bad = np.abs(h - ref) > tol
    assert not bad.any(), f"activities: {bad.sum()} of {bad.size} off, max abs err " \
                          f"{np.max(np.abs(h - ref)):.3g}"


def grad_magnitudes(r):
    """Sum of |terms| of every gradient element of an oracle step: (|dZ|^T |x_hat|, sum |dZ|)."""
    dz = np.abs(2.0 * r.dLdg[:, None] * r.h)
    return dz.T @ np.abs(r.xh), dz.sum(axis=0)


def ill_conditioned(grads, mags, lr=None, adam_eps=1e-8, tol=None, split=False):
    """Elements whose gradient was ill-conditioned at some step.

    A gradient element is a sum over the batch rows; rounding can change its
    sign only when |sum| is tiny against sum(|terms|).  Flagged: 0 < |g| <
    1e-5 sum(|terms|) (condition number above 1e5).  An exactly zero gradient
    (a feature that is zero in every row) gives an exactly zero Adam update on
    both sides and is not flagged.

    With `lr` (weights only), also flagged: elements whose Adam update
    amplifies the same rounding allowance beyond half the weight tolerance
    `tol`.  Adam's step g/(|g| + eps) has derivative eps/(|g| + eps)^2, so a
    gradient near eps in size turns an error e in g into a weight error of up
    to lr*eps*e/(|g| + eps)^2, with e = 1e-5 sum(|terms|) as above.  With
    split=True the two sets are returned apart: (sign-flip set, amplified set)."""
    cond = np.zeros(np.shape(grads[0]), bool)
    amp = np.zeros(np.shape(grads[0]), bool)
    for gr, mg in zip(grads, mags):
        a = np.abs(np.asarray(gr))
        mg = np.asarray(mg)
        cond |= (a > 0) & (a < 1e-5 * mg)
        if lr is not None:
            amp |= (a > 0) & (lr * adam_eps * 1e-5 * mg / (a + adam_eps) ** 2 > 0.5 * tol)
    return (cond, amp & ~cond) if split else cond | amp


class Conditioning:
    """The flags of ill_conditioned kept step by step, for runs too long to hold
    every step's gradients: add(grad, mag) per update of one tensor; the
    sign-flip flags are OR-ed, and for the Adam-amplified set the largest
    eps 1e-5 mag / (|g| + eps)^2 over the steps is kept, to be scaled by the
    learning rate when the set is taken."""

    def __init__(self, adam_eps=1e-8):
        self.eps = adam_eps
        self.cond = None
        self.q = None

    def add(self, grad, mag):
        a = np.abs(np.asarray(grad, np.float64))
        mg = np.asarray(mag, np.float64)
        c = (a > 0) & (a < 1e-5 * mg)
        q = np.where(a > 0, self.eps * 1e-5 * mg / (a + self.eps) ** 2, 0.0)
        self.cond = c if self.cond is None else self.cond | c
        self.q = q if self.q is None else np.maximum(self.q, q)

    def masks(self, lr, tol):
        """(sign-flip set, Adam-amplified set) as ill_conditioned(split=True)."""
        amp = np.zeros_like(self.cond) if lr is None else (lr * self.q > 0.5 * tol)
        return self.cond, amp & ~self.cond


def assert_weights(W, ref, grads, mags, what="W", rel=1e-3, outliers=0.0, outlier_rel=0.0,
                   lr=None, adam_eps=1e-8):
    """Weights after k Adam steps (see the module docstring).

    `lr`, `adam_eps`: pass them when W is a parameter updated by Adam with
    those settings (not for the moments), so elements whose update amplifies
    gradient rounding past the bar are set aside (see ill_conditioned).  The
    sign-flip set may hold at most 1e-3 of the elements, the amplified set at
    most 1e-2: the latter grows when gradients are small next to Adam's eps,
    and callers check the first moments (linear in the gradient, never
    amplified) beside the weights.

    `outliers` (bf16 comparisons only): the fraction of elements allowed to
    exceed `rel`, each still within `outlier_rel`.  With bf16 operands the two
    sides may round one operand of a gradient sum one bf16 ulp apart (the value
    sits within fp32 rounding of a bf16 rounding boundary), which moves that sum
    by 2^-8 of one term; Adam's per-element normalisation can turn that into a
    weight difference above the fp32 bar for the rare elements it touches.

    `grads` may instead be a Conditioning that has seen every update (then
    `mags` is not used)."""
    W = np.asarray(W, np.float64)
    if isinstance(grads, Conditioning):  # flags kept step by step (mags unused)
        cond, amp = grads.masks(lr, rel * np.abs(ref) + 1e-6)
    else:
        cond, amp = ill_conditioned(grads, mags, lr, adam_eps, rel * np.abs(ref) + 1e-6,
                                    split=True)
    assert cond.mean() <= 1e-3, f"{what}: ill-conditioned fraction {cond.mean():.2e} > 1e-3"
    assert amp.mean() <= 1e-2, f"{what}: Adam-amplified fraction {amp.mean():.2e} > 1e-2"
    flag = cond | amp
    err = np.abs(W - ref)
    bad = (err > rel * np.abs(ref) + 1e-6) & ~flag
    n_ok = int(outliers * bad.size)
    msg = f"{what}: {bad.sum()} of {bad.size} off, worst abs {np.max(err[~flag]):.3g}"
    assert bad.sum() <= n_ok, msg
    if bad.any():
        assert np.all(err[bad] <= outlier_rel * np.abs(ref[bad]) + 1e-5), msg


def decided(S_ref, rel=1e-4):
    """Rows whose oracle top-two score gap is at least `rel` relative."""
    top2 = np.sort(S_ref, axis=1)[:, -2:]
    return (top2[:, 1] - top2[:, 0]) >= rel * np.abs(top2[:, 1])


def assert_labels(pred, S_ref, pred_ref):
    ok = decided(S_ref)
    pred = np.asarray(pred)
    bad = (pred != pred_ref) & ok
    assert not bad.any(), f"labels: {bad.sum()} decided rows differ"
    return int(ok.sum())


def assert_negatives(y_neg, S_ref, y_ref, labels):
    """AdaptiveNEG labels: bit-exact where the oracle's two best wrong labels are
    at least 1e-4 apart (relative); elsewhere any wrong label tied with the best
    within that margin is valid."""
    S = np.array(S_ref, np.float64)
    n = np.arange(S.shape[0])
    inr = (labels >= 0) & (labels < S.shape[1])
    S[n[inr], labels[inr]] = -np.inf
    y_neg = np.asarray(y_neg)
    ok = decided(S)
    bad = (y_neg != y_ref) & ok
    assert not bad.any(), f"negatives: {bad.sum()} decided rows differ"
    assert not np.any(inr & (y_neg == labels)), "a true label was chosen as negative"
    best = S.max(axis=1)
    assert np.all(S[n, y_neg] >= best - 1e-4 * np.abs(best)), "an undecided row chose a weak label"
    return int(ok.sum())


def assert_rel_fro(W, ref, rel):
    d = np.linalg.norm(np.asarray(W, np.float64) - ref) / np.linalg.norm(ref)
    assert d <= rel, f"relative Frobenius error {d:.3g} > {rel}"
