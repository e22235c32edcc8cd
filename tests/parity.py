"""Tolerances of the GPU-vs-oracle comparisons (shared by the GPU tests and the bench).

fp32 path:
  goodness, scores: |dg| <= 1e-4 |g_ref| + 1e-7 max|g_ref|
  loss:             |dL| <= 1e-4 |L_ref|
  activities h:     |dh| <= 1e-4 |h_ref| + 1e-5 max|h_ref| (fp32 contraction over
                    d_in terms of unit-norm rows)
  weights after k Adam steps: |dW| <= 1e-3 |W_ref| + 1e-6 + 1e-5 lr E outside the
                    ill-conditioned set, i.e. elements whose oracle gradient had
                    0 < |g| < 1e-5 sum|terms| at some step (Adam's first steps move
                    by about lr*sign(g), so a gradient whose sum cancels down to
                    rounding-noise level can flip its update in any fp32
                    implementation); that set must be at most 1e-3 of the tensor.
                    E (Conditioning) bounds to first order how far the Adam
                    updates carry a gradient error of sum|terms| per step.
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
    """Per-element bookkeeping of one Adam-updated tensor over a run, fed every
    update's oracle gradient g and term magnitudes mag = sum of |terms|:

    * cond: the sign-flip set of ill_conditioned (0 < |g| < 1e-5 mag at some step);
    * E: a first-order bound on how far a gradient error of at most mag per
      step can move the parameter through the Adam updates, per unit learning
      rate (the bar multiplies it by lr and by the gradient allowance 1e-5).

    Adam's step t applies u_t = m_hat/(sqrt(v_hat) + eps), with
    m = beta1 m + (1 - beta1) g and v = beta2 v + (1 - beta2) g^2.  An error d_s
    in the gradient of step s <= t moves u_t by
      d_s [(1-beta1) beta1^(t-s) / (bc1 (sqrt(v_hat) + eps))
           - m_hat (1-beta2) beta2^(t-s) g_s / (bc2 sqrt(v_hat) (sqrt(v_hat) + eps)^2)]
    (bc1, bc2 the bias corrections of step t).  The term of the current step is
    taken with its sign (at t = 1 it is eps/(|g| + eps)^2, so the nearly
    sign-like first update is insensitive unless |g| is near eps); the terms
    of earlier steps, carried by the moments, are bounded in absolute value
    through the running sums A = sum beta1^(t-s) mag_s and
    B = sum beta2^(t-s) |g_s| mag_s.  E = sum over steps of the resulting bound
    on |du_t|.  It leaves out the feedback of weight differences into later
    gradients."""

    def __init__(self, beta1=0.9, beta2=0.999, adam_eps=1e-8):
        self.b1, self.b2, self.eps = beta1, beta2, adam_eps
        self.t = 0
        self.cond = self.E = None

    def add(self, grad, mag):
        g = np.asarray(grad, np.float64)
        e = np.asarray(mag, np.float64)
        b1, b2, eps = self.b1, self.b2, self.eps
        if self.t == 0:
            z = np.zeros_like(g)
            self.cond = np.zeros(g.shape, bool)
            self.m, self.v, self.A, self.B, self.E = z.copy(), z.copy(), z.copy(), z.copy(), z
            self.g_prev, self.e_prev = z, z
        self.t += 1
        t = self.t
        self.A = b1 * (self.A + self.e_prev)
        self.B = b2 * (self.B + np.abs(self.g_prev) * self.e_prev)
        self.m = b1 * self.m + (1 - b1) * g
        self.v = b2 * self.v + (1 - b2) * g * g
        bc1, bc2 = 1 - b1 ** t, 1 - b2 ** t
        mh = self.m / bc1
        sv = np.sqrt(self.v / bc2)
        den = np.where(sv > 0, sv, 1.0) * (sv + eps) ** 2
        same = np.abs((1 - b1) / (bc1 * (sv + eps)) - mh * (1 - b2) * g / (bc2 * den)) * e
        carried = ((1 - b1) * self.A / (bc1 * (sv + eps))
                   + np.abs(mh) * (1 - b2) * self.B / (bc2 * den))
        self.E = self.E + same + carried
        a = np.abs(g)
        self.cond = self.cond | ((a > 0) & (a < 1e-5 * e))
        self.g_prev, self.e_prev = g, e

    @staticmethod
    def of(grads, mags, adam_eps=1e-8):
        c = Conditioning(adam_eps=adam_eps)
        for g, m in zip(grads, mags):
            c.add(g, m)
        return c


def assert_weights(W, ref, grads, mags, what="W", rel=1e-3, outliers=0.0, outlier_rel=0.0,
                   lr=None, adam_eps=1e-8, grad_rel=1e-5):
    """Weights (or Adam moments) after k Adam steps (see the module docstring).

    The bar is |dW| <= rel |W_ref| + 1e-6 outside the sign-flip set (at most
    1e-3 of the elements).  For a parameter (`lr` given) it adds
    grad_rel lr E: the Adam updates' first-order response to a gradient error
    of grad_rel times the sum of |terms| at every step (Conditioning; grad_rel
    1e-5 is the gradient allowance of the sign-flip rule).  The moments are
    linear in the gradients and take no such term.  `grads`, `mags`: the
    lists of every update's oracle gradient and term magnitudes, or a
    Conditioning that has seen them (then `mags` is not used).

    `outliers` (bf16 comparisons only): the fraction of elements allowed to
    exceed the bar, each still within `outlier_rel`.  With bf16 operands the two
    sides may round one operand of a gradient sum one bf16 ulp apart (the value
    sits within fp32 rounding of a bf16 rounding boundary), which moves that sum
    by 2^-8 of one term; Adam's per-element normalisation can turn that into a
    weight difference above the fp32 bar for the rare elements it touches."""
    W = np.asarray(W, np.float64)
    c = grads if isinstance(grads, Conditioning) else Conditioning.of(grads, mags, adam_eps)
    cond = c.cond
    assert cond.mean() <= 1e-3, f"{what}: ill-conditioned fraction {cond.mean():.2e} > 1e-3"
    err = np.abs(W - ref)
    tol = rel * np.abs(ref) + 1e-6
    if lr is not None:
        tol = tol + grad_rel * lr * c.E
    bad = (err > tol) & ~cond
    n_ok = int(outliers * bad.size)
    msg = (f"{what}: {bad.sum()} of {bad.size} off, worst abs {np.max(err[~cond]):.3g}, "
           f"worst excess over the bar {np.max((err - tol)[~cond]):.3g}")
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


def divergence(W, mW, ref, cond, rel=2e-3, lr=None, grad_rel=1e-5):
    """How far one trained layer lies from the oracle's: the fraction of weights
    beyond the single-step bar (rel |W_ref| + 1e-6 + grad_rel lr E, outside the
    sign-flip set), and the relative Frobenius distances of W and of its first
    Adam moment."""
    W, mW = np.asarray(W, np.float64), np.asarray(mW, np.float64)
    tol = rel * np.abs(ref.W) + 1e-6 + (grad_rel * lr * cond.E if lr is not None else 0.0)
    off = (np.abs(W - ref.W) > tol) & ~cond.cond
    return {"frac": float(off.mean()),
            "fro_W": float(np.linalg.norm(W - ref.W) / np.linalg.norm(ref.W)),
            "fro_mW": float(np.linalg.norm(mW - ref.mW) / max(np.linalg.norm(ref.mW), 1e-300))}


def assert_run_like_fp32(dev, f32, refs, conds, trace, trace32, trace_ref, lr, bf16=True,
                         factor=4.0):
    """A multi-layer run against the oracle, bounded by what a plain float32
    evaluation of the same run (tests/fp32_eval.py) does.

    dev, f32: per layer (W, mW) of the device run and of the float32
    evaluation; refs: the oracle's layers; conds: their Conditioning.  For
    every layer, each divergence metric of the device (fraction of weights
    past the single-step bar, 2e-3 relative in bf16 and 1e-3 in fp32 plus the
    propagated allowance; relative Frobenius distance of W and of the first
    moment) and the largest relative difference of its loss trace must be at
    most `factor` times the float32 evaluation's, plus a floor (1e-4 of the
    elements, 1e-6, 1e-5 for the trace).  Every layer also stays within the
    workload's weight bar of the oracle as a relative Frobenius distance: 5e-2
    in bf16, 1e-3 in fp32.

    Why a relative bar: a later layer trains on activities produced by layers
    that already differ slightly from the oracle's, and in bf16 those
    activities' roundings go the other way where they sit within evaluation
    error of a rounding boundary.  Neither is a per-step effect that a
    single-step bar covers, and both sides move different elements (their
    summation orders differ), but a correct evaluation moves about as many by
    about as much."""
    rel, cap = (2e-3, 5e-2) if bf16 else (1e-3, 1e-3)
    for i, ((W, mW), (W32, mW32), R, c) in enumerate(zip(dev, f32, refs, conds)):
        d = divergence(W, mW, R, c, rel=rel, lr=lr)
        e = divergence(W32, mW32, R, c, rel=rel, lr=lr)
        floors = {"frac": 1e-4, "fro_W": 1e-6, "fro_mW": 1e-6}
        for k, fl in floors.items():
            assert d[k] <= factor * e[k] + fl, \
                f"layer {i} {k}: device {d[k]:.3g} vs float32 evaluation {e[k]:.3g}"
        assert d["fro_W"] <= cap, f"layer {i}: relative Frobenius distance {d['fro_W']:.3g}"
        tr = np.asarray(trace, np.float64)[i]
        t32 = np.asarray(trace32, np.float64)[i]
        tref = np.asarray(trace_ref, np.float64)[i]
        dt = np.max(np.abs(tr - tref) / np.abs(tref))
        d32 = np.max(np.abs(t32 - tref) / np.abs(tref))
        assert dt <= factor * d32 + 1e-5, \
            f"layer {i} loss trace: device {dt:.3g} vs float32 evaluation {d32:.3g}"
