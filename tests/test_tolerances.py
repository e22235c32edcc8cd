"""The parity bars themselves (tests/parity.py), checked on the CPU.

Two properties keep a bar honest: a correct implementation in fp32, with its
own summation order, passes it; and the oracle with a plausible mistake
planted in it fails it.  The fp32 step below is written here only for that
purpose (NumPy float32, BLAS summation order); the mistakes are planted in
copies of the oracle's step, never in the oracle itself.
"""
import numpy as np
import pytest

import oracle as O
from ffinputs import make_data, make_weights, random_labels
from parity import assert_goodness, assert_weights, grad_magnitudes, ill_conditioned

F32 = np.float32


def _fp32_steps(W, b, x, n_pos, k, hp):
    """k FF steps evaluated in float32 throughout."""
    W, b = W.astype(F32), b.astype(F32)
    mW, vW, mb, vb = (np.zeros_like(W), np.zeros_like(W), np.zeros_like(b), np.zeros_like(b))
    x = x.astype(F32)
    xh = x / (np.sqrt((x * x).sum(1, keepdims=True)) + F32(hp.norm_eps))
    for t in range(1, k + 1):
        h = np.maximum(xh @ W.T + b, F32(0))
        g = (h * h).sum(1)
        s = np.empty_like(g)
        s[:n_pos] = -1.0 / (1.0 + np.exp(g[:n_pos] - hp.theta)) / n_pos
        s[n_pos:] = 1.0 / (1.0 + np.exp(hp.theta - g[n_pos:])) / (len(g) - n_pos)
        dz = (2 * s)[:, None].astype(F32) * h
        for p, m, v, gr in ((W, mW, vW, dz.T @ xh), (b, mb, vb, dz.sum(0))):
            m[...] = F32(hp.beta1) * m + F32(1 - hp.beta1) * gr
            v[...] = F32(hp.beta2) * v + F32(1 - hp.beta2) * gr * gr
            mh = m / F32(1 - hp.beta1 ** t)
            vh = v / F32(1 - hp.beta2 ** t)
            p -= F32(hp.lr) * mh / (np.sqrt(vh) + F32(hp.adam_eps))
    return W, b, g


def _oracle_steps(W, b, x, n_pos, k, hp, grads=None):
    L = O.Layer.from_params(W, b)
    gW, mW, gb, mb = [], [], [], []
    for _ in range(k):
        r = O.layer_step(L, x, n_pos, hp)
        a, c = grad_magnitudes(r)
        gW.append(r.dW), mW.append(a), gb.append(r.db), mb.append(c)
    return L, r, gW, mW, gb, mb


CASES = [  # (data seed, weight seed, rows per half, d_in, d_out, steps)
    (7, 8, 96, 64, 136, 1),     # the smoke step
    (0, 1, 512, 784, 500, 3),   # the 784->500 layer of the small training config
    (30, 31, 150, 200, 260, 5),
]


@pytest.mark.parametrize("case", CASES)
def test_fp32_implementation_passes(case):
    sd, sw, n, d_in, d_out, k = case
    x_base, y, y_neg = make_data(sd, n, d_in)
    (W, b), = make_weights(sw, (d_in, d_out))
    x = np.concatenate([O.embed_labels(x_base, y, 10), O.embed_labels(x_base, y_neg, 10)])
    hp = O.HParams(theta=2.0, lr=0.03)
    W32, b32, g32 = _fp32_steps(W, b, x, n, k, hp)
    L, r, gW, mW, gb, mb = _oracle_steps(W, b, x, n, k, hp)
    assert_goodness(g32, r.g)
    assert_weights(W32, L.W, gW, mW, "W", lr=hp.lr, adam_eps=hp.adam_eps)
    assert_weights(b32, L.b, gb, mb, "b", lr=hp.lr, adam_eps=hp.adam_eps)
    assert ill_conditioned(gW, mW, hp.lr, hp.adam_eps, 1e-3 * np.abs(L.W) + 1e-6).mean() < 1e-3


def test_smoke_step_needs_the_adam_amplification_rule():
    """The smoke step has one weight whose gradient is 0.9e-8, next to Adam's
    eps: g/(|g| + eps) there moves by lr/4 per unit of relative gradient error,
    so rounding a correct fp32 implementation may make moves that weight past
    1e-3 relative.  The rule sets aside that element and nothing else."""
    x_base, y, y_neg = make_data(7, 96, 64)
    (W, b), = make_weights(8, (64, 136))
    x = np.concatenate([O.embed_labels(x_base, y, 10), O.embed_labels(x_base, y_neg, 10)])
    hp = O.HParams(theta=2.0, lr=0.03)
    L, r, gW, mW, _, _ = _oracle_steps(W, b, x, 96, 1, hp)
    plain = ill_conditioned(gW, mW)
    amp = ill_conditioned(gW, mW, hp.lr, hp.adam_eps, 1e-3 * np.abs(L.W) + 1e-6)
    assert plain.sum() == 0
    assert list(zip(*np.nonzero(amp))) == [(40, 25)]
    assert abs(r.dW[40, 25]) < 2e-8


@pytest.mark.parametrize("mistake", ["loss_all_rows", "neg_sign", "drop_bias", "no_bias_corr",
                                     "no_normalise", "transposed_dz"])
def test_planted_oracle_mistakes_fail(mistake):
    x_base, y, y_neg = make_data(30, 150, 200)
    (W, b), = make_weights(31, (200, 260))
    b = b + 0.05
    x = np.concatenate([O.embed_labels(x_base, y, 10), O.embed_labels(x_base, y_neg, 10)])
    hp = O.HParams(theta=2.0, lr=0.03)
    L, r, gW, mW, gb, mb = _oracle_steps(W, b, x, 150, 2, hp)

    M = O.Layer.from_params(W, b)
    for _ in range(2):
        xh = x if mistake == "no_normalise" else O.l2_normalise(x, hp.norm_eps)
        z = xh @ M.W.T + (0 if mistake == "drop_bias" else M.b)
        h = np.maximum(z, 0)
        g = (h * h).sum(1)
        _, dg = O.ff_loss(g, 150, hp.theta)
        if mistake == "loss_all_rows":
            dg = dg / 2
        if mistake == "neg_sign":
            dg[150:] = -dg[150:]
        dz = 2 * dg[:, None] * h
        if mistake == "transposed_dz":
            dz = dz[::-1]
        M.t += 1
        t = 1 if mistake == "no_bias_corr" else M.t
        M.W, M.mW, M.vW = O.adam(M.W, M.mW, M.vW, dz.T @ xh, t, hp.lr, hp.beta1, hp.beta2,
                                 hp.adam_eps)
        M.b, M.mb, M.vb = O.adam(M.b, M.mb, M.vb, dz.sum(0), t, hp.lr, hp.beta1, hp.beta2,
                                 hp.adam_eps)
    with pytest.raises(AssertionError):
        assert_weights(M.W, L.W, gW, mW, "W", lr=hp.lr, adam_eps=hp.adam_eps)
        assert_weights(M.b, L.b, gb, mb, "b", lr=hp.lr, adam_eps=hp.adam_eps)


@pytest.mark.parametrize("mistake", ["no_relu_mask", "grad_sign", "no_head_bias_grad",
                                     "label_shift"])
def test_planted_po_mistakes_fail(mistake):
    """The performance-optimised bars (weights with the Adam-amplified set aside,
    plus the first moments) catch mistakes planted in a copy of the step."""
    x_base, y, _ = make_data(120, 150, 64)
    x = O.embed_neutral(x_base, 10)
    (W, b), = make_weights(121, (64, 96))
    rng = np.random.default_rng(122)
    Wc, bc = rng.uniform(-0.2, 0.2, (10, 96)), rng.uniform(-0.1, 0.1, 10)
    hp, hhp = O.HParams(lr=0.01), O.HParams(lr=1e-3)
    L, Hd = O.Layer.from_params(W, b), O.Head.from_params(Wc, bc)
    M, MH = O.Layer.from_params(W, b), O.Head.from_params(Wc, bc)
    gW, mW = [], []
    for _ in range(2):
        xh, z, h, _ = O.layer_forward(L.W, L.b, x, 1e-8)
        _, d, _ = O.softmax_xent(h @ Hd.W.T + Hd.b, y)
        mW.append(np.abs((d @ Hd.W) * (z > 0)).T @ np.abs(xh))
        gW.append(O.po_layer_step(L, Hd, x, y, hp, hhp)[3])
        # the copy with the mistake
        xh, z, h, _ = O.layer_forward(M.W, M.b, x, 1e-8)
        yy = (y + 1) % 10 if mistake == "label_shift" else y
        _, d, _ = O.softmax_xent(h @ MH.W.T + MH.b, yy)
        if mistake == "grad_sign":
            d = -d
        dz = d @ MH.W if mistake == "no_relu_mask" else (d @ MH.W) * (z > 0)
        dbc = np.zeros(10) if mistake == "no_head_bias_grad" else d.sum(axis=0)
        M.t += 1
        MH.t += 1
        M.W, M.mW, M.vW = O.adam(M.W, M.mW, M.vW, dz.T @ xh, M.t, 0.01, 0.9, 0.999, 1e-8)
        M.b, M.mb, M.vb = O.adam(M.b, M.mb, M.vb, dz.sum(0), M.t, 0.01, 0.9, 0.999, 1e-8)
        MH.W, MH.mW, MH.vW = O.adam(MH.W, MH.mW, MH.vW, d.T @ h, MH.t, 1e-3, 0.9, 0.999, 1e-8)
        MH.b, MH.mb, MH.vb = O.adam(MH.b, MH.mb, MH.vb, dbc, MH.t, 1e-3, 0.9, 0.999, 1e-8)
    with pytest.raises(AssertionError):
        assert_weights(M.mW, L.mW, gW, mW, "mW")
        assert_weights(M.W, L.W, gW, mW, "W", lr=0.01)
        assert_weights(MH.b, Hd.b, [np.ones(10)], [np.ones(10)], "bc", lr=1e-3)


def test_r1_slack_covers_fp32_normalisation():
    """The bf16 goodness allowance for open R1 roundings (rows whose normalised
    input has an element within 2^-18 of a bf16 rounding change) covers what an
    fp32 normalisation does to the goodness, row by row, and is zero on every
    other row.  The input is sparse and narrow, as in the bf16 forward test
    where an fp32 normalisation moves a row by 1.2e-3."""
    from parity import r1_goodness_slack
    from ffinputs import random_matrix
    rows, d_in, d_out = 4000, 72, 600
    x = random_matrix(rows + 3 * d_in, rows, d_in, 0, 1, 0.6)
    (W, b), = make_weights(d_out + 5, (d_in, d_out))
    xh64 = O.l2_normalise(x, 1e-8)
    _, _, h_ref, g_ref = O.layer_forward(W, b, x, 1e-8, bf16=True)
    Wb = O.bf16_round(W)
    slack = r1_goodness_slack(Wb, xh64, h_ref)
    # the allowance is confined to rows with an open element
    lo = O.bf16_round(xh64 * (1 - 2.0 ** -18))
    hi = O.bf16_round(xh64 * (1 + 2.0 ** -18))
    open_rows = (lo != hi).any(axis=1)
    assert np.all(slack[~open_rows] == 0) and np.all(slack[open_rows] > 0)
    assert 0 < open_rows.sum() < rows // 4
    # every open element rounded the other way at once stays inside it
    for other in (lo, hi):
        _, _, _, g_alt = O.layer_forward(W, b, other, 1e-8, normalised=True, bf16=True)
        assert np.all(np.abs(g_alt - g_ref) <= slack + 1e-12 * np.abs(g_ref))
    # an fp32 normalisation (one summation order) passes the bar with it
    x32 = x.astype(np.float32)
    s32 = np.float32(1) / (np.sqrt((x32 * x32).sum(axis=1, dtype=np.float32)) + np.float32(1e-8))
    xh32 = O.bf16_round((x32 * s32[:, None]).astype(np.float64))
    _, _, _, g32 = O.layer_forward(W, b, xh32, 1e-8, normalised=True, bf16=True)
    assert_goodness(g32, g_ref, slack=slack)
    # the activity allowance covers the same extremes element by element
    from parity import r1_activity_slack
    D = r1_activity_slack(Wb, xh64)
    assert np.all(D[~open_rows] == 0)
    for other in (lo, hi, xh32):
        _, _, h_alt, _ = O.layer_forward(W, b, other, 1e-8, normalised=True, bf16=True)
        assert np.all(np.abs(h_alt - h_ref) <= D + 1e-12 * np.abs(h_ref))


def test_adam_propagation_bound_covers_perturbed_gradients():
    """Conditioning.E bounds the Adam updates' response to gradient errors: the
    oracle's own Adam, run over a recorded sequence of step gradients with each
    perturbed by up to kappa times its sum of |terms| (random signs), ends
    within kappa lr E of the unperturbed run, element by element; the sign-flip
    flags are those of ill_conditioned; at step 1 E is the derivative of
    g/(|g| + eps)."""
    from parity import Conditioning
    x_base, y, y_neg = make_data(7, 96, 64)
    (W, b), = make_weights(8, (64, 136))
    x = np.concatenate([O.embed_labels(x_base, y, 10), O.embed_labels(x_base, y_neg, 10)])
    hp = O.HParams(theta=2.0, lr=0.03)
    _, _, gW, mW, _, _ = _oracle_steps(W, b, x, 96, 6, hp)
    c = Conditioning.of(gW, mW)
    np.testing.assert_array_equal(c.cond, ill_conditioned(gW, mW))
    c1 = Conditioning.of(gW[:1], mW[:1])
    # (the step-1 terms cancel to eps/(|g| + eps)^2: about 1e-9 relative rounding)
    np.testing.assert_allclose(c1.E, 1e-8 * mW[0] / (np.abs(gW[0]) + 1e-8) ** 2, rtol=1e-8)

    def adam_run(grads):
        p, m, v = np.zeros_like(grads[0]), np.zeros_like(grads[0]), np.zeros_like(grads[0])
        for t, g in enumerate(grads, 1):
            p, m, v = O.adam(p, m, v, g, t, hp.lr, hp.beta1, hp.beta2, hp.adam_eps)
        return p
    base = adam_run(gW)
    rng = np.random.default_rng(3)
    kappa = 1e-7
    worst = 0.0
    for _ in range(4):
        pert = [g + kappa * m * rng.choice([-1.0, 1.0], g.shape) for g, m in zip(gW, mW)]
        diff = np.abs(adam_run(pert) - base)
        bound = kappa * hp.lr * c.E
        ok = ~c.cond
        assert np.all(diff[ok] <= 1.05 * bound[ok] + 1e-15)
        worst = max(worst, np.max(diff[ok] / np.maximum(bound[ok], 1e-300)))
    assert worst > 0.2  # the bound is not vacuous


@pytest.mark.parametrize("bf16", [False, True])
def test_run_bar_needed_by_float32_and_catches_mistakes(bf16, monkeypatch):
    """The run-level bar of multi-layer schedules (assert_run_like_fp32).  A
    float32 evaluation (tests/fp32_eval.py) of 4-epoch, 2-chapter training
    breaks the single-step elementwise bar in its hidden layers (in fp32 not in
    layer 0, whose inputs are given; in bf16 also there, since R3 rounds c h from
    an fp32 product), which is why multi-layer runs are bounded by the run-level
    bar; another float32 summation order passes that bar against the first;
    and the same run with a planted mistake fails it."""
    import fp32_eval as FE
    from parity import Conditioning, assert_run_like_fp32
    dims = (64, 96, 80, 48)
    x_base, y, _ = make_data(130, 300, 64)
    negs = [random_labels(131 + c, 300)[1] for c in range(2)]
    params = make_weights(139, dims)
    hp = O.HParams(lr=0.03, bf16=bf16)

    def run(Ls, obs=None):
        return O.chapter_train(Ls, x_base, y, negs, 10, 64, 4, 2, 2, hp, on_step=obs)
    refs = [O.Layer.from_params(W, b) for W, b in params]
    conds = [Conditioning() for _ in refs]

    def obs(l, r):
        conds[l].add(r.dW, grad_magnitudes(r)[0])
    t_ref = run(refs, obs)

    def f32(split=False, mistake=None):
        monkeypatch.setattr(FE, "SPLIT", split)
        monkeypatch.setattr(FE, "MISTAKE", mistake)
        with FE.fp32_evaluation():
            Ls = FE.layers32(params)
            return Ls, run(Ls)
    A, tA = f32()
    B, tB = f32(split=True)
    rel = 2e-3 if bf16 else 1e-3
    offs = []
    for L, R, c in zip(A, refs, conds):
        err = np.abs(L.W - R.W)
        offs.append(int(((err > rel * np.abs(R.W) + 1e-6 + 1e-5 * hp.lr * c.E) & ~c.cond).sum()))
    assert max(offs[1:]) > 0 and (bf16 or offs[0] == 0), offs
    pair = lambda Ls: [(L.W, L.mW) for L in Ls]  # noqa: E731
    assert_run_like_fp32(pair(B), pair(A), refs, conds, tB, tA, t_ref, hp.lr, bf16=bf16)
    for mistake in ("neg_sign", "no_bias_corr"):
        M, tM = f32(split=True, mistake=mistake)
        with pytest.raises(AssertionError):
            assert_run_like_fp32(pair(M), pair(A), refs, conds, tM, tA, t_ref, hp.lr, bf16=bf16)
