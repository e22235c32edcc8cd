"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these tests compares the oracle with itself: they use hand-derived
worked examples (tests/golden/hand_cases.json), closed forms, central finite
differences, PyTorch-CPU autograd and torch.optim.Adam in float64 (library
routines, used here only), brute force on tiny inputs, and invariances.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle as O
from ffinputs import make_data, make_weights, random_labels, random_matrix

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_cases.json")))


def _layer(case):
    return np.array(case["W"], float), np.array(case["b"], float)


# ---------------------------------------------------------------- worked examples
@pytest.mark.parametrize("name", ["layer_identity_34", "layer_asymmetric"])
def test_forward_hand(name):
    c = GOLD[name]
    W, b = _layer(c)
    xh, z, h, g = O.layer_forward(W, b, np.array(c["x"]), c["norm_eps"])
    np.testing.assert_allclose(xh, c["x_hat"], rtol=0, atol=1e-15)
    np.testing.assert_allclose(h, c["h"], rtol=0, atol=1e-14)
    np.testing.assert_allclose(g, c["g"], rtol=0, atol=1e-14)


@pytest.mark.parametrize("name", ["norm_eps_placement", "zero_row"])
def test_normalise_hand(name):
    c = GOLD[name]
    np.testing.assert_allclose(O.l2_normalise(np.array(c["x"]), c["norm_eps"]), c["x_hat"],
                               rtol=0, atol=1e-15)


@pytest.mark.parametrize("name", ["loss_at_threshold", "loss_log3", "loss_half_means"])
def test_loss_hand(name):
    c = GOLD[name]
    loss, dg = O.ff_loss(np.array(c["g"]), c["n_pos"], c["theta"])
    assert abs(loss - c["loss"]) < 1e-14
    np.testing.assert_allclose(dg, c["dLdg"], rtol=0, atol=1e-14)


def test_adam_hand():
    c = GOLD["adam_two_steps"]
    p, m, v = np.array([c["p0"]]), np.zeros(1), np.zeros(1)
    for t, (gr, want) in enumerate(zip(c["grads"], c["p"]), start=1):
        p, m, v = O.adam(p, m, v, np.array([gr]), t, c["lr"], c["beta1"], c["beta2"], c["eps"])
        assert abs(p[0] - want) < 1e-16


def test_embed_hand():
    c = GOLD["embed"]
    x = O.embed_labels(np.array(c["x_base"]), np.array(c["labels"]), c["n_classes"])
    np.testing.assert_array_equal(x, c["x"])


def test_grad_hand():
    c = GOLD["grad_one_unit"]
    W, b = _layer(c)
    xh, _, h, g = O.layer_forward(W, b, np.array(c["x"]), c["norm_eps"])
    np.testing.assert_allclose(g, c["g"], atol=1e-15)
    loss, dg = O.ff_loss(g, c["n_pos"], c["theta"])
    assert abs(loss - c["loss"]) < 1e-14
    dW, db = O.layer_grads(xh, h, dg)
    np.testing.assert_allclose(dW, c["dW"], atol=1e-15)
    np.testing.assert_allclose(db, c["db"], atol=1e-15)


# ---------------------------------------------------------------- closed forms
def test_goodness_is_squared_norm_of_relu():
    rng = np.random.default_rng(5)
    z = rng.normal(size=(7, 11))
    h = np.maximum(z, 0)
    g = O.goodness(h)
    for r in range(7):
        assert abs(g[r] - sum(v * v for v in z[r] if v > 0)) < 1e-12


def test_loss_derivative_is_logistic():
    """d/dg softplus(theta-g) = -sigma(theta-g); d/dg softplus(g-theta) = sigma(g-theta)."""
    theta = 2.0
    g = np.array([-3.0, 0.1, 1.9, 2.0, 2.5, 40.0, 3.0, -1.0])
    n_pos = 4
    _, dg = O.ff_loss(g, n_pos, theta)
    e = 1e-6
    for r in range(len(g)):
        gp, gm = g.copy(), g.copy()
        gp[r] += e
        gm[r] -= e
        num = (O.ff_loss(gp, n_pos, theta)[0] - O.ff_loss(gm, n_pos, theta)[0]) / (2 * e)
        assert abs(num - dg[r]) < 1e-8
    # the logistic closed form, independently of the oracle's sigmoid
    for r in range(len(g)):
        sgn, n = (-1, n_pos) if r < n_pos else (1, len(g) - n_pos)
        want = sgn / (1.0 + math.exp(-sgn * (g[r] - theta))) / n
        assert abs(dg[r] - want) < 1e-15


def test_softplus_sigmoid_extremes():
    x = np.array([-800.0, -30.0, 0.0, 30.0, 800.0])
    sp = O.softplus(x)
    assert np.all(np.isfinite(sp))
    assert sp[-1] == 800.0 and sp[0] == 0.0
    assert abs(sp[2] - math.log(2)) < 1e-15
    s = O.sigmoid(x)
    assert s[0] == 0.0 and s[-1] == 1.0 and s[2] == 0.5


def test_normalise_unit_and_scale_invariant():
    x = random_matrix(3, 9, 37, 0, 1, p_zero=0.5).astype(float)
    xh = O.l2_normalise(x, 1e-8)
    np.testing.assert_allclose(np.linalg.norm(xh, axis=1), 1.0, atol=1e-7)
    np.testing.assert_allclose(O.l2_normalise(7.5 * x, 1e-8), xh, atol=1e-8)


def test_adam_first_step_closed_form():
    rng = np.random.default_rng(9)
    g = rng.normal(size=50) * 10.0 ** rng.integers(-6, 2, 50)
    p0 = rng.normal(size=50)
    p, _, _ = O.adam(p0, np.zeros(50), np.zeros(50), g, 1, 0.03, 0.9, 0.999, 1e-8)
    np.testing.assert_allclose(p, p0 - 0.03 * g / (np.abs(g) + 1e-8), rtol=0, atol=1e-15)


def test_bf16_round_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(2)
    v = np.concatenate([rng.normal(size=4000) * 10.0 ** rng.integers(-8, 8, 4000),
                        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 0.0])])
    v32 = v.astype(np.float32)
    want = torch.from_numpy(v32).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(O.bf16_round(v32), want)


# ---------------------------------------------------------------- finite differences
def _tiny_problem(seed, d_in=5, d_out=3, n_pos=2, n_neg=2):
    rng = np.random.default_rng(seed)
    for _ in range(100):
        W = rng.normal(size=(d_out, d_in))
        b = rng.normal(size=d_out) * 0.1
        x = rng.uniform(0, 1, (n_pos + n_neg, d_in))
        z = O.layer_forward(W, b, x, 1e-8)[1]
        if np.min(np.abs(z)) > 1e-3:
            return W, b, x
    raise RuntimeError("no kink-free draw")


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_grads_finite_difference(seed):
    W, b, x = _tiny_problem(seed)
    n_pos, theta = 2, 0.7

    def loss_of(Wp, bp):
        return O.ff_loss(O.layer_forward(Wp, bp, x, 1e-8)[3], n_pos, theta)[0]

    xh, _, h, g = O.layer_forward(W, b, x, 1e-8)
    dW, db = O.layer_grads(xh, h, O.ff_loss(g, n_pos, theta)[1])
    e = 1e-6
    num = np.zeros_like(W)
    for i in range(W.shape[0]):
        for j in range(W.shape[1]):
            Wp, Wm = W.copy(), W.copy()
            Wp[i, j] += e
            Wm[i, j] -= e
            num[i, j] = (loss_of(Wp, b) - loss_of(Wm, b)) / (2 * e)
    numb = np.zeros_like(b)
    for i in range(b.shape[0]):
        bp, bm = b.copy(), b.copy()
        bp[i] += e
        bm[i] -= e
        numb[i] = (loss_of(W, bp) - loss_of(W, bm)) / (2 * e)
    assert np.max(np.abs(num - dW)) <= 1e-6 * max(1.0, np.max(np.abs(dW)))
    assert np.max(np.abs(numb - db)) <= 1e-6 * max(1.0, np.max(np.abs(db)))


# ---------------------------------------------------------------- PyTorch fp64 cross-check
def test_layer_steps_match_torch_autograd_adam():
    torch = pytest.importorskip("torch")
    x_base = random_matrix(11, 24, 40, 0, 1, p_zero=0.6)
    y, y_neg = random_labels(12, 24)
    (W0, b0), = make_weights(13, (40, 17))
    b0 = b0 + np.linspace(-0.05, 0.05, 17).astype(np.float32)
    hp = O.HParams(theta=2.0, lr=0.03)
    x = np.concatenate([O.embed_labels(x_base, y, 10), O.embed_labels(x_base, y_neg, 10)])
    n_pos = 24

    Wt = torch.tensor(W0, dtype=torch.float64, requires_grad=True)
    bt = torch.tensor(b0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([Wt, bt], lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.adam_eps)
    xt = torch.tensor(x, dtype=torch.float64)
    L = O.Layer.from_params(W0, b0)
    for step in range(4):
        xh = xt / (xt.norm(dim=1, keepdim=True) + hp.norm_eps)
        h = torch.relu(xh @ Wt.T + bt)
        g = (h * h).sum(1)
        loss = (torch.nn.functional.softplus(hp.theta - g[:n_pos]).mean()
                + torch.nn.functional.softplus(g[n_pos:] - hp.theta).mean())
        opt.zero_grad()
        loss.backward()
        r = O.layer_step(L, x, n_pos, hp)
        assert abs(r.loss - loss.item()) < 1e-12
        np.testing.assert_allclose(r.g, g.detach().numpy(), rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(r.dW, Wt.grad.numpy(), rtol=1e-10, atol=1e-14)
        np.testing.assert_allclose(r.db, bt.grad.numpy(), rtol=1e-10, atol=1e-14)
        opt.step()
        np.testing.assert_allclose(L.W, Wt.detach().numpy(), rtol=1e-11, atol=1e-13)
        np.testing.assert_allclose(L.b, bt.detach().numpy(), rtol=1e-11, atol=1e-13)


# ---------------------------------------------------------------- scoring
def test_score_hand_designed_net():
    """One layer whose unit k sees label feature k plus data feature k.

    For label c and data d >= 0 (C features after the label area), with
    s = 1/(||(e_c, d)|| + eps) the same for every c:
    g(c) = s^2 sum_k (delta_kc + d_k)^2 = s^2 (||d_{:C}||^2 + 2 d_c + 1),
    so the predicted label is argmax_c d_c.
    """
    C = 10
    rng = np.random.default_rng(4)
    data = rng.uniform(0, 1, (8, C))
    x_base = np.concatenate([rng.uniform(0, 1, (8, C)), data], axis=1)
    W = np.zeros((C, 2 * C))
    W[np.arange(C), np.arange(C)] = 1.0
    W[np.arange(C), C + np.arange(C)] = 1.0
    L = O.Layer.from_params(W, np.zeros(C))
    S, pred = O.score_labels([L], x_base, C, O.HParams())
    np.testing.assert_array_equal(pred, np.argmax(data, axis=1))
    s2 = 1.0 / (np.sqrt(1.0 + np.sum(data ** 2, 1)) + 1e-8) ** 2
    want = s2[:, None] * (np.sum(data ** 2, 1)[:, None] + 2 * data + 1)
    np.testing.assert_allclose(S, want, rtol=1e-12)


def test_score_brute_force_and_first_layer_skip():
    x_base, _, _ = make_data(3, 8, 30)
    layers = [O.Layer.from_params(W, b) for W, b in make_weights(4, (30, 12, 9))]
    hp = O.HParams()
    S0, p0 = O.score_labels(layers, x_base, 10, hp, 0)
    S1, p1 = O.score_labels(layers, x_base, 10, hp, 1)
    for n in range(8):
        tot0, tot1 = [], []
        for c in range(10):
            a = x_base[n].astype(float).copy()
            a[:10] = 0
            a[c] = 1
            gs = []
            for L in layers:
                a = a / (math.sqrt(float(a @ a)) + 1e-8)
                a = np.maximum(L.W @ a + L.b, 0)
                gs.append(float(a @ a))
            tot0.append(sum(gs))
            tot1.append(sum(gs[1:]))
        np.testing.assert_allclose(S0[n], tot0, rtol=1e-12)
        np.testing.assert_allclose(S1[n], tot1, rtol=1e-12)
        assert p0[n] == int(np.argmax(tot0)) and p1[n] == int(np.argmax(tot1))


def test_score_ties_go_to_lowest_label():
    C = 10
    x_base = np.ones((3, 25))
    W = np.zeros((4, 25))
    W[:, C:] = 1.0  # ignores the label area entirely: all labels tie
    L = O.Layer.from_params(W, np.zeros(4))
    _, pred = O.score_labels([L], x_base, C, O.HParams())
    np.testing.assert_array_equal(pred, 0)


def test_score_hidden_permutation_invariance():
    x_base, _, _ = make_data(6, 10, 30)
    (W1, b1), (W2, b2) = make_weights(7, (30, 16, 8))
    b1 = b1 + 0.01
    perm = np.random.default_rng(8).permutation(16)
    hp = O.HParams()
    A = [O.Layer.from_params(W1, b1), O.Layer.from_params(W2, b2)]
    B = [O.Layer.from_params(W1[perm], b1[perm]), O.Layer.from_params(W2[:, perm], b2)]
    SA, pa = O.score_labels(A, x_base, 10, hp)
    SB, pb = O.score_labels(B, x_base, 10, hp)
    np.testing.assert_allclose(SA, SB, rtol=1e-12)
    np.testing.assert_array_equal(pa, pb)


# ---------------------------------------------------------------- AdaptiveNEG
def test_adaptive_negatives_hand_designed_net():
    """With the hand-designed layer above, the score of label c rises with the
    data feature d_c, so the hardest wrong label is the largest d_c over the
    labels other than the true one: the runner-up when the true label is the
    largest, else the largest."""
    C = 10
    rng = np.random.default_rng(5)
    data = rng.uniform(0, 1, (40, C))
    x_base = np.concatenate([rng.uniform(0, 1, (40, C)), data], axis=1)
    W = np.zeros((C, 2 * C))
    W[np.arange(C), np.arange(C)] = 1.0
    W[np.arange(C), C + np.arange(C)] = 1.0
    L = O.Layer.from_params(W, np.zeros(C))
    order = np.argsort(-data, axis=1)
    y = np.where(np.arange(40) % 2 == 0, order[:, 0], rng.integers(0, C, 40)).astype(np.int32)
    _, y_neg = O.adaptive_negatives([L], x_base, y, C, O.HParams())
    want = np.where(order[:, 0] == y, order[:, 1], order[:, 0])
    np.testing.assert_array_equal(y_neg, want)


def test_adaptive_negatives_ties_and_exclusion():
    C = 10
    x_base = np.ones((4, 25))
    W = np.zeros((4, 25))
    W[:, C:] = 1.0  # every label ties
    L = O.Layer.from_params(W, np.zeros(4))
    y = np.array([0, 1, 9, 3], np.int32)
    _, y_neg = O.adaptive_negatives([L], x_base, y, C, O.HParams())
    np.testing.assert_array_equal(y_neg, [1, 0, 0, 0])


def test_adaptive_negatives_order_statistics():
    """On a random net: the chosen label is never the true one and beats or ties
    every other wrong label; a sort of each row by (-score, label) gives it."""
    x_base, y, _ = make_data(12, 30, 40)
    layers = _net(13, (40, 16, 12))
    for first in (0, 1):
        S, y_neg = O.adaptive_negatives(layers, x_base, y, 10, O.HParams(), first)
        S2, _ = O.score_labels(layers, x_base, 10, O.HParams(), first)
        np.testing.assert_array_equal(S, S2)
        for n in range(30):
            assert y_neg[n] != y[n]
            ranked = sorted(range(10), key=lambda c: (-S[n, c], c))
            assert y_neg[n] == next(c for c in ranked if c != y[n])


# ---------------------------------------------------------------- chapter schedules
def test_cooldown_closed_form():
    assert O.cooldown_lr(0.03, 0, 100, 50) == 0.03
    assert O.cooldown_lr(0.03, 49, 100, 50) == 0.03
    assert O.cooldown_lr(0.03, 50, 100, 50) == 0.03
    assert abs(O.cooldown_lr(0.03, 75, 100, 50) - 0.015) < 1e-18
    assert abs(O.cooldown_lr(0.03, 99, 100, 50) - 0.0006) < 1e-17
    assert O.cooldown_lr(0.03, 99, 100, 100) == 0.03  # no cooldown


def test_chapters_with_one_split_are_the_sequential_schedule():
    """S = 1 and no cooldown: every layer trains all its epochs on the final
    output of the layers below, which is the sequential FF schedule."""
    x_base, y, y_neg = make_data(60, 150, 30)
    params = make_weights(61, (30, 20, 16))
    a = [O.Layer.from_params(W, b) for W, b in params]
    b = [O.Layer.from_params(W, b) for W, b in params]
    hp = O.HParams(lr=0.03)
    ta = O.chapter_train(a, x_base, y, [y_neg], 10, 64, 2, 1, 2, hp)
    tb = O.train_sequential(b, x_base, y, y_neg, 10, 64, 2, hp)
    np.testing.assert_allclose(ta, tb, rtol=1e-13)
    for la, lb in zip(a, b):
        np.testing.assert_allclose(la.W, lb.W, rtol=1e-13)


def test_chapters_layer_major_order_and_negative_redraw():
    """The result depends only on the (layer, chapter) dependencies: running the
    same units layer-major, with every published version kept, agrees.  Each
    chapter uses its own negatives: a different redraw changes the result."""
    x_base, y, _ = make_data(62, 130, 30)
    negs = [random_labels(63 + c, 130)[1] for c in range(3)]
    params = make_weights(64, (30, 20, 16, 12))
    hp = O.HParams(lr=0.03)
    E, S, chunk = 3, 3, 64
    ref = [O.Layer.from_params(W, b) for W, b in params]
    t_ref = O.chapter_train(ref, x_base, y, negs, 10, chunk, E, S, 1, hp)
    # layer-major: layer l runs all its chapters, keeping every chapter's version
    layers = [O.Layer.from_params(W, b) for W, b in params]
    versions = []  # versions[l][c] = (W, b) published after chapter c
    chunks = O.chunk_bounds(130, chunk)
    t = np.zeros_like(t_ref)
    for li, L in enumerate(layers):
        versions.append([])
        for c in range(S):
            ins = []
            for (s0, b0) in chunks:
                a = O.chunk_input(x_base, y, negs[c], s0, b0, 10)
                for k in range(li):
                    W, bb = versions[k][c]
                    a = O.layer_forward(W, bb, a, 1e-8)[2]
                ins.append(a)
            for q, (s0, b0) in enumerate(chunks):
                hp_e = O.HParams(lr=O.cooldown_lr(0.03, c, E, 1))
                t[li, c * len(chunks) + q] = O.layer_step(L, ins[q], b0, hp_e).loss
            versions[li].append((L.W.copy(), L.b.copy()))
    np.testing.assert_allclose(t, t_ref, rtol=1e-13)
    other = [O.Layer.from_params(W, b) for W, b in params]
    t_other = O.chapter_train(other, x_base, y, [negs[0]] * 3, 10, chunk, E, S, 1, hp)
    assert np.any(t_other[:, len(chunks):] != t_ref[:, len(chunks):])
    np.testing.assert_array_equal(t_other[0, :len(chunks)], t_ref[0, :len(chunks)])


def _hand_adaptive_case(n=40, seed=5):
    """The hand-designed layer of the AdaptiveNEG test: label c's score rises
    with data feature d_c, so the hardest wrong label is the largest d_c over
    the labels other than the true one."""
    C = 10
    rng = np.random.default_rng(seed)
    data = rng.uniform(0, 1, (n, C))
    x_base = np.concatenate([rng.uniform(0, 1, (n, C)), data], axis=1)
    W = np.zeros((C, 2 * C))
    W[np.arange(C), np.arange(C)] = 1.0
    W[np.arange(C), C + np.arange(C)] = 1.0
    order = np.argsort(-data, axis=1)
    y = np.where(np.arange(n) % 2 == 0, order[:, 0], rng.integers(0, C, n)).astype(np.int32)
    want = np.where(order[:, 0] == y, order[:, 1], order[:, 0])
    return x_base, y, W, want


def test_adaptive_chapters_draw_negatives_from_the_network_at_chapter_start():
    """AdaptiveNEG chapters: chapter 0 takes the hardest wrong labels of the
    initial network (known by construction of the hand-designed layer); with
    the rate 0 the network never changes, so every chapter takes them."""
    x_base, y, W, want = _hand_adaptive_case()
    hp = O.HParams(lr=0.03)
    rec = []
    O.chapter_train([O.Layer.from_params(W, np.zeros(10))], x_base, y,
                    O.adaptive_chapter_negatives(x_base, y, 10, hp, record=rec), 10, 16, 4, 2, 4,
                    hp)
    assert len(rec) == 2
    np.testing.assert_array_equal(rec[0], want)
    assert np.all(rec[1] != y)
    rec0 = []
    hp0 = O.HParams(lr=0.0)
    O.chapter_train([O.Layer.from_params(W, np.zeros(10))], x_base, y,
                    O.adaptive_chapter_negatives(x_base, y, 10, hp0, record=rec0), 10, 16, 3, 3, 3,
                    hp0)
    for r in rec0:
        np.testing.assert_array_equal(r, want)


def test_adaptive_chapters_are_the_given_negatives_of_each_chapter_start():
    """Chapter c's AdaptiveNEG labels are adaptive_negatives of the network after
    chapter c-1: training on those labels as given negatives reproduces the run
    bit for bit, and the labels of chapter 1 are those of the network after a
    one-chapter run on chapter 0's labels."""
    x_base, y, _ = make_data(66, 120, 30)
    params = make_weights(67, (30, 20, 16))
    hp = O.HParams(lr=0.05)
    E, S, chunk, cool = 4, 2, 32, 2
    rec = []
    A = [O.Layer.from_params(W, b) for W, b in params]
    ta = O.chapter_train(A, x_base, y, O.adaptive_chapter_negatives(x_base, y, 10, hp, record=rec),
                         10, chunk, E, S, cool, hp)
    B = [O.Layer.from_params(W, b) for W, b in params]
    tb = O.chapter_train(B, x_base, y, rec, 10, chunk, E, S, cool, hp)
    np.testing.assert_array_equal(ta, tb)
    for la, lb in zip(A, B):
        np.testing.assert_array_equal(la.W, lb.W)
    C0 = [O.Layer.from_params(W, b) for W, b in params]
    np.testing.assert_array_equal(rec[0], O.adaptive_negatives(C0, x_base, y, 10, hp)[1])
    O.chapter_train(C0, x_base, y, [rec[0]], 10, chunk, E // S, 1, E, hp)  # chapter 0 only
    np.testing.assert_array_equal(rec[1], O.adaptive_negatives(C0, x_base, y, 10, hp)[1])
    assert np.any(rec[1] != rec[0])


# ---------------------------------------------------------------- softmax head
def test_embed_neutral_hand():
    x = np.arange(24, dtype=np.float32).reshape(2, 12) / 10
    e = O.embed_neutral(x, 10)
    np.testing.assert_array_equal(e[:, :10], 0.1)
    np.testing.assert_array_equal(e[:, 10:], x[:, 10:])


def test_softmax_xent_closed_forms_and_finite_differences():
    C, n = 10, 4
    loss, d, p = O.softmax_xent(np.zeros((n, C)), np.array([0, 3, 9, 3]))
    assert abs(loss - math.log(C)) < 1e-15
    want = np.full((n, C), 1.0 / C)
    want[np.arange(n), [0, 3, 9, 3]] -= 1.0
    np.testing.assert_allclose(d, want / n, atol=1e-16)
    rng = np.random.default_rng(3)
    z = rng.normal(0, 3, (5, 7))
    y = rng.integers(0, 7, 5)
    l0, d0, p0 = O.softmax_xent(z, y)
    np.testing.assert_allclose(p0.sum(axis=1), 1.0, rtol=1e-14)
    l1, _, _ = O.softmax_xent(z + 123.0, y)  # a shift of every logit changes nothing
    assert abs(l1 - l0) < 1e-12
    h = 1e-6
    for i, j in [(0, 0), (2, 5), (4, int(y[4]))]:
        zp, zm = z.copy(), z.copy()
        zp[i, j] += h
        zm[i, j] -= h
        fd = (O.softmax_xent(zp, y)[0] - O.softmax_xent(zm, y)[0]) / (2 * h)
        assert abs(fd - d0[i, j]) < 1e-8


def test_head_features_brute_force():
    x_base, _, _ = make_data(14, 6, 30)
    layers = _net(15, (30, 12, 9, 8))
    hp = O.HParams()
    A = O.head_features(layers, x_base, 10, hp, 1)
    assert A.shape == (6, 17)
    for n in range(6):
        a = [0.1] * 10 + [float(v) for v in x_base[n, 10:]]
        feats = []
        for li, L in enumerate(layers):
            nrm = math.sqrt(sum(v * v for v in a))
            a = [v / (nrm + 1e-8) for v in a]
            a = [max(0.0, sum(L.W[j, k] * a[k] for k in range(len(a))) + L.b[j])
                 for j in range(L.W.shape[0])]
            if li >= 1:
                nrm = math.sqrt(sum(v * v for v in a))
                feats += [v / (nrm + 1e-8) for v in a]
        np.testing.assert_allclose(A[n], feats, rtol=1e-12, atol=1e-15)


def test_head_steps_match_torch_autograd_adam():
    torch = pytest.importorskip("torch")
    x_base, y, _ = make_data(16, 40, 30)
    layers = _net(17, (30, 16, 12))
    rng = np.random.default_rng(18)
    W = rng.uniform(-0.2, 0.2, (10, 12))
    b = rng.uniform(-0.1, 0.1, 10)
    hp, hhp = O.HParams(), O.HParams(lr=1e-2)
    head = O.Head.from_params(W, b)
    A = torch.tensor(O.head_features(layers, x_base, 10, hp, 1))
    Wt = torch.tensor(W, requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    opt = torch.optim.Adam([Wt, bt], lr=1e-2, betas=(0.9, 0.999), eps=1e-8)
    for _ in range(3):
        loss, logits, dW, db = O.head_step(head, layers, x_base, y, 10, hp, hhp, 1)
        opt.zero_grad()
        lt = torch.nn.functional.cross_entropy(A @ Wt.T + bt, torch.tensor(y, dtype=torch.int64))
        lt.backward()
        assert abs(loss - lt.item()) < 1e-12
        np.testing.assert_allclose(dW, Wt.grad.numpy(), rtol=1e-10, atol=1e-15)
        np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-10, atol=1e-15)
        opt.step()
        np.testing.assert_allclose(head.W, Wt.detach().numpy(), rtol=1e-11, atol=1e-14)
        np.testing.assert_allclose(head.b, bt.detach().numpy(), rtol=1e-11, atol=1e-14)


def test_head_predict_is_argmax_with_lowest_tie():
    x_base, _, _ = make_data(19, 5, 30)
    layers = _net(20, (30, 12, 9))
    head = O.Head.from_params(np.zeros((10, 9)), np.array([0, 2, 2, 1, 0, 0, 0, 2, 0, 0.0]))
    logits, pred = O.head_predict(head, layers, x_base, 10, O.HParams(), 1)
    np.testing.assert_array_equal(pred, 1)
    np.testing.assert_allclose(logits, np.tile(head.b, (5, 1)))


# ---------------------------------------------------------------- Performance-Optimised PFF
def _po_case(seed, d_in=30, d_out=16, C=10, n=24):
    x_base, y, _ = make_data(seed, n, d_in)
    (W, b), = make_weights(seed + 1, (d_in, d_out))
    b = b + np.linspace(-0.05, 0.1, d_out).astype(np.float32)
    rng = np.random.default_rng(seed + 2)
    Wc = rng.uniform(-0.3, 0.3, (C, d_out))
    bc = rng.uniform(-0.1, 0.1, C)
    return O.embed_neutral(x_base, C), y, W, b, Wc, bc


def test_po_steps_match_torch_two_layer_backprop():
    """Layer + classifier trained together by autograd through both, Adam on each
    with its own learning rate (PyTorch fp64, library routines only here)."""
    torch = pytest.importorskip("torch")
    x, y, W, b, Wc, bc = _po_case(40)
    hp, hhp = O.HParams(lr=0.03), O.HParams(lr=1e-2)
    L, Hd = O.Layer.from_params(W, b), O.Head.from_params(Wc, bc)
    xt = torch.tensor(O.l2_normalise(x, 1e-8))
    P = [torch.tensor(v, dtype=torch.float64, requires_grad=True) for v in (W, b, Wc, bc)]
    opt_l = torch.optim.Adam(P[:2], lr=0.03, betas=(0.9, 0.999), eps=1e-8)
    opt_c = torch.optim.Adam(P[2:], lr=1e-2, betas=(0.9, 0.999), eps=1e-8)
    for _ in range(3):
        loss, h, logits, dW, db, dWc, dbc = O.po_layer_step(L, Hd, x, y, hp, hhp)
        opt_l.zero_grad()
        opt_c.zero_grad()
        ht = torch.relu(xt @ P[0].T + P[1])
        lt = torch.nn.functional.cross_entropy(ht @ P[2].T + P[3],
                                               torch.tensor(y, dtype=torch.int64))
        lt.backward()
        assert abs(loss - lt.item()) < 1e-12
        np.testing.assert_allclose(h, ht.detach().numpy(), rtol=1e-12, atol=1e-15)
        for got, t in zip((dW, db, dWc, dbc), P):
            np.testing.assert_allclose(got, t.grad.numpy(), rtol=1e-10, atol=1e-15)
        opt_l.step()
        opt_c.step()
        for got, t in zip((L.W, L.b, Hd.W, Hd.b), P):
            np.testing.assert_allclose(got, t.detach().numpy(), rtol=1e-11, atol=1e-14)


def test_po_bf16_gradient_within_rounding_bound():
    """In bf16 mode the weight gradient contracts bf16-rounded dZ and x_hat (R3,
    R1); it differs from the exact one by at most the rounding of those operands:
    |dW16 - dW| <= (2^-8 + 2^-8 + 2^-16) * sum |dz| |x_hat| elementwise."""
    x, y, W, b, Wc, bc = _po_case(41)
    hp16, hp = O.HParams(bf16=True), O.HParams()
    r16 = O.po_layer_step(O.Layer.from_params(W, b), O.Head.from_params(Wc, bc), x, y, hp16, hp)
    # the exact gradient on the same bf16 forward: dz from the same logits, unrounded
    xh16 = O.bf16_round(O.l2_normalise(x, 1e-8))
    z16 = xh16 @ O.bf16_round(W).T + b
    h16 = np.maximum(z16, 0)
    _, d, _ = O.softmax_xent(h16 @ Wc.T + bc, y)
    dz = (d @ Wc) * (z16 > 0)
    exact = dz.T @ xh16
    bound = (2.0 ** -8 + 2.0 ** -8 + 2.0 ** -16) * (np.abs(dz).T @ np.abs(xh16))
    assert np.all(np.abs(r16[3] - exact) <= bound + 1e-300)
    assert np.any(r16[3] != exact)  # the rounding is applied


def test_po_pipeline_layer_independence_and_one_layer():
    """Layer l's loss trace depends only on layers 0..l; with one layer the
    pipeline is the plain chunk-by-chunk sequence of steps."""
    x_base, y, _ = make_data(42, 150, 30)
    dims = (30, 20, 16, 12)
    params = make_weights(43, dims)
    rng = np.random.default_rng(44)
    heads = [rng.uniform(-0.2, 0.2, (10, d)) for d in dims[1:]]
    hp, hhp = O.HParams(lr=0.03), O.HParams(lr=1e-3)

    def run(ps, hs):
        Ls = [O.Layer.from_params(W, b) for W, b in ps]
        Hs = [O.Head.from_params(Wc, np.zeros(10)) for Wc in hs]
        return O.po_train_pipelined(Ls, Hs, x_base, y, 10, 64, 2, hp, hhp)

    t = run(params, heads)
    alt = list(params)
    alt[2] = (params[2][0] * 0.5, params[2][1])
    t2 = run(alt, heads[:2] + [heads[2] * 3.0])
    np.testing.assert_array_equal(t[:2], t2[:2])
    assert np.any(t[2] != t2[2])
    L = O.Layer.from_params(*params[0])
    Hd = O.Head.from_params(heads[0], np.zeros(10))
    seq = []
    for _ in range(2):
        for s, b in O.chunk_bounds(150, 64):
            seq.append(O.po_layer_step(L, Hd, O.embed_neutral(x_base[s:s + b], 10), y[s:s + b],
                                       hp, hhp)[0])
    np.testing.assert_array_equal(t[0], seq)


def test_po_schedules_agree_for_one_layer_and_when_frozen():
    """One layer: sequential and pipelined are the same chunk sequence.  With
    learning rates 0 (weights frozen) every layer sees the same activities in
    both schedules, so the traces agree for all layers."""
    x_base, y, _ = make_data(48, 130, 30)
    dims = (30, 20, 16)
    params = make_weights(49, dims)
    rng = np.random.default_rng(50)
    hw = [rng.uniform(-0.2, 0.2, (10, d)) for d in dims[1:]]

    def run(fn, k, lr, hlr):
        Ls = [O.Layer.from_params(W, b) for W, b in params[:k]]
        Hs = [O.Head.from_params(W, np.zeros(10)) for W in hw[:k]]
        return fn(Ls, Hs, x_base, y, 10, 64, 2, O.HParams(lr=lr), O.HParams(lr=hlr))

    np.testing.assert_array_equal(run(O.po_train_sequential, 1, 0.03, 1e-3),
                                  run(O.po_train_pipelined, 1, 0.03, 1e-3))
    np.testing.assert_allclose(run(O.po_train_sequential, 2, 0.0, 0.0),
                               run(O.po_train_pipelined, 2, 0.0, 0.0), rtol=1e-13)
    assert np.any(run(O.po_train_sequential, 2, 0.03, 1e-3)[1]
                  != run(O.po_train_pipelined, 2, 0.03, 1e-3)[1])


def test_po_predict_last_and_all_layers():
    x_base, _, _ = make_data(45, 20, 30)
    params = make_weights(46, (30, 16, 12))
    layers = [O.Layer.from_params(W, b) for W, b in params]
    rng = np.random.default_rng(47)
    heads = [O.Head.from_params(rng.normal(size=(10, d)), rng.normal(size=10)) for d in (16, 12)]
    zl, pl = O.po_predict(layers, heads, x_base, 10, O.HParams(), all_layers=False)
    za, pa = O.po_predict(layers, heads, x_base, 10, O.HParams(), all_layers=True)
    a = O.embed_neutral(x_base, 10)
    h1 = O.layer_forward(layers[0].W, layers[0].b, a, 1e-8)[2]
    h2 = O.layer_forward(layers[1].W, layers[1].b, h1, 1e-8)[2]
    z1 = h1 @ heads[0].W.T + heads[0].b
    z2 = h2 @ heads[1].W.T + heads[1].b
    np.testing.assert_allclose(zl, z2, rtol=1e-13)
    np.testing.assert_allclose(za, z1 + z2, rtol=1e-13)
    np.testing.assert_array_equal(pl, np.argmax(z2, axis=1))
    np.testing.assert_array_equal(pa, np.argmax(z1 + z2, axis=1))


# ---------------------------------------------------------------- schedules
def _net(seed, dims):
    return [O.Layer.from_params(W, b) for W, b in make_weights(seed, dims)]


def test_pipelined_equals_sequential_for_one_layer():
    x_base, y, y_neg = make_data(21, 50, 24)
    hp = O.HParams(lr=0.03)
    A, B = _net(22, (24, 9)), _net(22, (24, 9))
    ta = O.train_sequential(A, x_base, y, y_neg, 10, 16, 2, hp)
    tb = O.train_pipelined(B, x_base, y, y_neg, 10, 16, 2, hp)
    np.testing.assert_array_equal(ta, tb)
    np.testing.assert_array_equal(A[0].W, B[0].W)


def test_pipelined_order_invariance():
    x_base, y, y_neg = make_data(23, 45, 20)
    hp = O.HParams(lr=0.05)
    res = []
    for order in ["chunk_major", "layer_major", "wavefront"]:
        net = _net(24, (20, 12, 10, 8))
        tr = O.train_pipelined(net, x_base, y, y_neg, 10, 8, 1, hp, order=order)
        res.append((tr, [L.W for L in net]))
    for tr, Ws in res[1:]:
        np.testing.assert_array_equal(tr, res[0][0])
        for a, b in zip(Ws, res[0][1]):
            np.testing.assert_array_equal(a, b)


def test_schedules_agree_when_weights_frozen():
    """With lr=0 pre- and post-update activities coincide, so both schedules see the
    same inputs; each chunk loss then equals the loss of a plain forward pass."""
    x_base, y, y_neg = make_data(25, 30, 20)
    hp = O.HParams(lr=0.0)
    A, B = _net(26, (20, 12, 10)), _net(26, (20, 12, 10))
    ta = O.train_sequential(A, x_base, y, y_neg, 10, 8, 1, hp)
    tb = O.train_pipelined(B, x_base, y, y_neg, 10, 8, 1, hp)
    np.testing.assert_allclose(ta, tb, rtol=1e-13)
    for ci, (s, b) in enumerate(O.chunk_bounds(30, 8)):
        xs = x_base[s:s + b]
        a = np.concatenate([O.embed_labels(xs, y[s:s + b], 10), O.embed_labels(xs, y_neg[s:s + b], 10)])
        for li, L in enumerate(A):
            a = np.maximum(O.l2_normalise(a, 1e-8) @ L.W.T + L.b, 0)
            g = np.sum(a * a, 1)
            want = (np.mean(np.log1p(np.exp(2.0 - g[:b]))) + np.mean(np.log1p(np.exp(g[b:] - 2.0))))
            assert abs(ta[li, ci] - want) < 1e-12


def test_sequential_hands_over_final_weights():
    """Layer 2 of the sequential schedule trains on layer 1's output under its *final* weights."""
    x_base, y, y_neg = make_data(27, 12, 16)
    hp = O.HParams(lr=0.05)
    A = _net(28, (16, 10, 6))
    O.train_sequential(A, x_base, y, y_neg, 10, 12, 3, hp)
    B = _net(28, (16, 10, 6))
    x = np.concatenate([O.embed_labels(x_base, y, 10), O.embed_labels(x_base, y_neg, 10)])
    for _ in range(3):
        O.layer_step(B[0], x, 12, hp)
    h = np.maximum(O.l2_normalise(x, 1e-8) @ B[0].W.T + B[0].b, 0)  # final layer-1 weights
    for _ in range(3):
        O.layer_step(B[1], h, 12, hp)
    np.testing.assert_array_equal(A[1].W, B[1].W)


def test_pipelined_hands_over_pre_update_activities():
    x_base, y, y_neg = make_data(29, 6, 16)
    hp = O.HParams(lr=0.05)
    A = _net(30, (16, 10, 6))
    O.train_pipelined(A, x_base, y, y_neg, 10, 6, 1, hp)
    B = _net(30, (16, 10, 6))
    x = np.concatenate([O.embed_labels(x_base, y, 10), O.embed_labels(x_base, y_neg, 10)])
    h = np.maximum(O.l2_normalise(x, 1e-8) @ B[0].W.T + B[0].b, 0)  # weights before the step
    O.layer_step(B[0], x, 6, hp)
    O.layer_step(B[1], h, 6, hp)
    np.testing.assert_array_equal(A[1].W, B[1].W)


def test_chunking_ragged_tail():
    assert O.chunk_bounds(60000, 1024)[-1] == (59392, 608)
    assert len(O.chunk_bounds(60000, 1024)) == 59
    assert O.chunk_bounds(50000, 2048)[-1] == (49152, 848)
    assert len(O.chunk_bounds(50000, 2048)) == 25


# ---------------------------------------------------------------- bf16 emulation points
# bf16 mode rounds three operands to bfloat16 (round to nearest, ties to even):
# R1 the normalised layer input, R2 the weights, R3 dZ = 2 dL/dg h before the
# weight-gradient contraction; db, h, g and the loss stay unrounded.
def test_bf16_forward_hand_ties():
    """Ties of R1 and R2 go to the even neighbour, non-ties to the nearest; the
    bias and the accumulation are not rounded (hand-derived values)."""
    c = GOLD["bf16_forward_ties"]
    W, b = _layer(c)
    xh, z, h, g = O.layer_forward(W, b, np.array(c["x"], float), c["norm_eps"], bf16=True)
    np.testing.assert_array_equal(xh, c["x_hat"])
    np.testing.assert_array_equal(h, c["h"])
    np.testing.assert_allclose(g, c["g"], rtol=1e-15)


def test_bf16_step_hand_r3():
    """R3 rounds dZ = 2 dL/dg h (not dW, not h); db sums the unrounded dZ."""
    c = GOLD["bf16_step_r3"]
    W, b = _layer(c)
    L = O.Layer.from_params(W, b)
    r = O.layer_step(L, np.array(c["x"], float), c["n_pos"],
                     O.HParams(theta=c["theta"], norm_eps=c["norm_eps"], bf16=True))
    np.testing.assert_allclose(r.g, c["g"], rtol=1e-15)
    assert abs(r.loss - c["loss"]) <= 1e-15 * c["loss"]
    np.testing.assert_allclose(r.dLdg, c["dLdg"], rtol=1e-14)
    np.testing.assert_array_equal(r.dW, c["dW"])  # sums of products of bf16 values: exact
    np.testing.assert_allclose(r.db, c["db"], rtol=1e-14)


def _bf16_random_step(seed):
    x_base, y, y_neg = make_data(seed, 64, 48)
    (W, b), = make_weights(seed + 1, (48, 40))
    b = b + np.linspace(-0.05, 0.1, 40)
    x = np.concatenate([O.embed_labels(x_base, y, 10), O.embed_labels(x_base, y_neg, 10)])
    r = O.layer_step(O.Layer.from_params(W, b), x, 64, O.HParams(theta=1.0, bf16=True))
    return x, W, b, r


def test_bf16_weight_gradient_within_r3_rounding_bound():
    """On the same bf16 forward (R1, R2 applied), the weight gradient differs from
    the exact one only by the rounding of dZ: |dW16 - dW| <= (2^-8 + 2^-16) |dZ|^T
    |x_hat| elementwise (bf16 unit roundoff 2^-8, after the float32 conversion),
    and it does differ, so the rounding is applied."""
    x, W, b, r = _bf16_random_step(150)
    xh16 = O.bf16_round(O.l2_normalise(x, 1e-8))
    h16 = np.maximum(xh16 @ O.bf16_round(W).T + b, 0.0)
    np.testing.assert_array_equal(r.xh, xh16)
    np.testing.assert_allclose(r.h, h16, rtol=1e-14, atol=1e-16)
    g = (h16 * h16).sum(axis=1)
    n = 64
    s = np.where(np.arange(2 * n) < n, -1.0 / (1.0 + np.exp(g - 1.0)),
                 1.0 / (1.0 + np.exp(1.0 - g))) / n
    dz = 2.0 * s[:, None] * h16
    exact = dz.T @ xh16
    bound = (2.0 ** -8 + 2.0 ** -16) * (np.abs(dz).T @ np.abs(xh16))
    assert np.all(np.abs(r.dW - exact) <= bound + 1e-300)
    assert np.mean(r.dW != exact) > 0.5


def test_bf16_bias_gradient_is_unrounded():
    """db sums dZ before R3: it matches the sum of the unrounded dZ to fp64
    rounding and not the sum of the bf16-rounded dZ."""
    x, W, b, r = _bf16_random_step(151)
    dz = 2.0 * r.dLdg[:, None] * r.h
    np.testing.assert_allclose(r.db, dz.sum(axis=0), rtol=1e-13, atol=1e-18)
    rounded = O.bf16_round(dz).sum(axis=0)
    assert np.max(np.abs(r.db - rounded) / np.abs(r.db)) > 1e-4


@pytest.mark.parametrize("mistake", ["none", "round_dW", "round_h_then_scale", "rounded_db",
                                     "no_R1", "no_R2", "ties_away", "no_R3"])
def test_planted_bf16_mistakes_fail_the_hand_cases(mistake):
    """Each plausible mistake in the bf16 step, planted in a copy of it, changes a
    value of the hand-derived cases; the copy without a mistake matches them."""
    def rnd(v):
        if mistake != "ties_away":
            return O.bf16_round(v)
        f = np.asarray(v, np.float32).view(np.uint32).astype(np.uint64)
        return ((f + 0x8000) & 0xFFFF0000).astype(np.uint32).view(np.float32).astype(float)

    def step(case):
        W, b = _layer(case)
        x = np.array(case["x"], float)
        xh = O.l2_normalise(x, case["norm_eps"])
        xh = xh if mistake == "no_R1" else rnd(xh)
        Wr = W if mistake == "no_R2" else rnd(W)
        h = np.maximum(xh @ Wr.T + b, 0.0)
        g = (h * h).sum(axis=1)
        if "n_pos" not in case:
            return h, g, None, None
        _, dg = O.ff_loss(g, case["n_pos"], case["theta"])
        dz = 2.0 * dg[:, None] * h
        if mistake == "round_dW":
            dW = rnd(dz.T @ xh)
        elif mistake == "round_h_then_scale":
            dW = (2.0 * dg[:, None] * rnd(h)).T @ xh
        elif mistake == "no_R3":
            dW = dz.T @ xh
        else:
            dW = rnd(dz).T @ xh
        db = rnd(dz).sum(axis=0) if mistake == "rounded_db" else dz.sum(axis=0)
        return h, g, dW, db

    def matches():
        fwd, st = GOLD["bf16_forward_ties"], GOLD["bf16_step_r3"]
        h, g, _, _ = step(fwd)
        ok = np.array_equal(h, fwd["h"]) and np.allclose(g, fwd["g"], rtol=1e-15)
        h, g, dW, db = step(st)
        return (ok and np.allclose(g, st["g"], rtol=1e-15) and np.array_equal(dW, st["dW"])
                and np.allclose(db, st["db"], rtol=1e-14))

    assert matches() == (mistake == "none")
