"""GPU parity: the HIP path through the C ABI against the CPU oracle, same seeded inputs."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle as O  # noqa: E402
from ffinputs import (WORKLOADS, make_data, make_weights, make_workload,  # noqa: E402
                      random_labels, random_matrix)
from fp32_eval import fp32_evaluation, layers32  # noqa: E402
from parity import (Conditioning, assert_acts, assert_run_like_fp32,  # noqa: E402
                    assert_goodness, assert_labels, assert_loss, assert_negatives, assert_weights,
                    decided, grad_magnitudes, r1_activity_slack, r1_goodness_slack)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2404_08573_amd as P
    return P


DEV = "cuda:0"


def _t(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(DEV)


def _np(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def _pair_rows(x_base, y, y_neg, C=10):
    return np.concatenate([O.embed_labels(x_base, y, C), O.embed_labels(x_base, y_neg, C)])


def _observer(n_layers):
    """on_step for the oracle's schedules: per layer, the conditioning flags of
    every update of W and b (tests/parity.py Conditioning)."""
    cW = [Conditioning() for _ in range(n_layers)]
    cb = [Conditioning() for _ in range(n_layers)]

    def on_step(l, r):
        a, c = grad_magnitudes(r)
        cW[l].add(r.dW, a)
        cb[l].add(r.db, c)
    return on_step, cW, cb


BF16_WEIGHTS = dict(rel=2e-3, outliers=1e-5, outlier_rel=2e-2)


def _run_check(layers, trace, params, lr, run, bf16=True):
    """A multi-layer run against the oracle, within what a float32 evaluation of
    the same run does (tests/parity.py assert_run_like_fp32).
    run(layers, on_step) runs the oracle's schedule on those layers and returns
    its loss trace."""
    refs = [O.Layer.from_params(W, b) for W, b in params]
    on_step, cW, cb = _observer(len(refs))
    t_ref = run(refs, on_step)
    with fp32_evaluation():
        L32 = layers32(params)
        t32 = run(L32, None)
    for L, R in zip(layers, refs):
        assert L.step == R.t
    trace = _np(trace) if torch.is_tensor(trace) else trace
    assert_run_like_fp32([(_np(L.W), _np(L.mW)) for L in layers], [(L.W, L.mW) for L in L32],
                         refs, cW, trace, t32, t_ref, lr, bf16=bf16)
    return refs, cW, cb


def _assert_trained(layers, refs, cW, cb, lr, bf16=False):
    """Every layer's W, b and first moment against the oracle's after the same
    updates (the weight bar with its conditioning sets; bf16: its bf16 form)."""
    extra = BF16_WEIGHTS if bf16 else {}
    for i, (L, R) in enumerate(zip(layers, refs)):
        assert L.step == R.t, (i, L.step, R.t)
        assert_weights(_np(L.W), R.W, cW[i], None, f"layer {i} W", lr=lr, **extra)
        assert_weights(_np(L.b), R.b, cb[i], None, f"layer {i} b", lr=lr, **extra)
        assert_weights(_np(L.mW), R.mW, cW[i], None, f"layer {i} mW", **extra)


# ------------------------------------------------------------------ label embedding
@pytest.mark.parametrize("rows,d,C", [(1, 12, 10), (77, 784, 10), (33, 16, 16)])
def test_embed_labels_exact(P, rows, d, C):
    x = random_matrix(rows + d, rows, d, 0, 1, 0.5)
    lab = np.random.default_rng(rows).integers(0, C, rows).astype(np.int32)
    out = P.ff_embed_labels(_t(x), _t(lab), C)
    np.testing.assert_array_equal(_np(out), O.embed_labels(x, lab, C).astype(np.float32))


# ------------------------------------------------------------------ forward
# small shapes take the 64x64 tile, the last two the 128x128 tile (ragged in rows,
# columns and depth)
FWD_SHAPES = [(1, 12, 8), (130, 44, 132), (300, 200, 260), (1024, 784, 500), (257, 784, 2000),
              (129, 2000, 136), (2100, 788, 2004), (2048, 2000, 2000),
              (37, 4, 20), (300, 16384, 136)]  # the narrowest input; a wide one (large offsets)


@pytest.mark.parametrize("rows,d_in,d_out", FWD_SHAPES)
def test_forward_parity(P, rows, d_in, d_out):
    x = random_matrix(rows * 7 + d_in, rows, d_in, 0, 1, 0.6)
    (W, b), = make_weights(d_out + 3, (d_in, d_out))
    b = b + np.linspace(-0.02, 0.03, d_out).astype(np.float32)
    L = P.Layer(_t(W), _t(b))
    h = torch.empty(rows, d_out, device=DEV)
    g = torch.empty(rows, device=DEV)
    P.ff_layer_forward(L, P.HParams(), _t(x), h_out=h, goodness=g)
    _, _, h_ref, g_ref = O.layer_forward(W, b, x, 1e-8)
    assert_acts(_np(h), h_ref)
    assert_goodness(_np(g), g_ref)
    # goodness only: the kernels' variant without the activity store
    g2 = torch.empty(rows, device=DEV)
    P.ff_layer_forward(L, P.HParams(), _t(x), goodness=g2)
    assert_goodness(_np(g2), g_ref)


def test_forward_prenormalised_input(P):
    x = random_matrix(5, 200, 64, -1, 1)
    xh = O.l2_normalise(x, 1e-8).astype(np.float32)
    (W, b), = make_weights(6, (64, 40))
    L = P.Layer(_t(W), _t(b))
    g = torch.empty(200, device=DEV)
    P.ff_layer_forward(L, P.HParams(), _t(xh), x_normalised=True, goodness=g)
    assert_goodness(_np(g), O.layer_forward(W, b, xh, 0.0, normalised=True)[3])


def test_forward_zero_rows_and_empty(P):
    x = np.zeros((70, 32), np.float32)
    x[::3] = random_matrix(1, 24, 32, 0, 1)[: len(x[::3])]
    (W, b), = make_weights(2, (32, 24))
    b = b + 0.1
    L = P.Layer(_t(W), _t(b))
    g = torch.empty(70, device=DEV)
    P.ff_layer_forward(L, P.HParams(), _t(x), goodness=g)
    assert_goodness(_np(g), O.layer_forward(W, b, x, 1e-8)[3])
    P.ff_layer_forward(L, P.HParams(), _t(np.zeros((0, 32), np.float32)))  # no-op


# ------------------------------------------------------------------ training step
def _run_steps(P, x, n_pos, W, b, k, hp_kw, check_each=True):
    hp, ohp = P.HParams(**hp_kw), O.HParams(**hp_kw)
    L = P.Layer(_t(W), _t(b))
    ref = O.Layer.from_params(W, b)
    R, d_out = x.shape[0], W.shape[0]
    xd = _t(x.astype(np.float32))
    h = torch.empty(R, d_out, device=DEV)
    g = torch.empty(R, device=DEV)
    loss = torch.empty(1, device=DEV)
    gW, gb, mW, mb = [], [], [], []
    for _ in range(k):
        P.ff_layer_step(L, hp, xd, n_pos, R - n_pos, h_out=h, goodness=g, loss=loss)
        r = O.layer_step(ref, x, n_pos, ohp)
        gW.append(r.dW)
        gb.append(r.db)
        a, c = grad_magnitudes(r)
        mW.append(a)
        mb.append(c)
        if check_each:
            assert_goodness(_np(g), r.g)
            assert_loss(_np(loss)[0], r.loss)
            assert_acts(_np(h), r.h)
    assert L.step == k
    assert_weights(_np(L.W), ref.W, gW, mW, "W", lr=ohp.lr, adam_eps=ohp.adam_eps)
    assert_weights(_np(L.b), ref.b, gb, mb, "b", lr=ohp.lr, adam_eps=ohp.adam_eps)
    assert_weights(_np(L.mW), ref.mW, gW, mW, "mW")
    assert_weights(_np(L.vW), ref.vW, gW, mW, "vW", rel=2e-3)
    return L, ref


@pytest.mark.parametrize("n,d_in,d_out", [(16, 12, 8), (150, 200, 260), (512, 784, 500)])
def test_step_parity(P, n, d_in, d_out):
    x_base, y, y_neg = make_data(n + d_in, n, d_in)
    (W, b), = make_weights(d_out, (d_in, d_out))
    _run_steps(P, _pair_rows(x_base, y, y_neg), n, W, b, 1, dict(theta=2.0, lr=0.03))


def test_step_parity_five_steps_tiny_config_layer1(P):
    w = WORKLOADS["mnist_tiny_784_500x2"]
    x_base, y, y_neg = make_data(w.seed_data, w.n, w.dims[0], w.p_zero)
    (W, b), _ = make_weights(w.seed_w, w.dims)
    _run_steps(P, _pair_rows(x_base, y, y_neg), w.n, W, b, 5, dict(theta=2.0, lr=0.03))


def test_step_unequal_halves_and_hidden_input(P):
    x = random_matrix(40, 253, 96, 0, 2, 0.3)  # unnormalised non-negative activities
    (W, b), = make_weights(41, (96, 64))
    _run_steps(P, x, 3, W, b, 3, dict(theta=0.5, lr=0.01))


def test_step_full_size_2000x2000(P):
    """One step at the 2000->2000 layer shape with 1024+1024 rows (the mnist chunk)."""
    x = random_matrix(50, 2048, 2000, 0, 1, 0.5)
    (W, b), = make_weights(51, (2000, 2000))
    _run_steps(P, x, 1024, W, b, 1, dict(theta=2.0, lr=0.03))


def test_step_large_tiles_ragged(P):
    """Both products on their large tiles, ragged in every dimension (2060 rows, 2004 wide)."""
    x = random_matrix(52, 2060, 2004, 0, 1, 0.5)
    (W, b), = make_weights(53, (2004, 2004))
    _run_steps(P, x, 1031, W, b, 2, dict(theta=2.0, lr=0.01))


def test_step_workspace_too_small_changes_nothing(P):
    (W, b), = make_weights(3, (16, 8))
    L = P.Layer(_t(W), _t(b))
    x = _t(random_matrix(4, 8, 16, 0, 1))
    ws = torch.empty(64, dtype=torch.uint8, device=DEV)
    with pytest.raises(P.FFError) as e:
        P.ff_layer_step(L, P.HParams(), x, 4, 4, ws=ws)
    assert e.value.status == P.FF_ERR_WORKSPACE
    assert L.step == 0
    np.testing.assert_array_equal(_np(L.W), W)


# ------------------------------------------------------------------ label scoring
@pytest.mark.parametrize("first", [0, 1])
def test_score_parity_tiny_config(P, first):
    w = WORKLOADS["mnist_tiny_784_500x2"]
    x_base, _, _ = make_data(w.seed_data, w.n, w.dims[0], w.p_zero)
    params = make_weights(w.seed_w, w.dims)
    layers = [P.Layer(_t(W), _t(b)) for W, b in params]
    S = torch.empty(w.n, 10, device=DEV)
    _, pred = P.ff_score_labels(layers, P.HParams(), _t(x_base), 10, first, scores=S)
    S_ref, p_ref = O.score_labels([O.Layer.from_params(W, b) for W, b in params], x_base, 10,
                                  O.HParams(), first)
    assert_goodness(_np(S), S_ref, what="scores")
    assert_labels(_np(pred), S_ref, p_ref)


def test_score_ragged_blocks_and_tiny(P):
    """More images than one scoring pass holds (8192 inputs; a ragged last pass of
    5), odd label count."""
    n = 8197
    x_base, _, _ = make_data(60, n, 24, 0.5)
    params = make_weights(61, (24, 36, 20))
    layers = [P.Layer(_t(W), _t(b)) for W, b in params]
    S = torch.empty(n, 7, device=DEV)
    _, pred = P.ff_score_labels(layers, P.HParams(), _t(x_base), 7, 0, scores=S)
    S_ref, p_ref = O.score_labels([O.Layer.from_params(W, b) for W, b in params], x_base, 7,
                                  O.HParams(), 0)
    assert_goodness(_np(S), S_ref, what="scores")
    assert_labels(_np(pred), S_ref, p_ref)
    _, p1 = P.ff_score_labels(layers, P.HParams(), _t(x_base[:1]), 7, 1)
    assert _np(p1)[0] == O.score_labels([O.Layer.from_params(W, b) for W, b in params],
                                        x_base[:1], 7, O.HParams(), 1)[1][0]


def test_score_single_label(P):
    """One candidate label: every prediction is label 0 and each score is the
    goodness of the one embedding."""
    x_base, _, _ = make_data(62, 300, 48, 0.5)
    params = make_weights(63, (48, 64, 40))
    layers = [P.Layer(_t(W), _t(b)) for W, b in params]
    S = torch.empty(300, 1, device=DEV)
    _, pred = P.ff_score_labels(layers, P.HParams(), _t(x_base), 1, 0, scores=S)
    S_ref, p_ref = O.score_labels([O.Layer.from_params(W, b) for W, b in params], x_base, 1,
                                  O.HParams(), 0)
    assert_goodness(_np(S), S_ref, what="scores")
    assert (_np(pred) == 0).all() and (p_ref == 0).all()


@pytest.mark.parametrize("n_classes,first", [(16, 0), (17, 1), (20, 0)])
def test_score_label_counts_around_shared_base_limit(P, n_classes, first):
    """Up to 16 labels layer 0 runs once per input and expands per label in its
    epilogue; above that every labelled row is embedded and multiplied."""
    x_base, _, _ = make_data(66, 300, 40, 0.5)
    params = make_weights(67, (40, 68, 24, 12))
    layers = [P.Layer(_t(W), _t(b)) for W, b in params]
    S = torch.empty(300, n_classes, device=DEV)
    _, pred = P.ff_score_labels(layers, P.HParams(), _t(x_base), n_classes, first, scores=S)
    S_ref, p_ref = O.score_labels([O.Layer.from_params(W, b) for W, b in params], x_base,
                                  n_classes, O.HParams(), first)
    assert_goodness(_np(S), S_ref, what="scores")
    assert_labels(_np(pred), S_ref, p_ref)


def test_score_full_size(P):
    """All 10 000 inputs through 784->2000x4 under all 10 labels, every score and
    label against the oracle's brute force."""
    w = WORKLOADS["mnist_score_784_2000x4"]
    x_base, _, _ = make_data(w.seed_data, w.n, w.dims[0], w.p_zero)
    params = make_weights(w.seed_w, w.dims)
    layers = [P.Layer(_t(W), _t(b)) for W, b in params]
    S = torch.empty(w.n, 10, device=DEV)
    _, pred = P.ff_score_labels(layers, P.HParams(), _t(x_base), 10, 0, scores=S)
    Sg, pg = _np(S), _np(pred)
    # the device's own decision in its own precision: pred is the argmax of its scores
    np.testing.assert_array_equal(pg, np.argmax(Sg, axis=1))
    S_ref, p_ref = O.score_labels([O.Layer.from_params(W, b) for W, b in params], x_base, 10,
                                  O.HParams(), 0)
    assert_goodness(Sg, S_ref, what="scores")
    # random weights: the ten scores of an input lie close together, and about
    # 2 % of the inputs have their best two within 1e-4 (undecided)
    assert assert_labels(pg, S_ref, p_ref) > 0.95 * w.n


# ------------------------------------------------------------------ AdaptiveNEG
def _masked_argmax(S, labels):
    S = np.array(S, np.float64)
    inr = (labels >= 0) & (labels < S.shape[1])
    S[np.arange(S.shape[0])[inr], labels[inr]] = -np.inf
    return np.argmax(S, axis=1)


@pytest.mark.parametrize("first", [0, 1])
def test_adaptive_negatives_tiny_config(P, first):
    w = WORKLOADS["mnist_tiny_784_500x2"]
    x_base, y, _ = make_data(w.seed_data, w.n, w.dims[0], w.p_zero)
    params = make_weights(w.seed_w, w.dims)
    layers = [P.Layer(_t(W), _t(b)) for W, b in params]
    S = torch.empty(w.n, 10, device=DEV)
    _, y_neg = P.ff_adaptive_negatives(layers, P.HParams(), _t(x_base), _t(y), 10, first,
                                       scores=S)
    S_ref, n_ref = O.adaptive_negatives([O.Layer.from_params(W, b) for W, b in params], x_base,
                                        y, 10, O.HParams(), first)
    assert_goodness(_np(S), S_ref, what="scores")
    assert assert_negatives(_np(y_neg), S_ref, n_ref, y) > 0.9 * w.n
    np.testing.assert_array_equal(_np(y_neg), _masked_argmax(_np(S), y))


def test_adaptive_negatives_edge_labels(P):
    """Ragged scoring passes, 7 classes, true labels at both ends of the range,
    out-of-range labels (nothing excluded: plain prediction), and 2 classes."""
    x_base, _, _ = make_data(64, 2100, 24, 0.5)
    params = make_weights(65, (24, 36, 20))
    layers = [P.Layer(_t(W), _t(b)) for W, b in params]
    O_layers = [O.Layer.from_params(W, b) for W, b in params]
    labels = np.resize(np.array([0, 6, 3, -1, 7, 6, 0], np.int32), 2100)
    _, y_neg = P.ff_adaptive_negatives(layers, P.HParams(), _t(x_base), _t(labels), 7, 0)
    S_ref, n_ref = O.adaptive_negatives(O_layers, x_base, labels, 7, O.HParams(), 0)
    assert_negatives(_np(y_neg), S_ref, n_ref, labels)
    out = (labels < 0) | (labels >= 7)
    _, pred = P.ff_score_labels(layers, P.HParams(), _t(x_base), 7, 0)
    np.testing.assert_array_equal(_np(y_neg)[out], _np(pred)[out])
    lab2 = (np.arange(50) % 2).astype(np.int32)
    _, y2 = P.ff_adaptive_negatives(layers, P.HParams(), _t(x_base[:50]), _t(lab2), 2, 1)
    np.testing.assert_array_equal(_np(y2), 1 - lab2)


def test_adaptive_negatives_training_set_sampled(P):
    """Negatives for all 60 000 training samples under 784->2000x4 (the labels a
    chapter of AdaptiveNEG training would use); the oracle checks a sample."""
    w = WORKLOADS["mnist_784_2000x4"]
    x_base, y, _ = make_data(w.seed_data, w.n, w.dims[0], w.p_zero)
    params = make_weights(w.seed_w, w.dims)
    layers = [P.Layer(_t(W), _t(b)) for W, b in params]
    S = torch.empty(w.n, 10, device=DEV)
    _, y_neg = P.ff_adaptive_negatives(layers, P.HParams(), _t(x_base), _t(y), 10, 0, scores=S)
    Sg, ng = _np(S), _np(y_neg)
    np.testing.assert_array_equal(ng, _masked_argmax(Sg, y))
    assert not np.any(ng == y)
    idx = np.random.default_rng(1).choice(w.n, 16, replace=False)
    S_ref, n_ref = O.adaptive_negatives([O.Layer.from_params(W, b) for W, b in params],
                                        x_base[idx], y[idx], 10, O.HParams(), 0)
    assert_goodness(Sg[idx], S_ref, what="scores")
    assert_negatives(ng[idx], S_ref, n_ref, y[idx])


# ------------------------------------------------------------------ schedules
def _pipe(P, sched, n, dims, chunk, epochs, seed, hp_kw, streams=None, n_classes=10):
    x_base, y, y_neg = make_data(seed, n, dims[0])
    params = make_weights(seed + 1, dims)
    layers = [P.Layer(_t(W), _t(b)) for W, b in params]
    nc = -(-n // chunk)
    trace = torch.zeros(len(layers), nc * epochs, device=DEV)
    P.ff_pipeline_epoch(layers, P.HParams(**hp_kw), _t(x_base), _t(y), _t(y_neg), n_classes,
                        chunk, epochs, sched, streams=streams, loss_trace=trace)
    torch.cuda.synchronize()
    return layers, _np(trace), (x_base, y, y_neg, params)


@pytest.mark.parametrize("sched", [0, 1])
def test_pipeline_parity_small(P, sched):
    hp_kw = dict(theta=2.0, lr=0.03)
    dims = (64, 96, 80, 48)
    layers, trace, (x_base, y, y_neg, params) = _pipe(P, sched, 300, dims, 64, 2, 70, hp_kw)
    ref = [O.Layer.from_params(W, b) for W, b in params]
    fn = O.train_sequential if sched == 0 else O.train_pipelined
    on_step, cW, cb = _observer(len(ref))
    tr_ref = fn(ref, x_base, y, y_neg, 10, 64, 2, O.HParams(**hp_kw), on_step=on_step)
    np.testing.assert_allclose(trace, tr_ref, rtol=1e-4)
    assert all(L.step == tr_ref.shape[1] for L in layers)
    _assert_trained(layers, ref, cW, cb, hp_kw["lr"])


@pytest.mark.parametrize("sched", [0, 1])
def test_pipeline_parity_many_labels(P, sched):
    """17 label features: above the label count whose layer-0 products share the
    pair's base row, so every labelled row is embedded and multiplied."""
    hp_kw = dict(theta=2.0, lr=0.03)
    dims = (64, 96, 48)
    layers, trace, (x_base, y, y_neg, params) = _pipe(P, sched, 200, dims, 64, 1, 71, hp_kw,
                                                      n_classes=17)
    ref = [O.Layer.from_params(W, b) for W, b in params]
    fn = O.train_sequential if sched == 0 else O.train_pipelined
    on_step, cW, cb = _observer(len(ref))
    tr_ref = fn(ref, x_base, y, y_neg, 17, 64, 1, O.HParams(**hp_kw), on_step=on_step)
    np.testing.assert_allclose(trace, tr_ref, rtol=1e-4)
    _assert_trained(layers, ref, cW, cb, hp_kw["lr"])


def test_pipeline_schedule_invariance_bitwise(P):
    """Same result with one stream per layer, run twice, and with every layer on one stream."""
    hp_kw = dict(theta=2.0, lr=0.03)
    dims = (784, 256, 256, 256)
    a, ta, _ = _pipe(P, 1, 1500, dims, 256, 1, 80, hp_kw)
    b, tb, _ = _pipe(P, 1, 1500, dims, 256, 1, 80, hp_kw)
    s = torch.cuda.current_stream()
    c, tc, _ = _pipe(P, 1, 1500, dims, 256, 1, 80, hp_kw, streams=[s] * len(dims[1:]))
    np.testing.assert_array_equal(ta, tb)
    np.testing.assert_array_equal(ta, tc)
    for x, y, z in zip(a, b, c):
        np.testing.assert_array_equal(_np(x.W), _np(y.W))
        np.testing.assert_array_equal(_np(x.W), _np(z.W))


@pytest.mark.parametrize("sched", [0, 1])
def test_epoch_adam_launch_matches_fused_steps_bitwise(P, sched):
    """bf16 epochs run each step's Adam update as a launch of its own from the
    stored weight gradient; single layer steps fuse it into the product's
    epilogue.  A one-layer epoch (784 -> 256, 128-pair chunks, a ragged 44-pair
    last chunk) equals the same chunks' embedded rows through ff_layer_step,
    bit for bit: weights, moments, bias, bf16 shadow and per-chunk losses."""
    hp = P.HParams(theta=2.0, lr=0.01, dtype=P.FF_BF16)
    x_base, y, y_neg = make_data(190, 300, 784)
    (W, b), = make_weights(191, (784, 256))
    ep = P.Layer(_t(W), _t(b), True)
    nc = -(-300 // 128)
    trace = torch.zeros(1, nc, device=DEV)
    P.ff_pipeline_epoch([ep], hp, _t(x_base), _t(y), _t(y_neg), 10, 128, 1, sched,
                        loss_trace=trace)
    st = P.Layer(_t(W), _t(b), True)
    losses = []
    for c in range(nc):
        sl = slice(128 * c, min(300, 128 * (c + 1)))
        x = np.concatenate([O.embed_labels(x_base[sl], y[sl], 10),
                            O.embed_labels(x_base[sl], y_neg[sl], 10)]).astype(np.float32)
        k = sl.stop - sl.start
        loss = torch.empty(1, device=DEV)
        P.ff_layer_step(st, hp, _t(x), k, k, loss=loss)
        losses.append(_np(loss)[0])
    np.testing.assert_array_equal(_np(trace)[0], np.array(losses, np.float32))
    assert ep.step == st.step == nc
    for k in ("W", "b", "mW", "vW", "mb", "vb", "W_bf16"):
        np.testing.assert_array_equal(_np(getattr(ep, k)), _np(getattr(st, k)), err_msg=k)


def test_sequential_reforward_beside_next_layer_bitwise(P):
    """The sequential schedule's forward pass with a trained layer's final
    weights runs on a second stream beside the next layer's steps: the same
    result, bit for bit, as with every layer on one stream (two epochs, so later
    passes reuse the finished activities)."""
    hp_kw = dict(theta=2.0, lr=0.03)
    dims = (784, 256, 256, 256)
    a, ta, _ = _pipe(P, 0, 1500, dims, 256, 2, 81, hp_kw)
    s = torch.cuda.current_stream()
    b, tb, _ = _pipe(P, 0, 1500, dims, 256, 2, 81, hp_kw, streams=[s] * len(dims[1:]))
    np.testing.assert_array_equal(ta, tb)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(_np(x.W), _np(y.W))
        np.testing.assert_array_equal(_np(x.b), _np(y.b))


def test_sequential_reforward_beside_next_layer_bitwise_bf16(P):
    """bf16: the forward pass with a trained layer's final weights beside the
    next layer's steps on a second stream (256-pair chunks and a ragged 220-pair
    last one, two epochs) gives the same result, bit for bit, as on one stream."""
    hp = P.HParams(theta=2.0, lr=0.01, dtype=P.FF_BF16)
    dims = (784, 256, 256, 256)
    x_base, y, y_neg = make_data(82, 1500, dims[0])
    params = make_weights(83, dims)
    out = []
    for streams in (None, [torch.cuda.current_stream()] * 3):
        layers = [P.Layer(_t(W), _t(b), bf16_shadow=True) for W, b in params]
        trace = torch.zeros(3, 2 * 6, device=DEV)
        P.ff_pipeline_epoch(layers, hp, _t(x_base), _t(y), _t(y_neg), 10, 256, 2,
                            P.FF_SEQUENTIAL, streams=streams, loss_trace=trace)
        out.append((layers, _np(trace)))
    np.testing.assert_array_equal(out[0][1], out[1][1])
    for x, z in zip(out[0][0], out[1][0]):
        for k in ("W", "b", "mW", "W_bf16"):
            np.testing.assert_array_equal(_np(getattr(x, k)), _np(getattr(z, k)), err_msg=k)


@pytest.mark.parametrize("sched", [0, 1])
def test_schedule_parity_bf16_three_layers(P, sched):
    """Three bf16 layers, 230 pairs in 50-pair chunks (a ragged 30-pair last one),
    both schedules (pipelined: layers 1 and 2 take their normalised bf16 operand
    and its transpose from the loss pass of the layer before), against the
    bf16-emulating oracle within what a float32 evaluation of the same run does."""
    hp_kw = dict(theta=2.0, lr=0.01)
    dims = (64, 96, 80, 48)
    x_base, y, y_neg = make_data(92, 230, 64)
    params = make_weights(93, dims)
    layers = [P.Layer(_t(W), _t(b), bf16_shadow=True) for W, b in params]
    trace = torch.zeros(3, 5, device=DEV)
    P.ff_pipeline_epoch(layers, P.HParams(dtype=P.FF_BF16, **hp_kw), _t(x_base), _t(y),
                        _t(y_neg), 10, 50, 1, sched, loss_trace=trace)
    torch.cuda.synchronize()
    fn = O.train_sequential if sched == 0 else O.train_pipelined
    _run_check(layers, trace, params, hp_kw["lr"], lambda Ls, obs: fn(
        Ls, x_base, y, y_neg, 10, 50, 1, O.HParams(bf16=True, **hp_kw), on_step=obs))


def test_pipeline_full_size_bench_config(P):
    """The timed training epoch at its full size and launch configuration (60 000
    pairs, 784->2000x4, 58 chunks of 1024+1024 rows and a ragged one of 608+608,
    one stream per layer): every entry of the 4 x 59 loss trace and the final
    weights and first moments of all four layers against the oracle's pipelined
    run over the whole set; the epoch is bitwise the same when run again and
    when every layer shares one stream."""

    w = WORKLOADS["mnist_784_2000x4_pipelined"]
    x_base, y, y_neg, params = make_workload(w)
    hp_kw = dict(theta=w.theta, lr=w.lr, beta1=w.beta1, beta2=w.beta2, adam_eps=w.adam_eps,
                 norm_eps=w.norm_eps)
    xd, yd, ynd = _t(x_base), _t(y), _t(y_neg)
    nc = len(w.chunks())

    def run(streams):
        layers = [P.Layer(_t(W), _t(b)) for W, b in params]
        trace = torch.zeros(w.n_layers, nc, device=DEV)
        P.ff_pipeline_epoch(layers, P.HParams(**hp_kw), xd, yd, ynd, w.n_classes,
                            w.chunk_pairs, 1, P.FF_PIPELINED, streams=streams, loss_trace=trace)
        torch.cuda.synchronize()
        return [_np(L.W) for L in layers], _np(trace)

    cur = torch.cuda.current_stream()
    four = [cur] + [torch.cuda.Stream() for _ in range(w.n_layers - 1)]
    Wa, ta = run(four)
    Wb, tb = run(four)
    Wc, tc = run([cur] * w.n_layers)
    np.testing.assert_array_equal(ta, tb)
    np.testing.assert_array_equal(ta, tc)
    for a, b, c in zip(Wa, Wb, Wc):
        np.testing.assert_array_equal(a, b)
        np.testing.assert_array_equal(a, c)
        assert np.isfinite(a).all()

    layers = [P.Layer(_t(W), _t(b)) for W, b in params]
    trace = torch.zeros(w.n_layers, nc, device=DEV)
    P.ff_pipeline_epoch(layers, P.HParams(**hp_kw), xd, yd, ynd, w.n_classes, w.chunk_pairs, 1,
                        P.FF_PIPELINED, streams=four, loss_trace=trace)
    torch.cuda.synchronize()
    ref = [O.Layer.from_params(W, b) for W, b in params]
    on_step, cW, cb = _observer(w.n_layers)
    tr_ref = O.train_pipelined(ref, x_base, y, y_neg, w.n_classes, w.chunk_pairs, 1,
                               O.HParams(**hp_kw), on_step=on_step)
    np.testing.assert_array_equal(_np(trace), ta)
    np.testing.assert_allclose(ta, tr_ref, rtol=1e-4)
    _assert_trained(layers, ref, cW, cb, w.lr)


def _subset_chunks(w, which):
    """The samples of chunks `which` of workload w, in that order (full-size
    chunks, including the ragged last one, without the ones between)."""
    x_base, y, y_neg, params = make_workload(w)
    idx = np.concatenate([np.arange(s, s + b) for i, (s, b) in enumerate(w.chunks())
                          if i in which])
    return x_base[idx], y[idx], y_neg[idx], params


def test_cifar_pipeline_full_shape_bf16(P):
    """The CIFAR-shaped bf16 pipeline at its full shape and launch configuration
    (3072->3072x4, bf16 operands, 2048+2048 rows per step, one stream per layer)
    over its first two chunks and its ragged last one (848+848 rows): the loss
    trace, weights and first moments against the bf16-emulating oracle."""
    w = WORKLOADS["cifar_3072x4_bf16_pipelined"]
    nc = len(w.chunks())
    x_base, y, y_neg, params = _subset_chunks(w, (0, 1, nc - 1))
    hp_kw = dict(theta=w.theta, lr=w.lr)
    layers = [P.Layer(_t(W), _t(b), bf16_shadow=True) for W, b in params]
    trace = torch.zeros(w.n_layers, 3, device=DEV)
    cur = torch.cuda.current_stream()
    P.ff_pipeline_epoch(layers, P.HParams(dtype=P.FF_BF16, **hp_kw), _t(x_base), _t(y),
                        _t(y_neg), w.n_classes, w.chunk_pairs, 1, P.FF_PIPELINED,
                        streams=[cur] + [torch.cuda.Stream() for _ in range(w.n_layers - 1)],
                        loss_trace=trace)
    torch.cuda.synchronize()
    assert [b for _, b in O.chunk_bounds(len(y), w.chunk_pairs)] == [2048, 2048, 848]
    _run_check(layers, trace, params, w.lr, lambda Ls, obs: O.train_pipelined(
        Ls, x_base, y, y_neg, w.n_classes, w.chunk_pairs, 1, O.HParams(bf16=True, **hp_kw),
        on_step=obs))


def test_mnist_bf16_sequential_full_shape(P):
    """The bf16 MNIST-shaped sequential schedule at its full shape (784->2000x4,
    1024+1024 rows per step, the final-weights forward pass on a second stream)
    over its first two chunks: 8 layer-steps against the bf16-emulating oracle."""
    w = WORKLOADS["mnist_784_2000x4_bf16"]
    x_base, y, y_neg, params = _subset_chunks(w, (0, 1))
    hp_kw = dict(theta=w.theta, lr=w.lr)
    layers = [P.Layer(_t(W), _t(b), bf16_shadow=True) for W, b in params]
    trace = torch.zeros(w.n_layers, 2, device=DEV)
    cur = torch.cuda.current_stream()
    P.ff_pipeline_epoch(layers, P.HParams(dtype=P.FF_BF16, **hp_kw), _t(x_base), _t(y),
                        _t(y_neg), w.n_classes, w.chunk_pairs, 1, P.FF_SEQUENTIAL,
                        streams=[cur, torch.cuda.Stream()] + [cur] * (w.n_layers - 2),
                        loss_trace=trace)
    torch.cuda.synchronize()
    _run_check(layers, trace, params, w.lr, lambda Ls, obs: O.train_sequential(
        Ls, x_base, y, y_neg, w.n_classes, w.chunk_pairs, 1, O.HParams(bf16=True, **hp_kw),
        on_step=obs))


def test_tiny_config_end_to_end(P):
    """784->500->500, 512 pairs full batch, 5 steps per layer layer by layer, then scoring."""
    w = WORKLOADS["mnist_tiny_784_500x2"]
    x_base, y, y_neg = make_data(w.seed_data, w.n, w.dims[0], w.p_zero)
    params = make_weights(w.seed_w, w.dims)
    layers = [P.Layer(_t(W), _t(b)) for W, b in params]
    hp_kw = dict(theta=w.theta, lr=w.lr)
    trace = torch.zeros(2, 5, device=DEV)
    P.ff_pipeline_epoch(layers, P.HParams(**hp_kw), _t(x_base), _t(y), _t(y_neg), 10, w.n,
                        w.epochs, 0, loss_trace=trace)
    S = torch.empty(w.n, 10, device=DEV)
    _, pred = P.ff_score_labels(layers, P.HParams(**hp_kw), _t(x_base), 10, 0, scores=S)
    ref = [O.Layer.from_params(W, b) for W, b in params]
    tr_ref = O.train_sequential(ref, x_base, y, y_neg, 10, w.n, w.epochs, O.HParams(**hp_kw))
    np.testing.assert_allclose(_np(trace), tr_ref, rtol=1e-4)
    S_ref, p_ref = O.score_labels(ref, x_base, 10, O.HParams(**hp_kw))
    assert_goodness(_np(S), S_ref, rel=1e-3, what="scores after training")
    n_dec = assert_labels(_np(pred), S_ref, p_ref)
    assert n_dec >= 0.9 * w.n


# ------------------------------------------------------------------ bf16 operands
# (4200, 72, 4100) and (4100, 136, 3000) take the four-wave 256x192 bf16 tile,
# (8300, 72, 4100) the 256x256 one (two tiles per CU), all with ragged row,
# column and k tails.
BF16_FWD_SHAPES = [(1, 16, 8), (300, 200, 260), (2048, 784, 2000), (2100, 2000, 2004),
                   (4200, 72, 4100), (4100, 136, 3000), (8300, 72, 4100),
                   (37, 8, 20), (300, 16384, 136),  # the narrowest input; a wide one
                   (8192, 520, 1000)]  # two 128x128 workgroups per CU (two LDS stages)


@pytest.mark.parametrize("rows,d_in,d_out", BF16_FWD_SHAPES)
def test_forward_parity_bf16(P, rows, d_in, d_out):
    x = random_matrix(rows + 3 * d_in, rows, d_in, 0, 1, 0.6)
    (W, b), = make_weights(d_out + 5, (d_in, d_out))
    b = b + np.linspace(-0.02, 0.03, d_out).astype(np.float32)
    L = P.Layer(_t(W), _t(b), bf16_shadow=True)
    h = torch.empty(rows, d_out, device=DEV)
    g = torch.empty(rows, device=DEV)
    P.ff_layer_forward(L, P.HParams(dtype=P.FF_BF16), _t(x), h_out=h, goodness=g)
    _, _, h_ref, g_ref = O.layer_forward(W, b, x, 1e-8, bf16=True)
    Wb, xh = O.bf16_round(W), O.l2_normalise(x, 1e-8)
    slack = r1_goodness_slack(Wb, xh, h_ref)
    assert_goodness(_np(g), g_ref, slack=slack)
    assert_acts(_np(h), h_ref, slack=r1_activity_slack(Wb, xh))
    # goodness only: the kernels' variant without the activity store
    g2 = torch.empty(rows, device=DEV)
    P.ff_layer_forward(L, P.HParams(dtype=P.FF_BF16), _t(x), goodness=g2)
    assert_goodness(_np(g2), g_ref, slack=slack)


def _run_steps_bf16(P, x, n_pos, W, b, k, hp_kw):
    hp = P.HParams(dtype=P.FF_BF16, **hp_kw)
    ohp = O.HParams(bf16=True, **hp_kw)
    L = P.Layer(_t(W), _t(b), bf16_shadow=True)
    ref = O.Layer.from_params(W, b)
    ref32 = O.Layer.from_params(W, b)
    R = x.shape[0]
    xd = _t(x.astype(np.float32))
    g = torch.empty(R, device=DEV)
    loss = torch.empty(1, device=DEV)
    gW, mW = [], []
    for step in range(k):
        P.ff_layer_step(L, hp, xd, n_pos, R - n_pos, goodness=g, loss=loss)
        if step == 0:
            Wb0 = O.bf16_round(ref.W)
        r = O.layer_step(ref, x, n_pos, ohp)
        O.layer_step(ref32, x, n_pos, O.HParams(**hp_kw))
        gW.append(r.dW)
        mW.append(grad_magnitudes(r)[0])
        if step == 0:  # same weights on both sides: the forward's own bar
            assert_goodness(_np(g), r.g,
                            slack=r1_goodness_slack(Wb0, O.l2_normalise(x, 1e-8), r.h))
        assert_loss(_np(loss)[0], r.loss)
    assert_weights(_np(L.W), ref.W, gW, mW, "W (vs bf16-emulating oracle)", rel=2e-3,
                   outliers=1e-5, outlier_rel=2e-2, lr=ohp.lr, adam_eps=ohp.adam_eps)
    # the shadow is the rounded master
    np.testing.assert_array_equal(
        _np(L.W_bf16).view(np.uint16),
        (_np(L.W).view(np.uint32).astype(np.uint64) + 0x7FFF
         + ((_np(L.W).view(np.uint32) >> 16) & 1)).astype(np.uint32).__rshift__(16).astype(np.uint16))
    # the workload's bar against the fp32 oracle
    d = np.linalg.norm(_np(L.W) - ref32.W) / np.linalg.norm(ref32.W)
    assert d <= 5e-2, f"bf16 weights vs fp32 oracle: relative error {d:.3g}"
    return L


def _bf16_rne(w):
    """Round-to-nearest-even bf16 bits of fp32 values (finite inputs)."""
    u = w.view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


@pytest.mark.parametrize("d_out,d_in", [(4, 4), (12, 20), (2000, 784), (3072, 3072)])
def test_bf16_shadow_refresh_exact(P, d_out, d_in):
    """ff_refresh_bf16_shadow: every weight rounded to nearest even."""
    W = random_matrix(d_out * 31 + d_in, d_out, d_in, -2, 2)
    W[0, 0] = np.float32(1.00390625)  # a tie between two bf16 values: rounds to even
    L = P.Layer(_t(W), _t(np.zeros(d_out, np.float32)), bf16_shadow=True)
    L.W_bf16.zero_()
    P.ff_refresh_bf16_shadow(L)
    got = _np(L.W_bf16).view(np.uint16)
    np.testing.assert_array_equal(got, _bf16_rne(W))
    assert got[0, 0] == 0x3F80


@pytest.mark.parametrize("n,d_in,d_out,k", [(24, 16, 12, 2), (150, 200, 260, 3), (1024, 784, 2000, 2)])
def test_step_parity_bf16(P, n, d_in, d_out, k):
    x_base, y, y_neg = make_data(n + d_out, n, d_in)
    (W, b), = make_weights(d_out + 1, (d_in, d_out))
    _run_steps_bf16(P, _pair_rows(x_base, y, y_neg), n, W, b, k, dict(theta=2.0, lr=0.01))


def test_step_parity_bf16_large_tiles_ragged(P):
    # 16 x 16 weight-gradient tiles of 128x128: one per CU (three register stages)
    x = random_matrix(54, 2060, 2008, 0, 1, 0.5)
    (W, b), = make_weights(55, (2008, 2004))
    _run_steps_bf16(P, x, 1031, W, b, 2, dict(theta=2.0, lr=0.01))


def test_step_parity_bf16_two_tiles_per_cu(P):
    # 24 x 24 weight-gradient tiles (two register stages).  The batch is not
    # tiny: the device takes the R3 rounding of c*h from its fp32 forward, and
    # over a 70-row batch the rounding differences against the fp64 oracle
    # exceed the weight bar on the CPU too (1400 of 9e6 weights).
    x = random_matrix(56, 1024, 3000, 0, 1, 0.5)
    (W, b), = make_weights(57, (3000, 3000))
    _run_steps_bf16(P, x, 512, W, b, 2, dict(theta=2.0, lr=0.01))


def test_score_parity_bf16(P):
    """bf16 scoring through two layers.  One layer: every score within 1e-4 plus
    the open-R1 allowance.  Two layers: the second layer's input comes from an
    fp32 product, so some of its R1 roundings go the other way in any
    evaluation short of the oracle's float64; the device's scores stay within 4x
    of what a float32 evaluation of the same scoring does (tests/fp32_eval.py),
    and labels are bit-exact where the oracle's top two are further apart than
    that."""
    x_base, _, _ = make_data(62, 300, 64)
    params = make_weights(63, (64, 96, 40))
    layers = [P.Layer(_t(W), _t(b), bf16_shadow=True) for W, b in params]
    hp, ohp = P.HParams(dtype=P.FF_BF16), O.HParams(bf16=True)
    S = torch.empty(300, 10, device=DEV)
    P.ff_score_labels(layers[:1], hp, _t(x_base), 10, 0, scores=S)
    W0, b0 = params[0]
    S1, _ = O.score_labels([O.Layer.from_params(W0, b0)], x_base, 10, ohp, 0)
    slack = np.stack([r1_goodness_slack(O.bf16_round(W0), O.l2_normalise(xc, 1e-8),
                                        O.layer_forward(W0, b0, xc, 1e-8, bf16=True)[2])
                      for xc in (O.embed_labels(x_base, np.full(300, c), 10) for c in range(10))],
                     axis=1)
    assert_goodness(_np(S), S1, slack=slack, what="bf16 one-layer scores")
    _, pred = P.ff_score_labels(layers, hp, _t(x_base), 10, 0, scores=S)
    S_ref, p_ref = O.score_labels([O.Layer.from_params(W, b) for W, b in params], x_base, 10,
                                  ohp, 0)
    with fp32_evaluation():
        S32, _ = O.score_labels(layers32(params), x_base, 10, ohp, 0)
    e_dev = np.max(np.abs(_np(S) - S_ref) / np.abs(S_ref))
    e32 = np.max(np.abs(S32 - S_ref) / np.abs(S_ref))
    assert e_dev <= 4 * e32 + 1e-6, f"scores: device {e_dev:.3g}, float32 evaluation {e32:.3g}"
    margin = max(1e-4, 8 * e32)
    ok = decided(S_ref, margin)
    np.testing.assert_array_equal(_np(pred)[ok], p_ref[ok])
    assert ok.sum() > 250


def test_pipeline_parity_bf16(P):
    hp_kw = dict(theta=2.0, lr=0.01)
    dims = (64, 96, 80)
    x_base, y, y_neg = make_data(90, 200, 64)
    params = make_weights(91, dims)
    layers = [P.Layer(_t(W), _t(b), bf16_shadow=True) for W, b in params]
    trace = torch.zeros(2, 4, device=DEV)
    P.ff_pipeline_epoch(layers, P.HParams(dtype=P.FF_BF16, **hp_kw), _t(x_base), _t(y),
                        _t(y_neg), 10, 50, 1, P.FF_PIPELINED, loss_trace=trace)
    ref = [O.Layer.from_params(W, b) for W, b in params]
    on_step, cW, cb = _observer(len(ref))
    tr = O.train_pipelined(ref, x_base, y, y_neg, 10, 50, 1, O.HParams(bf16=True, **hp_kw),
                           on_step=on_step)
    np.testing.assert_allclose(_np(trace), tr, rtol=1e-4)
    _assert_trained(layers, ref, cW, cb, hp_kw["lr"], bf16=True)


# ------------------------------------------------------------------ kernel timing
def test_profile_counts_and_kind_mask(P):
    """Every launch of a step is timed and its work counted; a kind mask times
    only the selected kinds."""
    (W, b), = make_weights(90, (64, 96))
    L = P.Layer(_t(W), _t(b))
    x = _t(random_matrix(91, 40, 64, 0, 1))
    P.ff_layer_step(L, P.HParams(), x, 20, 20)
    torch.cuda.synchronize()
    P.ff_profile_start(64)
    P.ff_layer_step(L, P.HParams(), x, 20, 20)
    allk = P.ff_profile_stop()
    for k in ("embed_norm", "forward", "loss", "dw_adam"):
        assert allk[k]["launches"] == 1 and allk[k]["total_ms"] > 0, k
    assert allk["forward"]["flops"] == 2.0 * 40 * 64 * 96
    assert allk["dw_adam"]["flops"] == 2.0 * 96 * 64 * 40
    P.ff_profile_start(64, kinds=["forward"])
    P.ff_layer_step(L, P.HParams(), x, 20, 20)
    only = P.ff_profile_stop()
    assert only["forward"]["launches"] == 1
    assert all(v["launches"] == 0 for k, v in only.items() if k != "forward")


# ------------------------------------------------------------------ softmax prediction layer
def _head_case(seed, dims, C, n, first):
    x_base, y, _ = make_data(seed, n, dims[0])
    y = (y % C).astype(np.int32)
    params = make_weights(seed + 1, dims)
    D = sum(dims[1 + first:])
    rng = np.random.default_rng(seed + 2)
    Wh = rng.uniform(-0.3, 0.3, (C, D)).astype(np.float32)
    bh = rng.uniform(-0.1, 0.1, C).astype(np.float32)
    return x_base, y, params, Wh, bh


@pytest.mark.parametrize("dims,C,n,first", [((784, 500, 500), 10, 512, 1),
                                            ((64, 96, 80, 48), 10, 37, 1),
                                            ((64, 96, 80, 48), 16, 300, 0),
                                            ((64, 96, 80, 48), 7, 129, 0),
                                            ((24, 36, 20), 3, 65, 1),
                                            ((24, 36, 20), 2, 130, 1),
                                            # the most feature blocks (8), each under one chunk
                                            ((16, 4, 8, 12, 4, 8, 4, 4, 8), 16, 3, 0),
                                            ((24, 8, 4), 2, 1, 1)])
def test_head_predict_parity(P, dims, C, n, first):
    x_base, _, params, Wh, bh = _head_case(92, dims, C, n, first)
    layers = [P.Layer(_t(W), _t(b)) for W, b in params]
    head = P.Head(_t(Wh), _t(bh))
    logits = torch.empty(n, C, device=DEV)
    _, pred = P.ff_head_predict(layers, P.HParams(), head, _t(x_base), first, logits=logits)
    ref_layers = [O.Layer.from_params(W, b) for W, b in params]
    z_ref, p_ref = O.head_predict(O.Head.from_params(Wh, bh), ref_layers, x_base, C, O.HParams(),
                                  first)
    assert_acts(_np(logits), z_ref)  # logits can cancel to near 0: floor 1e-5 of the largest
    assert_labels(_np(pred), z_ref, p_ref)
    np.testing.assert_array_equal(_np(pred), np.argmax(_np(logits), axis=1))


@pytest.mark.parametrize("dims,C,n,lr", [((784, 500, 500), 10, 512, 1e-4),
                                         ((64, 96, 80, 48), 10, 300, 1e-2)])
def test_head_steps_parity(P, dims, C, n, lr):
    x_base, y, params, Wh, bh = _head_case(93, dims, C, n, 1)
    layers = [P.Layer(_t(W), _t(b)) for W, b in params]
    head = P.Head(_t(Wh), _t(bh))
    ref_layers = [O.Layer.from_params(W, b) for W, b in params]
    ref = O.Head.from_params(Wh, bh)
    hp, ohp = P.HParams(), O.HParams()
    hhp, ohhp = P.HParams(lr=lr), O.HParams(lr=lr)
    loss = torch.empty(1, device=DEV)
    A = O.head_features(ref_layers, x_base, C, ohp, 1)
    gW, gb, mW, mb = [], [], [], []
    for _ in range(3):
        P.ff_head_step(layers, hp, head, hhp, _t(x_base), _t(y), 1, loss=loss)
        l_ref, _, dW, db = O.head_step(ref, ref_layers, x_base, y, C, ohp, ohhp, 1)
        assert_loss(_np(loss)[0], l_ref)
        gW.append(dW)
        gb.append(db)
    # gradient magnitudes for the conditioning rule: sum of |terms| of each element
    r0 = O.Head.from_params(Wh, bh)
    for _ in range(3):
        z = A @ r0.W.T + r0.b
        _, d, _ = O.softmax_xent(z, y)
        mW.append(np.abs(d).T @ np.abs(A))
        mb.append(np.abs(d).sum(axis=0))
        O.head_step(r0, ref_layers, x_base, y, C, ohp, ohhp, 1)
    assert head.step == 3
    assert_weights(_np(head.W), ref.W, gW, mW, "head W", lr=lr, adam_eps=1e-8)
    assert_weights(_np(head.b), ref.b, gb, mb, "head b", lr=lr, adam_eps=1e-8)
    # the FF layers are untouched
    for L, (W, b) in zip(layers, params):
        np.testing.assert_array_equal(_np(L.W), W)
        assert L.step == 0


def test_head_bf16_layers(P):
    dims, C, n = (64, 96, 80, 48), 10, 200
    x_base, y, params, Wh, bh = _head_case(94, dims, C, n, 1)
    layers = [P.Layer(_t(W), _t(b), bf16_shadow=True) for W, b in params]
    head = P.Head(_t(Wh), _t(bh))
    logits = torch.empty(n, C, device=DEV)
    P.ff_head_predict(layers, P.HParams(dtype=P.FF_BF16), head, _t(x_base), 1, logits=logits)
    ref_layers = [O.Layer.from_params(W, b) for W, b in params]
    z_ref, _ = O.head_predict(O.Head.from_params(Wh, bh), ref_layers, x_base, C,
                              O.HParams(bf16=True), 1)
    assert_acts(_np(logits), z_ref, rel=1e-3, floor=1e-3)


def test_head_full_size_sampled(P):
    """Softmax prediction of all 10 000 inputs through 784->2000x4 (6000 features)."""
    w = WORKLOADS["mnist_score_784_2000x4"]
    x_base, _, _ = make_data(w.seed_data, w.n, w.dims[0], w.p_zero)
    params = make_weights(w.seed_w, w.dims)
    rng = np.random.default_rng(95)
    Wh = rng.uniform(-0.05, 0.05, (10, 6000)).astype(np.float32)
    bh = np.zeros(10, np.float32)
    layers = [P.Layer(_t(W), _t(b)) for W, b in params]
    logits = torch.empty(w.n, 10, device=DEV)
    _, pred = P.ff_head_predict(layers, P.HParams(), P.Head(_t(Wh), _t(bh)), _t(x_base), 1,
                                logits=logits)
    zg, pg = _np(logits), _np(pred)
    np.testing.assert_array_equal(pg, np.argmax(zg, axis=1))
    idx = np.random.default_rng(2).choice(w.n, 16, replace=False)
    z_ref, p_ref = O.head_predict(O.Head.from_params(Wh, bh),
                                  [O.Layer.from_params(W, b) for W, b in params], x_base[idx], 10,
                                  O.HParams(), 1)
    assert_acts(zg[idx], z_ref)
    assert_labels(pg[idx], z_ref, p_ref)


# ------------------------------------------------------------------ Performance-Optimised PFF
def _po_case(seed, d_in, d_out, C, rows):
    x_base, y, _ = make_data(seed, rows, d_in)
    y = (y % C).astype(np.int32)
    (W, b), = make_weights(seed + 1, (d_in, d_out))
    b = b + np.linspace(-0.02, 0.05, d_out).astype(np.float32)
    rng = np.random.default_rng(seed + 2)
    Wc = rng.uniform(-0.2, 0.2, (C, d_out)).astype(np.float32)
    bc = rng.uniform(-0.1, 0.1, C).astype(np.float32)
    return O.embed_neutral(x_base, C).astype(np.float32), y, W, b, Wc, bc


def _po_mags(L, Hd, x, y, hp):
    """Sum of |terms| of every weight-gradient element at the oracle's current
    weights (for the conditioning rule), before the step is taken."""
    xh, z, h, _ = O.layer_forward(L.W, L.b, x, hp.norm_eps, False, hp.bf16)
    _, d, _ = O.softmax_xent(h @ Hd.W.T + Hd.b, y)
    dz = np.abs((d @ Hd.W) * (z > 0))
    return (dz.T @ np.abs(xh), dz.sum(axis=0), np.abs(d).T @ np.abs(h), np.abs(d).sum(axis=0))


@pytest.mark.parametrize("d_in,d_out,C,rows,bf16", [(64, 96, 10, 150, False),
                                                    (784, 2000, 10, 1024, False),
                                                    (200, 260, 16, 77, False),
                                                    (64, 96, 10, 150, True)])
def test_po_layer_steps_parity(P, d_in, d_out, C, rows, bf16):
    x, y, W, b, Wc, bc = _po_case(100 + d_in, d_in, d_out, C, rows)
    hp_kw = dict(lr=0.01)
    hp = P.HParams(dtype=P.FF_BF16 if bf16 else P.FF_F32, **hp_kw)
    ohp = O.HParams(bf16=bf16, **hp_kw)
    hhp, ohhp = P.HParams(lr=1e-3), O.HParams(lr=1e-3)
    L = P.Layer(_t(W), _t(b), bf16_shadow=bf16)
    Hd = P.Head(_t(Wc), _t(bc))
    ref, refh = O.Layer.from_params(W, b), O.Head.from_params(Wc, bc)
    h = torch.empty(rows, d_out, device=DEV)
    loss = torch.empty(1, device=DEV)
    grads = {k: [] for k in ("W", "b", "Wc", "bc")}
    mags = {k: [] for k in ("W", "b", "Wc", "bc")}
    rel = 1e-3 if bf16 else 1e-4
    for step in range(3):
        for k, m in zip(("W", "b", "Wc", "bc"), _po_mags(ref, refh, x, y, ohp)):
            mags[k].append(m)
        P.ff_po_layer_step(L, Hd, hp, hhp, _t(x), _t(y), h_out=h, loss=loss)
        l_ref, h_ref, _, dW, db, dWc, dbc = O.po_layer_step(ref, refh, x, y, ohp, ohhp)
        for k, g in zip(("W", "b", "Wc", "bc"), (dW, db, dWc, dbc)):
            grads[k].append(g)
        assert_loss(_np(loss)[0], l_ref, rel=rel)
        if step == 0:  # later, the weights agree only to the weight bar (Adam-amplified elements)
            assert_acts(_np(h), h_ref, rel=rel, floor=1e-3 if bf16 else 1e-5)
    assert L.step == 3 and Hd.step == 3
    extra = dict(rel=2e-3, outliers=1e-5, outlier_rel=2e-2) if bf16 else {}
    # first moments: linear in the gradients, so every gradient element is checked
    assert_weights(_np(L.mW), ref.mW, grads["W"], mags["W"], "mW", **extra)
    assert_weights(_np(Hd.mW), refh.mW, grads["Wc"], mags["Wc"], "mWc", **extra)
    assert_weights(_np(L.W), ref.W, grads["W"], mags["W"], "W", lr=0.01, **extra)
    assert_weights(_np(L.b), ref.b, grads["b"], mags["b"], "b", lr=0.01, **extra)
    assert_weights(_np(Hd.W), refh.W, grads["Wc"], mags["Wc"], "Wc", lr=1e-3, **extra)
    assert_weights(_np(Hd.b), refh.b, grads["bc"], mags["bc"], "bc", lr=1e-3, **extra)


@pytest.mark.parametrize("sched", [0, 1])
def test_po_epoch_parity(P, sched):
    dims, C, n, chunk = (64, 96, 80, 48), 10, 300, 64
    x_base, y, _ = make_data(110, n, dims[0])
    params = make_weights(111, dims)
    rng = np.random.default_rng(112)
    hws = [rng.uniform(-0.2, 0.2, (C, d)).astype(np.float32) for d in dims[1:]]
    layers = [P.Layer(_t(W), _t(b)) for W, b in params]
    heads = [P.Head(_t(Wc), torch.zeros(C, device=DEV)) for Wc in hws]
    nc = -(-n // chunk)
    trace = torch.zeros(len(layers), 2 * nc, device=DEV)
    P.ff_po_epoch(layers, heads, P.HParams(lr=0.01), P.HParams(lr=1e-3), _t(x_base), _t(y), C,
                  chunk, 2, sched, loss_trace=trace)
    torch.cuda.synchronize()
    ref = [O.Layer.from_params(W, b) for W, b in params]
    refh = [O.Head.from_params(Wc, np.zeros(C)) for Wc in hws]
    fn = O.po_train_sequential if sched == 0 else O.po_train_pipelined
    cond = {k: [Conditioning() for _ in ref] for k in ("W", "b", "Wc", "bc")}
    ohp = O.HParams(lr=0.01)

    def on_step(l, Lpre, Hpre, x, yy, res):
        for k, m, g in zip(("W", "b", "Wc", "bc"), _po_mags(Lpre, Hpre, x, yy, ohp), res[3:7]):
            cond[k][l].add(g, m)
    tr_ref = fn(ref, refh, x_base, y, C, chunk, 2, ohp, O.HParams(lr=1e-3), on_step=on_step)
    np.testing.assert_allclose(_np(trace), tr_ref, rtol=1e-4)
    for i, (L, R, Hd, RH) in enumerate(zip(layers, ref, heads, refh)):
        assert L.step == 2 * nc and Hd.step == 2 * nc
        assert_weights(_np(L.mW), R.mW, cond["W"][i], None, f"{i} mW")
        assert_weights(_np(Hd.mW), RH.mW, cond["Wc"][i], None, f"{i} mWc")
        assert_weights(_np(L.W), R.W, cond["W"][i], None, f"{i} W", lr=0.01)
        assert_weights(_np(L.b), R.b, cond["b"][i], None, f"{i} b", lr=0.01)
        assert_weights(_np(Hd.W), RH.W, cond["Wc"][i], None, f"{i} Wc", lr=1e-3)
        assert_weights(_np(Hd.b), RH.b, cond["bc"][i], None, f"{i} bc", lr=1e-3)


@pytest.mark.parametrize("all_layers", [False, True])
def test_po_predict_parity(P, all_layers):
    dims, C, n = (64, 96, 80, 48), 10, 203
    x_base, _, _ = make_data(113, n, dims[0])
    params = make_weights(114, dims)
    rng = np.random.default_rng(115)
    hw = [(rng.uniform(-0.3, 0.3, (C, d)).astype(np.float32),
           rng.uniform(-0.1, 0.1, C).astype(np.float32)) for d in dims[1:]]
    layers = [P.Layer(_t(W), _t(b)) for W, b in params]
    heads = [P.Head(_t(W), _t(b)) for W, b in hw]
    logits = torch.empty(n, C, device=DEV)
    _, pred = P.ff_po_predict(layers, heads, P.HParams(), _t(x_base), all_layers, logits=logits)
    z_ref, p_ref = O.po_predict([O.Layer.from_params(W, b) for W, b in params],
                                [O.Head.from_params(W, b) for W, b in hw], x_base, C,
                                O.HParams(), all_layers)
    assert_acts(_np(logits), z_ref)
    assert_labels(_np(pred), z_ref, p_ref)


# ------------------------------------------------------------------ chapter schedules (Alg. 1 / 2)
def _chapter(P, assignment, n_streams, dims=(64, 96, 80, 48), n=300, chunk=64, E=4, S=2, cool=2,
             bf16=False, seed=130):
    x_base, y, _ = make_data(seed, n, dims[0])
    negs = np.stack([random_labels(seed + 1 + c, n)[1] for c in range(S)]).astype(np.int32)
    params = make_weights(seed + 9, dims)
    layers = [P.Layer(_t(W), _t(b), bf16_shadow=bf16) for W, b in params]
    nc = -(-n // chunk)
    trace = torch.zeros(len(layers), E * nc, device=DEV)
    hp = P.HParams(lr=0.03, dtype=P.FF_BF16 if bf16 else P.FF_F32)
    P.ff_chapter_train(layers, hp, _t(x_base), _t(y), _t(negs), 10, chunk, E, S, cool, assignment,
                       n_streams=n_streams, loss_trace=trace)
    torch.cuda.synchronize()
    return layers, _np(trace), (x_base, y, negs, params, chunk, E, S, cool)


@pytest.mark.parametrize("assignment,n_streams", [(0, None), (1, 2)])
def test_chapter_parity(P, assignment, n_streams):
    layers, trace, (x_base, y, negs, params, chunk, E, S, cool) = _chapter(P, assignment,
                                                                            n_streams)
    ref = [O.Layer.from_params(W, b) for W, b in params]
    on_step, cW, cb = _observer(len(ref))
    t_ref = O.chapter_train(ref, x_base, y, list(negs), 10, chunk, E, S, cool, O.HParams(lr=0.03),
                            on_step=on_step)
    np.testing.assert_allclose(trace, t_ref, rtol=1e-4)
    _assert_trained(layers, ref, cW, cb, 0.03)


def test_chapter_assignments_agree_bitwise(P):
    """Single-Layer (one stream per layer) and All-Layers (chapters dealt to 1
    or 3 streams) run the same (layer, chapter) graph: identical results."""
    a, ta, _ = _chapter(P, 0, None, E=6, S=3, cool=3)
    b, tb, _ = _chapter(P, 1, 3, E=6, S=3, cool=3)
    c, tc, _ = _chapter(P, 1, 1, E=6, S=3, cool=3)
    np.testing.assert_array_equal(ta, tb)
    np.testing.assert_array_equal(ta, tc)
    for x, y_, z in zip(a, b, c):
        np.testing.assert_array_equal(_np(x.W), _np(y_.W))
        np.testing.assert_array_equal(_np(x.W), _np(z.W))


def test_chapter_parity_bf16(P):
    layers, trace, (x_base, y, negs, params, chunk, E, S, cool) = _chapter(P, 0, None, bf16=True)
    _run_check(layers, trace, params, 0.03, lambda Ls, obs: O.chapter_train(
        Ls, x_base, y, list(negs), 10, chunk, E, S, cool, O.HParams(lr=0.03, bf16=True),
        on_step=obs))


# ------------------------------------------------------------------ hand-derived bf16 cases
def test_bf16_hand_cases_on_gpu(P):
    """The hand-derived bf16 cases (tests/golden/hand_cases.json): R1 and R2 ties
    to even give bit-exact activities (every product is exact in fp32), and
    the R3-rounded weight gradient appears in the first Adam moment as
    (1 - beta1) dW; the loss and goodness agree to fp32 rounding."""
    import json
    import os
    gold = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_cases.json")))
    c = gold["bf16_forward_ties"]
    W, b = np.array(c["W"], np.float32), np.array(c["b"], np.float32)
    L = P.Layer(_t(W), _t(b), bf16_shadow=True)
    h = torch.empty(1, 4, device=DEV)
    g = torch.empty(1, device=DEV)
    hp = P.HParams(dtype=P.FF_BF16, norm_eps=0.0)
    P.ff_layer_forward(L, hp, _t(np.array(c["x"], np.float32)), h_out=h, goodness=g)
    np.testing.assert_array_equal(_np(h), np.array(c["h"], np.float32))
    np.testing.assert_allclose(_np(g), c["g"], rtol=1e-6)
    c = gold["bf16_step_r3"]
    # one unit, padded with three all-zero units (layer widths are multiples of 4):
    # their activities are 0, so they add nothing to the goodness and get dW = 0
    W = np.zeros((4, 8), np.float32)
    W[0] = c["W"][0]
    b = np.zeros(4, np.float32)
    L = P.Layer(_t(W), _t(b), bf16_shadow=True)
    g = torch.empty(2, device=DEV)
    loss = torch.empty(1, device=DEV)
    hp = P.HParams(dtype=P.FF_BF16, norm_eps=0.0, theta=c["theta"])
    P.ff_layer_step(L, hp, _t(np.array(c["x"], np.float32)), 1, 1, goodness=g, loss=loss)
    np.testing.assert_allclose(_np(g), c["g"], rtol=1e-6)
    np.testing.assert_allclose(_np(loss)[0], c["loss"], rtol=1e-6)
    one_m_b1 = np.float32(1) - np.float32(0.9)  # the device's (1 - beta1) in fp32
    dW = np.zeros((4, 8))
    dW[0] = c["dW"][0]
    np.testing.assert_allclose(_np(L.mW) / one_m_b1, dW, rtol=1e-6, atol=0)
    np.testing.assert_allclose(_np(L.mb)[0] / one_m_b1, c["db"][0], rtol=1e-5)
    np.testing.assert_array_equal(_np(L.mb)[1:], 0)


# ------------------------------------------------------------------ exact ties
def test_score_exact_ties_go_to_lowest_label(P):
    """Labels 3, 5 and 7 carry identical weight columns in layer 0, so their
    embeddings give the same activities and scores bit for bit (the label
    feature is the only difference); they are made the strongest labels, so
    every prediction is 3, and an AdaptiveNEG row whose true label is 3 takes 5."""
    x_base, _, _ = make_data(140, 500, 64)
    params = make_weights(141, (64, 48, 32))
    W0 = params[0][0].copy()
    col = np.abs(W0[:, 3]) + 0.5
    for c in (3, 5, 7):
        W0[:, c] = col
    params[0] = (W0, params[0][1])
    layers = [P.Layer(_t(W), _t(b)) for W, b in params]
    S = torch.empty(500, 10, device=DEV)
    _, pred = P.ff_score_labels(layers, P.HParams(), _t(x_base), 10, 0, scores=S)
    Sg = _np(S)
    np.testing.assert_array_equal(Sg[:, 3], Sg[:, 5])
    np.testing.assert_array_equal(Sg[:, 3], Sg[:, 7])
    S_ref, p_ref = O.score_labels([O.Layer.from_params(W, b) for W, b in params], x_base, 10,
                                  O.HParams(), 0)
    assert_goodness(Sg, S_ref, what="scores")
    # in the oracle the three agree to fp64 rounding (its sums take the label
    # term in a different position) and lead every other label
    tied = S_ref[:, [3, 5, 7]]
    np.testing.assert_allclose(tied, np.repeat(tied[:, :1], 3, axis=1), rtol=1e-12)
    assert np.all(tied.min(axis=1) > np.delete(S_ref, [3, 5, 7], axis=1).max(axis=1) * 1.001)
    np.testing.assert_array_equal(_np(pred), 3)
    labels = np.where(np.arange(500) % 2 == 0, 3, 5).astype(np.int32)
    _, y_neg = P.ff_adaptive_negatives(layers, P.HParams(), _t(x_base), _t(labels), 10, 0)
    np.testing.assert_array_equal(_np(y_neg), np.where(labels == 3, 5, 3))


# ------------------------------------------------------------------ checkpoint / resume
def test_checkpoint_resume_bitwise(P):
    """Two pipelined epochs in one call, against one epoch, a checkpoint of every
    layer's W, b, Adam moments and step count copied to host memory, fresh
    layers restored from it, and a second epoch: bit for bit the same weights,
    moments and loss trace."""
    hp = P.HParams(theta=2.0, lr=0.03)
    dims = (784, 256, 256, 128)
    x_base, y, y_neg = make_data(150, 900, dims[0])
    params = make_weights(151, dims)
    xd, yd, ynd = _t(x_base), _t(y), _t(y_neg)
    nc = -(-900 // 128)
    whole = [P.Layer(_t(W), _t(b)) for W, b in params]
    tw = torch.zeros(3, 2 * nc, device=DEV)
    P.ff_pipeline_epoch(whole, hp, xd, yd, ynd, 10, 128, 2, P.FF_PIPELINED, loss_trace=tw)
    first = [P.Layer(_t(W), _t(b)) for W, b in params]
    t1 = torch.zeros(3, nc, device=DEV)
    P.ff_pipeline_epoch(first, hp, xd, yd, ynd, 10, 128, 1, P.FF_PIPELINED, loss_trace=t1)
    ckpt = [{k: _np(getattr(L, k)).copy() for k in ("W", "b", "mW", "vW", "mb", "vb")}
            | {"step": L.step} for L in first]
    del first
    torch.cuda.synchronize()
    resumed = []
    for c in ckpt:
        L = P.Layer(_t(c["W"]), _t(c["b"]))
        for k in ("mW", "vW", "mb", "vb"):
            getattr(L, k).copy_(_t(c[k]))
        L.step = c["step"]
        resumed.append(L)
    t2 = torch.zeros(3, nc, device=DEV)
    P.ff_pipeline_epoch(resumed, hp, xd, yd, ynd, 10, 128, 1, P.FF_PIPELINED, loss_trace=t2)
    np.testing.assert_array_equal(np.concatenate([_np(t1), _np(t2)], axis=1), _np(tw))
    for a, b in zip(whole, resumed):
        assert a.step == b.step == 2 * nc
        for k in ("W", "b", "mW", "vW", "mb", "vb"):
            np.testing.assert_array_equal(_np(getattr(a, k)), _np(getattr(b, k)))


# ------------------------------------------------------------------ failure handling
def test_failed_weight_update_launch_keeps_the_step(P):
    """A layer step whose weight-update launch fails (forced by the test hook,
    which enqueues nothing for it) returns FF_ERR_HIP with the Adam step count
    and the weights unchanged; retried, the step matches a step that never
    failed, bit for bit (same bias correction t = 1)."""
    x = _t(random_matrix(160, 256, 96, 0, 1, 0.5))
    (W, b), = make_weights(161, (96, 64))
    L, ok = P.Layer(_t(W), _t(b)), P.Layer(_t(W), _t(b))
    hp = P.HParams()
    P.ff_fail_next_launch("dw_adam")
    try:
        with pytest.raises(P.FFError) as e:
            P.ff_layer_step(L, hp, x, 128, 128)
    finally:
        P.ff_fail_next_launch(None)
    assert e.value.status == P.FF_ERR_HIP and L.step == 0
    np.testing.assert_array_equal(_np(L.W), W)
    P.ff_layer_step(L, hp, x, 128, 128)
    P.ff_layer_step(ok, hp, x, 128, 128)
    assert L.step == ok.step == 1
    for k in ("W", "b", "mW", "vW"):
        np.testing.assert_array_equal(_np(getattr(L, k)), _np(getattr(ok, k)))


def test_caller_streams_keep_the_workspace_they_use(P):
    """An epoch on caller streams (none of them the current one) with the
    workspace allocated by the binding: the binding marks it in use by those
    streams, so memory allocated and overwritten on the current stream right
    after the call does not land on it; the result equals the one-stream run."""
    hp = P.HParams(theta=2.0, lr=0.03)
    dims = (784, 512, 512, 512)
    x_base, y, y_neg = make_data(170, 2000, dims[0])
    params = make_weights(171, dims)
    xd, yd, ynd = _t(x_base), _t(y), _t(y_neg)
    cur = torch.cuda.current_stream()
    ref = [P.Layer(_t(W), _t(b)) for W, b in params]
    P.ff_pipeline_epoch(ref, hp, xd, yd, ynd, 10, 256, 2, P.FF_PIPELINED, streams=[cur] * 3)
    torch.cuda.synchronize()
    side = [torch.cuda.Stream() for _ in range(3)]
    for s_ in side:
        s_.wait_stream(cur)
    layers = [P.Layer(_t(W), _t(b)) for W, b in params]
    for s_ in side:
        s_.wait_stream(cur)
    need = P.ff_pipeline_workspace_size(layers, 2000, 256, P.FF_PIPELINED)
    P.ff_pipeline_epoch(layers, hp, xd, yd, ynd, 10, 256, 2, P.FF_PIPELINED, streams=side)
    junk = torch.empty(need // 4 + 1024, device=DEV)
    junk.fill_(float("nan"))
    for s_ in side:
        cur.wait_stream(s_)
    torch.cuda.synchronize()
    for a, b in zip(layers, ref):
        np.testing.assert_array_equal(_np(a.W), _np(b.W))


# ------------------------------------------------------------------ AdaptiveNEG chapters
def _adaptive_chapters(P, assignment, n_streams, bf16=False, seed=180):
    dims = (64, 96, 80, 48)
    n, chunk, E, S, cool = 300, 64, 4, 2, 2
    x_base, y, _ = make_data(seed, n, dims[0])
    params = make_weights(seed + 1, dims)
    # layer 0's label columns scaled apart (factors 1 + 0.4 k over a fixed
    # permutation): every sample's scores then separate by more than 1e-4, so
    # each AdaptiveNEG choice is decided and both sides train on the same labels
    W0 = params[0][0].copy()
    W0[:, :10] *= (1.0 + 0.4 * np.random.default_rng(seed + 2).permutation(10))[None, :]
    params[0] = (W0.astype(np.float32), params[0][1])
    layers = [P.Layer(_t(W), _t(b), bf16_shadow=bf16) for W, b in params]
    nc = -(-n // chunk)
    trace = torch.zeros(len(layers), E * nc, device=DEV)
    hp = P.HParams(lr=0.03, dtype=P.FF_BF16 if bf16 else P.FF_F32)
    negs = P.ff_chapter_train_adaptive(layers, hp, _t(x_base), _t(y), 10, chunk, E, S, cool,
                                       assignment, 0, n_streams=n_streams, loss_trace=trace)
    torch.cuda.synchronize()
    return layers, _np(trace), _np(negs), (x_base, y, params, chunk, E, S, cool)


@pytest.mark.parametrize("assignment,n_streams", [(0, None), (1, 2)])
def test_adaptive_chapters_parity(P, assignment, n_streams):
    """AdaptiveNEG chapters on the device against the oracle's: each chapter's
    negatives (bit-exact on rows whose two best wrong labels are decided at
    1e-4, never the true label), the loss trace and the weights."""
    layers, trace, negs, (x_base, y, params, chunk, E, S, cool) = _adaptive_chapters(
        P, assignment, n_streams)
    rec, scores = [], []
    hp = O.HParams(lr=0.03)

    def run(Ls, obs):
        draw = O.adaptive_chapter_negatives(x_base, y, 10, hp, record=rec if obs else None)

        def negatives(c, Ls_):
            if obs:
                scores.append(O.score_labels(Ls_, x_base, 10, hp, 0)[0])
            return draw(c, Ls_)
        return O.chapter_train(Ls, x_base, y, negatives, 10, chunk, E, S, cool, hp, on_step=obs)
    # later layers train on the published output of trained layers: weights
    # within what a float32 evaluation of the same chapters does; layer 0
    # (its inputs given) at the elementwise bar
    refs, cW, cb = _run_check(layers, trace, params, 0.03, run, bf16=False)
    for c in range(S):
        assert assert_negatives(negs[c], scores[c], rec[c], y) == len(y)  # every row decided
        np.testing.assert_array_equal(negs[c], rec[c])
    assert len(np.unique(np.concatenate(rec))) > 2
    _assert_trained(layers[:1], refs[:1], cW, cb, 0.03)


def test_adaptive_chapters_assignments_agree_bitwise(P):
    a, ta, na, _ = _adaptive_chapters(P, 0, None)
    b, tb, nb, _ = _adaptive_chapters(P, 1, 3)
    np.testing.assert_array_equal(na, nb)
    np.testing.assert_array_equal(ta, tb)
    for x, y_ in zip(a, b):
        np.testing.assert_array_equal(_np(x.W), _np(y_.W))
