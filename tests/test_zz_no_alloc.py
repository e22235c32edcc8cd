"""The no-allocation layer step (ff_layer_step_noalloc) against ff_layer_step:
the same kernels, with the scratch in the library's fixed device array instead
of a caller workspace, so every output is bit for bit the same.  Two calls in
a row, the second on a smaller input (the scratch keeps the first call's
contents), fp32 and bf16; and the size limit is refused on the host."""
import ctypes

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from ffinputs import make_data, make_weights, random_matrix  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def P():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2404_08573_amd as P
    return P


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _np(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


@pytest.mark.parametrize("bf16", [False, True])
def test_noalloc_step_matches_the_workspace_step(P, bf16):
    hp = P.HParams(theta=2.0, lr=0.03, dtype=P.FF_BF16 if bf16 else P.FF_F32)
    (W, b), = make_weights(200, (784, 2000))
    a = P.Layer(_t(W), _t(b), bf16_shadow=bf16)   # no-allocation entry point
    r = P.Layer(_t(W), _t(b), bf16_shadow=bf16)   # workspace entry point
    for rows, seed, with_h in ((2048, 201, False), (300, 202, True)):
        x = _t(random_matrix(seed, rows, 784, 0, 1, 0.5))
        outs = []
        for L, noalloc in ((a, True), (r, False)):
            h = torch.full((rows, 2000), -1.0, device=DEV) if with_h else None
            g = torch.full((rows,), -1.0, device=DEV)
            loss = torch.full((1,), -1.0, device=DEV)
            if noalloc:
                P.ff_layer_step_noalloc(L, hp, x, rows // 2, rows - rows // 2, h_out=h,
                                        goodness=g, loss=loss)
            else:
                P.ff_layer_step(L, hp, x, rows // 2, rows - rows // 2, h_out=h, goodness=g,
                                loss=loss)
            outs.append([_np(t) for t in (g, loss) + ((h,) if with_h else ())])
        for u, v in zip(*outs):
            np.testing.assert_array_equal(u, v)
        assert a.step == r.step
        for k in ("W", "b", "mW", "vW", "mb", "vb") + (("W_bf16",) if bf16 else ()):
            np.testing.assert_array_equal(_np(getattr(a, k)), _np(getattr(r, k)))


def test_noalloc_step_refuses_what_does_not_fit(P):
    """4096 rows of a 3072 -> 3072 bf16 layer without h_out would need the
    activities in scratch (50 MB): refused before anything is enqueued."""
    (W, b), = make_weights(203, (3072, 3072))
    L = P.Layer(_t(W), _t(b), bf16_shadow=True)
    x = torch.zeros(4096, 3072, device=DEV)
    with pytest.raises(P.FFError) as e:
        P.ff_layer_step_noalloc(L, P.HParams(dtype=P.FF_BF16), x, 2048, 2048)
    assert e.value.status == P.FF_ERR_UNSUPPORTED and L.step == 0
    h = torch.empty(4096, 3072, device=DEV)
    P.ff_layer_step_noalloc(L, P.HParams(dtype=P.FF_BF16), x + 1.0, 2048, 2048, h_out=h)
    assert L.step == 1
