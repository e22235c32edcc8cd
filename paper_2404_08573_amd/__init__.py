"""MI355X (gfx950) Forward-Forward hot path: HIP kernels behind the C ABI of include/ff.h.

The entry points (``ff_layer_step``, ``ff_score_labels``, ``ff_pipeline_epoch``,
...) live in ``paper_2404_08573_amd._lib`` and are re-exported here on first
access.  Accessing them without a built ``libff.so`` raises ImportError: there
is no CPU fallback.
"""
import importlib


def __getattr__(name):
    if name.startswith("__"):
        raise AttributeError(name)
    mod = importlib.import_module(__name__ + "._lib")
    if name == "_lib":
        return mod
    try:
        return getattr(mod, name)
    except AttributeError:
        raise AttributeError(f"module {__name__!r} has no attribute {name!r}") from None
