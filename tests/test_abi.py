"""C-ABI checks that need no GPU: the library loads, exports every symbol that
include/ff.h declares, and rejects bad arguments on the host before any launch."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ff.h")


@pytest.fixture(scope="module")
def P():
    import paper_2404_08573_amd as P
    P.LIB  # raises ImportError if libff.so is not built
    return P


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ff_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_entry_points():
    names = declared_symbols()
    for must in ["ff_layer_step", "ff_score_labels", "ff_pipeline_epoch", "ff_layer_forward",
                 "ff_embed_labels", "ff_step_workspace_size", "ff_score_workspace_size",
                 "ff_pipeline_workspace_size", "ff_status_string", "ff_last_error",
                 "ff_refresh_bf16_shadow", "ff_adaptive_negatives"]:
        assert must in names


def test_library_exports_every_declared_symbol(P):
    lib = ctypes.CDLL(P._lib.LIB_PATH)
    for name in declared_symbols():
        assert hasattr(lib, name), name
    assert set(P._lib.EXPORTS) == set(declared_symbols())


def test_status_strings(P):
    L = P.LIB
    assert L.ff_status_string(0) == b"FF_OK"
    assert L.ff_status_string(-3) == b"FF_ERR_WORKSPACE"
    assert L.ff_status_string(7) == b"FF_UNKNOWN_STATUS"


def test_workspace_sizes(P):
    a = P.ff_step_workspace_size(2048, 2000, 2000, P.FF_F32)
    b = P.ff_step_workspace_size(1024, 2000, 2000, P.FF_F32)
    c = P.ff_step_workspace_size(2048, 2000, 2000, P.FF_BF16)
    assert a > b > 0 and c > 0
    assert a >= 2048 * 2000 * 4 * 2  # normalised input + activities
    assert c >= 2048 * 2000 * (2 + 4)  # bf16: bf16 normalised input + fp32 activities
    assert P.ff_step_workspace_size(0, 10, 10, 0) == 0


def _layer(P, d_in=16, d_out=8, bad=None):
    fake = ctypes.c_void_p(256)  # never dereferenced: validation fails first
    kw = dict(d_in=d_in, d_out=d_out, W=fake, b=fake, mW=fake, vW=fake, mb=fake, vb=fake,
              W_bf16=None, step=0)
    if bad:
        kw.update(bad)
    return P._lib.ff_layer(**kw)


def _hp(P, **kw):
    h = P.HParams(**kw)
    return h.c()


@pytest.mark.parametrize("case,status", [
    ("n_pos0", -1), ("n_neg0", -1), ("x_null", -1), ("d_in_odd", -2), ("d_out0", -1),
    ("no_moments", -1), ("bad_dtype", -1), ("bf16_no_shadow", -1), ("ws_null", -3),
    ("ws_small", -3), ("beta_out_of_range", -1), ("too_wide", -2)])
def test_layer_step_rejects_on_host(P, case, status):
    L = _layer(P)
    hp = _hp(P)
    x = ctypes.c_void_p(4096)
    n_pos, n_neg, ws, ws_bytes = 4, 4, ctypes.c_void_p(1 << 20), 1 << 30
    if case == "n_pos0":
        n_pos = 0
    elif case == "n_neg0":
        n_neg = 0
    elif case == "x_null":
        x = None
    elif case == "d_in_odd":
        L = _layer(P, d_in=15)
    elif case == "d_out0":
        L = _layer(P, d_out=0)
    elif case == "no_moments":
        L = _layer(P, bad=dict(mW=None))
    elif case == "bad_dtype":
        hp = _hp(P, dtype=5)
    elif case == "bf16_no_shadow":
        hp = _hp(P, dtype=P.FF_BF16)
    elif case == "ws_null":
        ws = None
    elif case == "ws_small":
        ws_bytes = 100
    elif case == "beta_out_of_range":
        hp = _hp(P, beta2=1.0)
    elif case == "too_wide":
        L = _layer(P, d_in=(1 << 20) + 4)  # past FF_MAX_WIDTH
    st = P.LIB.ff_layer_step(ctypes.byref(L), ctypes.byref(hp), x, n_pos, n_neg, 0, None, None,
                             None, ws, ws_bytes, None)
    assert st == status, P.LIB.ff_last_error()
    assert L.step == 0  # nothing enqueued, no state change
    assert P.LIB.ff_last_error()


def test_score_labels_rejects_on_host(P):
    layers = (P._lib.ff_layer * 2)(_layer(P, 16, 8), _layer(P, 12, 8))  # does not chain
    hp = _hp(P)
    ws = ctypes.c_void_p(1 << 20)
    st = P.LIB.ff_score_labels(layers, 2, 0, ctypes.byref(hp), ctypes.c_void_p(4096), 5, 10, None,
                               ctypes.c_void_p(8192), ws, 1 << 30, None)
    assert st == -1 and b"does not match" in P.LIB.ff_last_error()
    layers = (P._lib.ff_layer * 2)(_layer(P, 16, 8), _layer(P, 8, 8))
    st = P.LIB.ff_score_labels(layers, 2, 2, ctypes.byref(hp), ctypes.c_void_p(4096), 5, 10, None,
                               ctypes.c_void_p(8192), ws, 1 << 30, None)
    assert st == -1 and b"first_scored_layer" in P.LIB.ff_last_error()
    st = P.LIB.ff_score_labels(layers, 2, 0, ctypes.byref(hp), ctypes.c_void_p(4096), 5, 17, None,
                               ctypes.c_void_p(8192), ws, 1 << 30, None)
    assert st == -1 and b"n_classes" in P.LIB.ff_last_error()
    # n == 0 is a no-op that succeeds without touching the device
    st = P.LIB.ff_score_labels(layers, 2, 0, ctypes.byref(hp), None, 0, 10, None, None, None, 0,
                               None)
    assert st == 0


def test_adaptive_negatives_rejects_on_host(P):
    layers = (P._lib.ff_layer * 2)(_layer(P, 16, 8), _layer(P, 8, 8))
    hp = _hp(P)
    ws = ctypes.c_void_p(1 << 20)
    args = [layers, 2, 0, ctypes.byref(hp), ctypes.c_void_p(4096), ctypes.c_void_p(4096), 5, 10,
            None, ctypes.c_void_p(8192), ws, 1 << 30, None]
    one = list(args)
    one[7] = 1
    assert P.LIB.ff_adaptive_negatives(*one) == -1
    assert b"no wrong label" in P.LIB.ff_last_error()
    nolab = list(args)
    nolab[5] = None
    assert P.LIB.ff_adaptive_negatives(*nolab) == -1
    noout = list(args)
    noout[9] = None
    assert P.LIB.ff_adaptive_negatives(*noout) == -1
    small = list(args)
    small[11] = 16
    assert P.LIB.ff_adaptive_negatives(*small) == -3


def test_head_rejects_on_host(P):
    layers = (P._lib.ff_layer * 3)(_layer(P, 16, 12), _layer(P, 12, 8), _layer(P, 8, 8))
    hp = _hp(P)
    fake = ctypes.c_void_p(256)

    def head(d_feat=16, C=10, **kw):
        f = dict(d_feat=d_feat, n_classes=C, W=fake, b=fake, mW=fake, vW=fake, mb=fake, vb=fake,
                 step=0)
        f.update(kw)
        return P._lib.ff_head(**f)

    ws = ctypes.c_void_p(1 << 20)

    def step(h, first=1, labels=ctypes.c_void_p(4096), n=5):
        return P.LIB.ff_head_step(layers, 3, first, ctypes.byref(hp), ctypes.byref(h),
                                  ctypes.byref(hp), ctypes.c_void_p(4096), labels, n, None, ws,
                                  1 << 30, None)

    # every case is rejected on the host before anything is enqueued
    for h, first, status, msg in [(head(d_feat=12), 1, -1, b"d_feat"),
                                  (head(), 3, -1, b"first_layer"),
                                  (head(C=1), 1, -1, b"n_classes"),
                                  (head(C=17), 1, -1, b"n_classes"),
                                  (head(mW=None), 1, -1, b"moment")]:
        assert step(h, first) == status, msg
        assert msg in P.LIB.ff_last_error()
    assert step(head(), labels=None) == -1
    h = head()
    assert P.LIB.ff_head_step(layers, 3, 1, ctypes.byref(hp), ctypes.byref(h), ctypes.byref(hp),
                              ctypes.c_void_p(4096), ctypes.c_void_p(4096), 5, None, ws, 16,
                              None) == -3
    assert h.step == 0
    assert P.LIB.ff_head_predict(layers, 3, 1, ctypes.byref(hp), ctypes.byref(head()),
                                 ctypes.c_void_p(4096), 5, None, None, ws, 1 << 30, None) == -1
    assert P.LIB.ff_head_workspace_size(layers, 3, 3, 5, 10, 0) == 0  # first_layer out of range
    assert P.LIB.ff_head_workspace_size(layers, 3, 1, 5, 10, 0) > 5 * (12 + 8 + 8) * 4


def test_chapter_rejects_on_host(P):
    layers = (P._lib.ff_layer * 2)(_layer(P, 16, 8), _layer(P, 8, 8))
    hp = _hp(P)
    streams = (ctypes.c_void_p * 2)(None, None)

    def call(epochs=4, splits=2, assignment=0, n_streams=2, ws_bytes=1 << 30):
        return P.LIB.ff_chapter_train(layers, 2, ctypes.byref(hp), ctypes.c_void_p(4096),
                                      ctypes.c_void_p(4096), ctypes.c_void_p(4096), 100, 10, 32,
                                      epochs, splits, 2, assignment, n_streams, streams, None,
                                      ctypes.c_void_p(1 << 20), ws_bytes)

    assert call(epochs=5) == -1  # not a multiple of splits
    assert call(assignment=2) == -1
    assert call(n_streams=1) == -1  # Single-Layer needs one stream per layer
    assert call(ws_bytes=10) == -3
    assert layers[0].step == 0 and layers[1].step == 0


def test_chapter_adaptive_rejects_on_host(P):
    layers = (P._lib.ff_layer * 2)(_layer(P, 16, 8), _layer(P, 8, 8))
    hp = _hp(P)
    streams = (ctypes.c_void_p * 2)(None, None)

    def call(n_classes=10, first=0, epochs=4, ws_bytes=1 << 30, y_neg=ctypes.c_void_p(4096)):
        return P.LIB.ff_chapter_train_adaptive(layers, 2, ctypes.byref(hp), ctypes.c_void_p(4096),
                                               ctypes.c_void_p(4096), y_neg, 100, n_classes, 32,
                                               epochs, 2, 2, 0, first, 2, streams, None,
                                               ctypes.c_void_p(1 << 20), ws_bytes)

    assert call(n_classes=1) == -1  # no wrong label to choose
    assert call(first=2) == -1  # first_scored_layer past the last layer
    assert call(epochs=3) == -1
    assert call(y_neg=None) == -1
    need = P.LIB.ff_chapter_adaptive_workspace_size(layers, 2, 100, 10, 32, 2, 0)
    assert need > P.LIB.ff_chapter_workspace_size(layers, 2, 100, 32, 2, 0)
    assert call(ws_bytes=need - 512) == -3
    assert layers[0].step == 0 and layers[1].step == 0


def test_failed_launch_leaves_the_step_count(P):
    """A launch that fails (forced by the test hook before anything is
    enqueued) makes the entry point return FF_ERR_HIP with the Adam step count
    unchanged; the hook fires once, and -1 disarms it."""
    L = _layer(P)
    hp = _hp(P)
    assert P.LIB.ff_fail_next_launch(99) == -1
    assert P.LIB.ff_fail_next_launch(1) == 0  # the forward product
    try:
        # normalised fp32 rows: the forward product is the step's first launch
        st = P.LIB.ff_layer_step(ctypes.byref(L), ctypes.byref(hp), ctypes.c_void_p(4096), 4, 4,
                                 1, None, None, None, ctypes.c_void_p(1 << 20), 1 << 30, None)
        assert st == -4 and L.step == 0
        assert b"failed" in P.LIB.ff_last_error()
    finally:
        assert P.LIB.ff_fail_next_launch(-1) == 0


def test_pipeline_rejects_on_host(P):
    layers = (P._lib.ff_layer * 2)(_layer(P, 16, 8), _layer(P, 8, 8))
    hp = _hp(P)
    streams = (ctypes.c_void_p * 2)(None, None)
    args = [layers, 2, ctypes.byref(hp), ctypes.c_void_p(4096), ctypes.c_void_p(4096),
            ctypes.c_void_p(4096), 100, 10, 32, 1, 1, streams, None, ctypes.c_void_p(1 << 20),
            1 << 30]
    bad_sched = list(args)
    bad_sched[10] = 3
    assert P.LIB.ff_pipeline_epoch(*bad_sched) == -1
    zero_chunk = list(args)
    zero_chunk[8] = 0
    assert P.LIB.ff_pipeline_epoch(*zero_chunk) == -1
    small_ws = list(args)
    small_ws[14] = 10
    assert P.LIB.ff_pipeline_epoch(*small_ws) == -3
    assert layers[0].step == 0 and layers[1].step == 0


def test_embed_rejects_on_host(P):
    L = P.LIB
    assert L.ff_embed_labels(ctypes.c_void_p(64), ctypes.c_void_p(64), 3, 8, 10,
                             ctypes.c_void_p(64), None) == -1  # n_classes > d
    assert L.ff_embed_labels(ctypes.c_void_p(64), ctypes.c_void_p(64), 3, 10, 4,
                             ctypes.c_void_p(64), None) == -2  # d not a multiple of 4
    assert L.ff_embed_labels(None, None, 0, 12, 10, None, None) == 0  # empty


def test_graft_build_entry_binds_exports(P, monkeypatch):
    """__graft_entry__.build() after its compile step (stubbed here: the library
    is already built) must load the library and bind every export."""
    import importlib
    import sys
    sys.path.insert(0, ROOT)
    import paper_2404_08573_amd.build as B
    monkeypatch.setattr(B, "build", lambda *a, **k: None)
    entry = importlib.import_module("__graft_entry__")
    entry.build()


STRUCTS = {  # C struct -> the binding's ctypes class name
    "ff_layer": "ff_layer", "ff_head": "ff_head", "ff_hparams": "ff_hparams",
    "ff_kernel_stats": "ff_kernel_stats", "ff_launch_record": "ff_launch_record"}
ENUMS = ["FF_F32", "FF_BF16", "FF_SEQUENTIAL", "FF_PIPELINED", "FF_SINGLE_LAYER",
         "FF_ALL_LAYERS", "FF_KERNEL_EMBED_NORM", "FF_KERNEL_FORWARD", "FF_KERNEL_LOSS",
         "FF_KERNEL_DW_ADAM", "FF_KERNEL_GOODNESS", "FF_KERNEL_ARGMAX", "FF_KERNEL_SHADOW",
         "FF_KERNEL_HEAD", "FF_KERNEL_TRANSPOSE", "FF_KERNEL_ADAM", "FF_KERNEL_KINDS"]


def test_binding_layouts_match_the_header(P, tmp_path):
    """Every struct the binding passes has the C header's size and field offsets
    (a C program compiled against include/ff.h prints them), and the binding's
    constants and kernel-kind names follow the header's enums."""
    import json
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("no C compiler")
    L = P._lib
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "ff.h"', 'int main(void) {',
             '  printf("{");']
    for c in STRUCTS:
        fields = [f for f, _ in getattr(L, STRUCTS[c])._fields_]
        offs = ", ".join(f'\\"{f}\\": %zu' for f in fields)
        args = ", ".join(f"offsetof({c}, {f})" for f in fields)
        lines.append(f'  printf("\\"{c}\\": {{\\"size\\": %zu, {offs}}}, ", sizeof({c}), {args});')
    for e in ENUMS:
        lines.append(f'  printf("\\"{e}\\": %d, ", (int){e});')
    lines += ['  printf("\\"end\\": 0}");', '  return 0;', '}']
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o",
                    str(exe)], check=True)
    got = json.loads(subprocess.run([str(exe)], check=True, capture_output=True,
                                    text=True).stdout)
    for c, cls in STRUCTS.items():
        ct = getattr(L, cls)
        assert got[c]["size"] == ctypes.sizeof(ct), c
        for f, _ in ct._fields_:
            assert got[c][f] == getattr(ct, f).offset, (c, f)
    assert (got["FF_F32"], got["FF_BF16"]) == (P.FF_F32, P.FF_BF16)
    assert (got["FF_SEQUENTIAL"], got["FF_PIPELINED"]) == (P.FF_SEQUENTIAL, P.FF_PIPELINED)
    assert (got["FF_SINGLE_LAYER"], got["FF_ALL_LAYERS"]) == (P.FF_SINGLE_LAYER,
                                                              P.FF_ALL_LAYERS)
    names = {"EMBED_NORM": "embed_norm", "FORWARD": "forward", "LOSS": "loss",
             "DW_ADAM": "dw_adam", "GOODNESS": "goodness", "ARGMAX": "argmax",
             "SHADOW": "bf16_shadow", "HEAD": "head", "TRANSPOSE": "transpose", "ADAM": "adam"}
    assert got["FF_KERNEL_KINDS"] == len(L.KERNEL_KINDS) == len(names)
    for e, n in names.items():
        assert L.KERNEL_KINDS[got["FF_KERNEL_" + e]] == n, e
