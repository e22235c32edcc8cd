"""ctypes binding of libff.so (include/ff.h).  Argument marshalling only.

Every function here has the name of the C entry point it calls and does no
arithmetic of the method: it checks tensor devices/dtypes/shapes, passes raw
device pointers and the current HIP stream, and raises ``FFError`` on a
non-OK status.  PyTorch provides device memory and streams.  The library must
have been built (``__graft_entry__.build()``); importing without it raises.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from ctypes import POINTER, c_float, c_int32, c_int64, c_size_t, c_void_p
from typing import List, Optional, Sequence

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libff.so")

FF_OK, FF_ERR_INVALID_ARG, FF_ERR_UNSUPPORTED, FF_ERR_WORKSPACE, FF_ERR_HIP = 0, -1, -2, -3, -4
FF_F32, FF_BF16 = 0, 1
FF_SEQUENTIAL, FF_PIPELINED = 0, 1
FF_SINGLE_LAYER, FF_ALL_LAYERS = 0, 1

EXPORTS = ["ff_status_string", "ff_last_error", "ff_embed_labels", "ff_step_workspace_size",
           "ff_layer_forward", "ff_layer_step", "ff_refresh_bf16_shadow",
           "ff_score_workspace_size", "ff_score_labels", "ff_adaptive_negatives",
           "ff_head_workspace_size", "ff_head_step", "ff_head_predict",
           "ff_chapter_workspace_size", "ff_chapter_train",
           "ff_chapter_adaptive_workspace_size", "ff_chapter_train_adaptive",
           "ff_po_step_workspace_size", "ff_po_layer_step", "ff_po_epoch_workspace_size",
           "ff_po_epoch", "ff_po_predict_workspace_size", "ff_po_predict",
           "ff_pipeline_workspace_size",
           "ff_pipeline_epoch", "ff_profile_start", "ff_profile_stop", "ff_profile_stop_launches",
           "ff_fail_next_launch",
           "ff_layer_step_noalloc"]

KERNEL_KINDS = ["embed_norm", "forward", "loss", "dw_adam", "goodness", "argmax", "bf16_shadow",
                "head", "transpose", "adam"]


class FFError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{LIB.ff_status_string(status).decode()}: {msg}")
        self.status = status


class ff_layer(ctypes.Structure):
    _fields_ = [("d_in", c_int32), ("d_out", c_int32), ("W", c_void_p), ("b", c_void_p),
                ("mW", c_void_p), ("vW", c_void_p), ("mb", c_void_p), ("vb", c_void_p),
                ("W_bf16", c_void_p), ("step", c_int64)]


class ff_head(ctypes.Structure):
    _fields_ = [("d_feat", c_int32), ("n_classes", c_int32), ("W", c_void_p), ("b", c_void_p),
                ("mW", c_void_p), ("vW", c_void_p), ("mb", c_void_p), ("vb", c_void_p),
                ("step", c_int64)]


class ff_kernel_stats(ctypes.Structure):
    _fields_ = [("launches", c_int64), ("total_ms", ctypes.c_double), ("flops", ctypes.c_double),
                ("bytes", ctypes.c_double)]


class ff_launch_record(ctypes.Structure):
    _fields_ = [("kind", c_int32), ("m", c_int32), ("n", c_int32), ("k", c_int32),
                ("aux", c_int32), ("ms", c_float), ("flops", ctypes.c_double),
                ("bytes", ctypes.c_double)]


class ff_hparams(ctypes.Structure):
    _fields_ = [("theta", c_float), ("lr", c_float), ("beta1", c_float), ("beta2", c_float),
                ("adam_eps", c_float), ("norm_eps", c_float), ("dtype", c_int32)]


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                          "(python -m paper_2404_08573_amd.build); there is no fallback path")
    lib = ctypes.CDLL(LIB_PATH)
    P = c_void_p
    sig = {
        "ff_status_string": (ctypes.c_char_p, [c_int32]),
        "ff_last_error": (ctypes.c_char_p, []),
        "ff_embed_labels": (c_int32, [P, P, c_int32, c_int32, c_int32, P, P]),
        "ff_step_workspace_size": (c_size_t, [c_int32, c_int32, c_int32, c_int32]),
        "ff_layer_forward": (c_int32, [POINTER(ff_layer), POINTER(ff_hparams), P, c_int32, c_int32,
                                       P, P, P, c_size_t, P]),
        "ff_layer_step": (c_int32, [POINTER(ff_layer), POINTER(ff_hparams), P, c_int32, c_int32,
                                    c_int32, P, P, P, P, c_size_t, P]),
        "ff_refresh_bf16_shadow": (c_int32, [POINTER(ff_layer), P]),
        "ff_score_workspace_size": (c_size_t, [POINTER(ff_layer), c_int32, c_int32, c_int32,
                                               c_int32]),
        "ff_score_labels": (c_int32, [POINTER(ff_layer), c_int32, c_int32, POINTER(ff_hparams), P,
                                      c_int32, c_int32, P, P, P, c_size_t, P]),
        "ff_adaptive_negatives": (c_int32, [POINTER(ff_layer), c_int32, c_int32,
                                            POINTER(ff_hparams), P, P, c_int32, c_int32, P, P, P,
                                            c_size_t, P]),
        "ff_head_workspace_size": (c_size_t, [POINTER(ff_layer), c_int32, c_int32, c_int32,
                                              c_int32, c_int32]),
        "ff_head_step": (c_int32, [POINTER(ff_layer), c_int32, c_int32, POINTER(ff_hparams),
                                   POINTER(ff_head), POINTER(ff_hparams), P, P, c_int32, P, P,
                                   c_size_t, P]),
        "ff_head_predict": (c_int32, [POINTER(ff_layer), c_int32, c_int32, POINTER(ff_hparams),
                                      POINTER(ff_head), P, c_int32, P, P, P, c_size_t, P]),
        "ff_chapter_workspace_size": (c_size_t, [POINTER(ff_layer), c_int32, c_int32, c_int32,
                                                 c_int32, c_int32]),
        "ff_chapter_train": (c_int32, [POINTER(ff_layer), c_int32, POINTER(ff_hparams), P, P, P,
                                       c_int32, c_int32, c_int32, c_int32, c_int32, c_int32,
                                       c_int32, c_int32, POINTER(c_void_p), P, P, c_size_t]),
        "ff_chapter_adaptive_workspace_size": (c_size_t, [POINTER(ff_layer), c_int32, c_int32,
                                                          c_int32, c_int32, c_int32, c_int32]),
        "ff_chapter_train_adaptive": (c_int32, [POINTER(ff_layer), c_int32, POINTER(ff_hparams), P,
                                                P, P, c_int32, c_int32, c_int32, c_int32,
                                                c_int32, c_int32, c_int32, c_int32, c_int32,
                                                POINTER(c_void_p), P, P, c_size_t]),
        "ff_po_step_workspace_size": (c_size_t, [c_int32] * 5),
        "ff_po_layer_step": (c_int32, [POINTER(ff_layer), POINTER(ff_head), POINTER(ff_hparams),
                                       POINTER(ff_hparams), P, P, c_int32, c_int32, P, P, P,
                                       c_size_t, P]),
        "ff_po_epoch_workspace_size": (c_size_t, [POINTER(ff_layer), c_int32, c_int32, c_int32,
                                                  c_int32, c_int32, c_int32]),
        "ff_po_epoch": (c_int32, [POINTER(ff_layer), POINTER(ff_head), c_int32,
                                  POINTER(ff_hparams), POINTER(ff_hparams), P, P, c_int32,
                                  c_int32, c_int32, c_int32, c_int32, POINTER(c_void_p), P, P,
                                  c_size_t]),
        "ff_po_predict_workspace_size": (c_size_t, [POINTER(ff_layer), c_int32, c_int32, c_int32,
                                                    c_int32]),
        "ff_po_predict": (c_int32, [POINTER(ff_layer), POINTER(ff_head), c_int32,
                                    POINTER(ff_hparams), P, c_int32, c_int32, P, P, P, c_size_t,
                                    P]),
        "ff_pipeline_workspace_size": (c_size_t, [POINTER(ff_layer), c_int32, c_int32, c_int32,
                                                  c_int32, c_int32]),
        "ff_pipeline_epoch": (c_int32, [POINTER(ff_layer), c_int32, POINTER(ff_hparams), P, P, P,
                                        c_int32, c_int32, c_int32, c_int32, c_int32,
                                        POINTER(c_void_p), P, P, c_size_t]),
        "ff_profile_start": (c_int32, [c_int32, ctypes.c_uint32]),
        "ff_profile_stop": (c_int32, [POINTER(ff_kernel_stats)]),
        "ff_profile_stop_launches": (c_int32, [POINTER(ff_kernel_stats), POINTER(ff_launch_record),
                                               c_int32, POINTER(c_int32)]),
        "ff_fail_next_launch": (c_int32, [c_int32]),
        "ff_layer_step_noalloc": (c_int32, [POINTER(ff_layer), POINTER(ff_hparams), P, c_int32,
                                            c_int32, c_int32, P, P, P, P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype, f.argtypes = res, args
    return lib


LIB = _load()


def _check(status: int):
    if status != FF_OK:
        raise FFError(status, LIB.ff_last_error().decode())


def _ptr(t: Optional[torch.Tensor], dtype=None, numel=None, name="tensor"):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} has {t.numel()} elements, needs {numel}")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream if isinstance(s, torch.cuda.Stream) else int(s)


def _hold(tensors, streams):
    """Buffers this binding allocated (on the current stream) and handed to
    work enqueued on `streams`: mark them in use by every stream other than the
    current one, so that torch's caching allocator does not hand their memory
    to a later allocation before that work has finished."""
    cur = torch.cuda.current_stream().cuda_stream
    for s in streams:
        if s is None:
            continue
        if not isinstance(s, torch.cuda.Stream):
            s = torch.cuda.ExternalStream(int(s))
        if s.cuda_stream != cur:
            for t in tensors:
                if t is not None:
                    t.record_stream(s)


@dataclasses.dataclass
class HParams:
    theta: float = 2.0
    lr: float = 0.03
    beta1: float = 0.9
    beta2: float = 0.999
    adam_eps: float = 1e-8
    norm_eps: float = 1e-8
    dtype: int = FF_F32

    def c(self) -> ff_hparams:
        return ff_hparams(self.theta, self.lr, self.beta1, self.beta2, self.adam_eps,
                          self.norm_eps, self.dtype)


class Layer:
    """Device buffers of one FF layer (fp32 master W, b, Adam moments, optional bf16 shadow)."""

    def __init__(self, W: torch.Tensor, b: torch.Tensor, bf16_shadow: bool = False):
        dev = W.device
        self.W = W.detach().to(dev, torch.float32).contiguous().clone()
        self.b = b.detach().to(dev, torch.float32).contiguous().clone()
        self.mW = torch.zeros_like(self.W)
        self.vW = torch.zeros_like(self.W)
        self.mb = torch.zeros_like(self.b)
        self.vb = torch.zeros_like(self.b)
        self.W_bf16 = torch.empty(self.W.shape, dtype=torch.int16, device=dev) if bf16_shadow else None
        self.step = 0
        self.d_out, self.d_in = self.W.shape
        if bf16_shadow:
            ff_refresh_bf16_shadow(self)

    def c(self) -> ff_layer:
        return ff_layer(self.d_in, self.d_out, self.W.data_ptr(), self.b.data_ptr(),
                        self.mW.data_ptr(), self.vW.data_ptr(), self.mb.data_ptr(),
                        self.vb.data_ptr(),
                        self.W_bf16.data_ptr() if self.W_bf16 is not None else None, self.step)


class Head:
    """Device buffers of the softmax prediction layer: W [C][d_feat], b [C], Adam moments."""

    def __init__(self, W: torch.Tensor, b: torch.Tensor):
        self.W = W.detach().to(torch.float32).contiguous().clone()
        self.b = b.detach().to(self.W.device, torch.float32).contiguous().clone()
        self.mW = torch.zeros_like(self.W)
        self.vW = torch.zeros_like(self.W)
        self.mb = torch.zeros_like(self.b)
        self.vb = torch.zeros_like(self.b)
        self.step = 0
        self.n_classes, self.d_feat = self.W.shape

    def c(self) -> ff_head:
        return ff_head(self.d_feat, self.n_classes, self.W.data_ptr(), self.b.data_ptr(),
                       self.mW.data_ptr(), self.vW.data_ptr(), self.mb.data_ptr(),
                       self.vb.data_ptr(), self.step)


def _layers_c(layers: Sequence[Layer]):
    arr = (ff_layer * len(layers))(*[L.c() for L in layers])
    return arr


def workspace(nbytes: int, device="cuda") -> torch.Tensor:
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


# ----------------------------------------------------------------------------- entry points
def ff_embed_labels(x_base: torch.Tensor, labels: torch.Tensor, n_classes: int,
                    out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    rows, d = x_base.shape
    mine = [torch.empty_like(x_base)] if out is None else []
    out = mine[0] if mine else out
    _hold(mine, [stream])
    _check(LIB.ff_embed_labels(_ptr(x_base, torch.float32, name="x_base"),
                                _ptr(labels, torch.int32, rows, "labels"), rows, d, n_classes,
                                _ptr(out, torch.float32, rows * d, "out"), _stream(stream)))
    return out


def ff_step_workspace_size(rows: int, d_in: int, d_out: int, dtype: int = FF_F32) -> int:
    return LIB.ff_step_workspace_size(rows, d_in, d_out, dtype)


def ff_layer_forward(layer: Layer, hp: HParams, x: torch.Tensor, x_normalised: bool = False,
                     h_out: Optional[torch.Tensor] = None, goodness: Optional[torch.Tensor] = None,
                     ws: Optional[torch.Tensor] = None, stream=None):
    rows = x.shape[0]
    if ws is None:
        ws = workspace(ff_step_workspace_size(max(rows, 1), layer.d_in, layer.d_out, hp.dtype),
                       x.device)
        _hold([ws], [stream])
    Lc = layer.c()
    _check(LIB.ff_layer_forward(ctypes.byref(Lc), ctypes.byref(hp.c()),
                                 _ptr(x, torch.float32, rows * layer.d_in, "x"), rows,
                                 int(x_normalised), _ptr(h_out, torch.float32, rows * layer.d_out,
                                                         "h_out"),
                                 _ptr(goodness, torch.float32, rows, "goodness"),
                                 _ptr(ws, torch.uint8), ws.numel(), _stream(stream)))
    return h_out, goodness


def ff_layer_step(layer: Layer, hp: HParams, x: torch.Tensor, n_pos: int, n_neg: int,
                  x_normalised: bool = False, h_out: Optional[torch.Tensor] = None,
                  goodness: Optional[torch.Tensor] = None, loss: Optional[torch.Tensor] = None,
                  ws: Optional[torch.Tensor] = None, stream=None):
    R = n_pos + n_neg
    if ws is None:
        ws = workspace(ff_step_workspace_size(max(R, 1), layer.d_in, layer.d_out, hp.dtype),
                       x.device)
        _hold([ws], [stream])
    Lc = layer.c()
    st = LIB.ff_layer_step(ctypes.byref(Lc), ctypes.byref(hp.c()),
                            _ptr(x, torch.float32, R * layer.d_in, "x"), n_pos, n_neg,
                            int(x_normalised), _ptr(h_out, torch.float32, R * layer.d_out, "h_out"),
                            _ptr(goodness, torch.float32, R, "goodness"),
                            _ptr(loss, torch.float32, 1, "loss"), _ptr(ws, torch.uint8),
                            ws.numel(), _stream(stream))
    layer.step = Lc.step
    _check(st)
    return h_out, goodness, loss


NOALLOC_SCRATCH_BYTES = 128 << 20  # FF_NOALLOC_SCRATCH_BYTES of include/ff.h


def ff_layer_step_noalloc(layer: Layer, hp: HParams, x: torch.Tensor, n_pos: int, n_neg: int,
                          x_normalised: bool = False, h_out: Optional[torch.Tensor] = None,
                          goodness: Optional[torch.Tensor] = None,
                          loss: Optional[torch.Tensor] = None, stream=None):
    """ff_layer_step without a workspace: the library's fixed device scratch is
    used (calls overlapping on one GPU race; the caller orders them)."""
    R = n_pos + n_neg
    Lc = layer.c()
    st = LIB.ff_layer_step_noalloc(ctypes.byref(Lc), ctypes.byref(hp.c()),
                                    _ptr(x, torch.float32, R * layer.d_in, "x"), n_pos, n_neg,
                                    int(x_normalised),
                                    _ptr(h_out, torch.float32, R * layer.d_out, "h_out"),
                                    _ptr(goodness, torch.float32, R, "goodness"),
                                    _ptr(loss, torch.float32, 1, "loss"), _stream(stream))
    layer.step = Lc.step
    _check(st)
    return h_out, goodness, loss


def ff_refresh_bf16_shadow(layer: Layer, stream=None):
    Lc = layer.c()
    _check(LIB.ff_refresh_bf16_shadow(ctypes.byref(Lc), _stream(stream)))


def ff_score_workspace_size(layers: Sequence[Layer], n: int, n_classes: int,
                            dtype: int = FF_F32) -> int:
    return LIB.ff_score_workspace_size(_layers_c(layers), len(layers), n, n_classes, dtype)


def ff_score_labels(layers: Sequence[Layer], hp: HParams, x_base: torch.Tensor, n_classes: int,
                    first_scored_layer: int = 0, scores: Optional[torch.Tensor] = None,
                    pred: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                    stream=None):
    n = x_base.shape[0]
    dev = x_base.device
    if pred is None:
        pred = torch.empty(n, dtype=torch.int32, device=dev)
        _hold([pred], [stream])
    if ws is None:
        ws = workspace(ff_score_workspace_size(layers, max(n, 1), n_classes, hp.dtype), dev)
        _hold([ws], [stream])
    arr = _layers_c(layers)
    _check(LIB.ff_score_labels(arr, len(layers), first_scored_layer, ctypes.byref(hp.c()),
                                _ptr(x_base, torch.float32, n * layers[0].d_in, "x_base"), n,
                                n_classes, _ptr(scores, torch.float32, n * n_classes, "scores"),
                                _ptr(pred, torch.int32, n, "pred"), _ptr(ws, torch.uint8),
                                ws.numel(), _stream(stream)))
    return scores, pred


def ff_adaptive_negatives(layers: Sequence[Layer], hp: HParams, x_base: torch.Tensor,
                          labels: torch.Tensor, n_classes: int, first_scored_layer: int = 0,
                          scores: Optional[torch.Tensor] = None,
                          y_neg: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                          stream=None):
    """AdaptiveNEG: y_neg[n] = argmax over c != labels[n] of the goodness scores."""
    n = x_base.shape[0]
    dev = x_base.device
    if y_neg is None:
        y_neg = torch.empty(n, dtype=torch.int32, device=dev)
        _hold([y_neg], [stream])
    if ws is None:
        ws = workspace(ff_score_workspace_size(layers, max(n, 1), n_classes, hp.dtype), dev)
        _hold([ws], [stream])
    arr = _layers_c(layers)
    _check(LIB.ff_adaptive_negatives(
        arr, len(layers), first_scored_layer, ctypes.byref(hp.c()),
        _ptr(x_base, torch.float32, n * layers[0].d_in, "x_base"),
        _ptr(labels, torch.int32, n, "labels"), n, n_classes,
        _ptr(scores, torch.float32, n * n_classes, "scores"), _ptr(y_neg, torch.int32, n, "y_neg"),
        _ptr(ws, torch.uint8), ws.numel(), _stream(stream)))
    return scores, y_neg


def ff_head_workspace_size(layers: Sequence[Layer], first_layer: int, n: int, n_classes: int,
                           dtype: int = FF_F32) -> int:
    return LIB.ff_head_workspace_size(_layers_c(layers), len(layers), first_layer, n, n_classes,
                                      dtype)


def ff_head_step(layers: Sequence[Layer], hp: HParams, head: Head, head_hp: HParams,
                 x_base: torch.Tensor, labels: torch.Tensor, first_layer: int = 1,
                 loss: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                 stream=None):
    """One Adam step of the softmax prediction layer on the batch x_base (labels)."""
    n = x_base.shape[0]
    if ws is None:
        ws = workspace(ff_head_workspace_size(layers, first_layer, max(n, 1), head.n_classes,
                                              hp.dtype), x_base.device)
        _hold([ws], [stream])
    Hc = head.c()
    st = LIB.ff_head_step(_layers_c(layers), len(layers), first_layer, ctypes.byref(hp.c()),
                          ctypes.byref(Hc), ctypes.byref(head_hp.c()),
                          _ptr(x_base, torch.float32, n * layers[0].d_in, "x_base"),
                          _ptr(labels, torch.int32, n, "labels"), n,
                          _ptr(loss, torch.float32, 1, "loss"), _ptr(ws, torch.uint8),
                          ws.numel(), _stream(stream))
    head.step = Hc.step
    _check(st)
    return loss


def ff_head_predict(layers: Sequence[Layer], hp: HParams, head: Head, x_base: torch.Tensor,
                    first_layer: int = 1, logits: Optional[torch.Tensor] = None,
                    pred: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                    stream=None):
    """Softmax prediction: (logits or None, pred)."""
    n = x_base.shape[0]
    dev = x_base.device
    if pred is None:
        pred = torch.empty(n, dtype=torch.int32, device=dev)
        _hold([pred], [stream])
    if ws is None:
        ws = workspace(ff_head_workspace_size(layers, first_layer, max(n, 1), head.n_classes,
                                              hp.dtype), dev)
        _hold([ws], [stream])
    _check(LIB.ff_head_predict(_layers_c(layers), len(layers), first_layer, ctypes.byref(hp.c()),
                               ctypes.byref(head.c()),
                               _ptr(x_base, torch.float32, n * layers[0].d_in, "x_base"), n,
                               _ptr(logits, torch.float32, n * head.n_classes, "logits"),
                               _ptr(pred, torch.int32, n, "pred"), _ptr(ws, torch.uint8),
                               ws.numel(), _stream(stream)))
    return logits, pred


def ff_chapter_train(layers: List[Layer], hp: HParams, x_base: torch.Tensor, y_pos: torch.Tensor,
                     y_neg_chapters: torch.Tensor, n_classes: int, chunk_pairs: int, epochs: int,
                     splits: int, cooldown_start: int, assignment: int = FF_SINGLE_LAYER,
                     streams: Optional[Sequence] = None, n_streams: Optional[int] = None,
                     loss_trace: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None):
    """Chapter-granularity training (Alg. 1 / Alg. 2); y_neg_chapters [splits][n].  With
    streams=None, worker streams are created (one per layer for FF_SINGLE_LAYER, n_streams
    for FF_ALL_LAYERS) and joined back into the current stream before returning."""
    n = x_base.shape[0]
    dev = x_base.device
    nc = (n + chunk_pairs - 1) // chunk_pairs
    ns = len(layers) if assignment == FF_SINGLE_LAYER else (n_streams or len(layers))
    own = streams is None
    cur = torch.cuda.current_stream(dev)
    if own:
        streams = [torch.cuda.Stream(dev) for _ in range(ns)]
        for s in streams:
            s.wait_stream(cur)
    if ws is None:
        ws = workspace(LIB.ff_chapter_workspace_size(_layers_c(layers), len(layers), n,
                                                     chunk_pairs, len(streams), hp.dtype), dev)
        _hold([ws], streams)
    sarr = (c_void_p * len(streams))(*[_stream(s) for s in streams])
    arr = _layers_c(layers)
    st = LIB.ff_chapter_train(arr, len(layers), ctypes.byref(hp.c()),
                              _ptr(x_base, torch.float32, n * layers[0].d_in, "x_base"),
                              _ptr(y_pos, torch.int32, n, "y_pos"),
                              _ptr(y_neg_chapters, torch.int32, splits * n, "y_neg_chapters"), n,
                              n_classes, chunk_pairs, epochs, splits, cooldown_start, assignment,
                              len(streams), sarr,
                              _ptr(loss_trace, torch.float32, len(layers) * epochs * nc,
                                   "loss_trace"), _ptr(ws, torch.uint8), ws.numel())
    for L, Lc in zip(layers, arr):
        L.step = Lc.step
    if own:
        for s in streams:
            cur.wait_stream(s)
    _check(st)


def ff_chapter_train_adaptive(layers: List[Layer], hp: HParams, x_base: torch.Tensor,
                              y_pos: torch.Tensor, n_classes: int, chunk_pairs: int, epochs: int,
                              splits: int, cooldown_start: int,
                              assignment: int = FF_SINGLE_LAYER, first_scored_layer: int = 0,
                              y_neg_chapters: Optional[torch.Tensor] = None,
                              streams: Optional[Sequence] = None, n_streams: Optional[int] = None,
                              loss_trace: Optional[torch.Tensor] = None,
                              ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """AdaptiveNEG chapters: as ff_chapter_train, with each chapter's wrong labels
    computed on the device when the chapter starts; returns them, [splits][n]."""
    n = x_base.shape[0]
    dev = x_base.device
    nc = (n + chunk_pairs - 1) // chunk_pairs
    ns = len(layers) if assignment == FF_SINGLE_LAYER else (n_streams or len(layers))
    own = streams is None
    cur = torch.cuda.current_stream(dev)
    if own:
        streams = [torch.cuda.Stream(dev) for _ in range(ns)]
        for s in streams:
            s.wait_stream(cur)
    if y_neg_chapters is None:
        y_neg_chapters = torch.empty(splits, n, dtype=torch.int32, device=dev)
        _hold([y_neg_chapters], streams)
    if ws is None:
        ws = workspace(LIB.ff_chapter_adaptive_workspace_size(
            _layers_c(layers), len(layers), n, n_classes, chunk_pairs, len(streams), hp.dtype), dev)
        _hold([ws], streams)
    sarr = (c_void_p * len(streams))(*[_stream(s) for s in streams])
    arr = _layers_c(layers)
    st = LIB.ff_chapter_train_adaptive(
        arr, len(layers), ctypes.byref(hp.c()),
        _ptr(x_base, torch.float32, n * layers[0].d_in, "x_base"),
        _ptr(y_pos, torch.int32, n, "y_pos"),
        _ptr(y_neg_chapters, torch.int32, splits * n, "y_neg_chapters"), n, n_classes,
        chunk_pairs, epochs, splits, cooldown_start, assignment, first_scored_layer,
        len(streams), sarr,
        _ptr(loss_trace, torch.float32, len(layers) * epochs * nc, "loss_trace"),
        _ptr(ws, torch.uint8), ws.numel())
    for L, Lc in zip(layers, arr):
        L.step = Lc.step
    if own:
        for s in streams:
            cur.wait_stream(s)
    _check(st)
    return y_neg_chapters


def _heads_c(heads: Sequence[Head]):
    return (ff_head * len(heads))(*[h.c() for h in heads])


def ff_po_layer_step(layer: Layer, head: Head, hp: HParams, head_hp: HParams, x: torch.Tensor,
                     labels: torch.Tensor, x_normalised: bool = False,
                     h_out: Optional[torch.Tensor] = None, loss: Optional[torch.Tensor] = None,
                     ws: Optional[torch.Tensor] = None, stream=None):
    """One performance-optimised step of a layer and its classifier on x (labels)."""
    rows = x.shape[0]
    if ws is None:
        ws = workspace(LIB.ff_po_step_workspace_size(max(rows, 1), layer.d_in, layer.d_out,
                                                     head.n_classes, hp.dtype), x.device)
        _hold([ws], [stream])
    Lc, Hc = layer.c(), head.c()
    st = LIB.ff_po_layer_step(ctypes.byref(Lc), ctypes.byref(Hc), ctypes.byref(hp.c()),
                              ctypes.byref(head_hp.c()),
                              _ptr(x, torch.float32, rows * layer.d_in, "x"),
                              _ptr(labels, torch.int32, rows, "labels"), rows, int(x_normalised),
                              _ptr(h_out, torch.float32, rows * layer.d_out, "h_out"),
                              _ptr(loss, torch.float32, 1, "loss"), _ptr(ws, torch.uint8),
                              ws.numel(), _stream(stream))
    layer.step, head.step = Lc.step, Hc.step
    _check(st)


def ff_po_epoch(layers: List[Layer], heads: List[Head], hp: HParams, head_hp: HParams,
                x_base: torch.Tensor, labels: torch.Tensor, n_classes: int, chunk: int,
                epochs: int = 1, schedule: int = FF_PIPELINED, streams: Optional[Sequence] = None,
                loss_trace: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None):
    """Performance-optimised training epoch(s); streams as for ff_pipeline_epoch."""
    n = x_base.shape[0]
    dev = x_base.device
    nc = (n + chunk - 1) // chunk
    own = streams is None
    cur = torch.cuda.current_stream(dev)
    if own:
        streams = [cur] + [torch.cuda.Stream(dev) for _ in range(len(layers) - 1)]
        for s in streams[1:]:
            s.wait_stream(cur)
    if ws is None:
        ws = workspace(LIB.ff_po_epoch_workspace_size(_layers_c(layers), len(layers), n,
                                                      n_classes, chunk, schedule, hp.dtype), dev)
        _hold([ws], streams)
    sarr = (c_void_p * len(layers))(*[_stream(s) for s in streams])
    arr, harr = _layers_c(layers), _heads_c(heads)
    st = LIB.ff_po_epoch(arr, harr, len(layers), ctypes.byref(hp.c()), ctypes.byref(head_hp.c()),
                         _ptr(x_base, torch.float32, n * layers[0].d_in, "x_base"),
                         _ptr(labels, torch.int32, n, "labels"), n, n_classes, chunk, epochs,
                         schedule, sarr,
                         _ptr(loss_trace, torch.float32, len(layers) * nc * epochs, "loss_trace"),
                         _ptr(ws, torch.uint8), ws.numel())
    for L, Lc in zip(layers, arr):
        L.step = Lc.step
    for h, hc in zip(heads, harr):
        h.step = hc.step
    if own:
        for s in streams[1:]:
            cur.wait_stream(s)
    _check(st)


def ff_po_predict(layers: Sequence[Layer], heads: Sequence[Head], hp: HParams,
                  x_base: torch.Tensor, all_layers: bool = True,
                  logits: Optional[torch.Tensor] = None, pred: Optional[torch.Tensor] = None,
                  ws: Optional[torch.Tensor] = None, stream=None):
    """Prediction of a performance-optimised network: (logits or None, pred)."""
    n = x_base.shape[0]
    dev = x_base.device
    C = heads[0].n_classes
    if pred is None:
        pred = torch.empty(n, dtype=torch.int32, device=dev)
        _hold([pred], [stream])
    if ws is None:
        ws = workspace(LIB.ff_po_predict_workspace_size(_layers_c(layers), len(layers),
                                                        max(n, 1), C, hp.dtype), dev)
        _hold([ws], [stream])
    _check(LIB.ff_po_predict(_layers_c(layers), _heads_c(heads), len(layers),
                             ctypes.byref(hp.c()),
                             _ptr(x_base, torch.float32, n * layers[0].d_in, "x_base"), n,
                             int(all_layers), _ptr(logits, torch.float32, n * C, "logits"),
                             _ptr(pred, torch.int32, n, "pred"), _ptr(ws, torch.uint8),
                             ws.numel(), _stream(stream)))
    return logits, pred


def ff_pipeline_workspace_size(layers: Sequence[Layer], n: int, chunk_pairs: int, schedule: int,
                               dtype: int = FF_F32) -> int:
    return LIB.ff_pipeline_workspace_size(_layers_c(layers), len(layers), n, chunk_pairs,
                                           schedule, dtype)


def ff_pipeline_epoch(layers: List[Layer], hp: HParams, x_base: torch.Tensor, y_pos: torch.Tensor,
                      y_neg: torch.Tensor, n_classes: int, chunk_pairs: int, epochs: int = 1,
                      schedule: int = FF_SEQUENTIAL, streams: Optional[Sequence] = None,
                      loss_trace: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None):
    """Enqueue the epoch(s).  With streams=None, per-layer streams are created and
    joined back into the current stream before returning (still asynchronous to
    the host)."""
    n = x_base.shape[0]
    dev = x_base.device
    nc = (n + chunk_pairs - 1) // chunk_pairs
    own = streams is None
    cur = torch.cuda.current_stream(dev)
    if own:
        streams = [cur] + [torch.cuda.Stream(dev) for _ in range(len(layers) - 1)]
        for s in streams[1:]:
            s.wait_stream(cur)
    if ws is None:
        ws = workspace(ff_pipeline_workspace_size(layers, n, chunk_pairs, schedule, hp.dtype), dev)
        _hold([ws], streams)
    sarr = (c_void_p * len(layers))(*[_stream(s) for s in streams])
    arr = _layers_c(layers)
    st = LIB.ff_pipeline_epoch(arr, len(layers), ctypes.byref(hp.c()),
                                _ptr(x_base, torch.float32, n * layers[0].d_in, "x_base"),
                                _ptr(y_pos, torch.int32, n, "y_pos"),
                                _ptr(y_neg, torch.int32, n, "y_neg"), n, n_classes, chunk_pairs,
                                epochs, schedule, sarr,
                                _ptr(loss_trace, torch.float32, len(layers) * nc * epochs,
                                     "loss_trace"), _ptr(ws, torch.uint8), ws.numel())
    for L, Lc in zip(layers, arr):
        L.step = Lc.step
    if own:
        for s in streams[1:]:
            cur.wait_stream(s)
    _check(st)
    return loss_trace


def ff_fail_next_launch(kind: Optional[str]):
    """Test aid: the next launch of kernel kind `kind` (a KERNEL_KINDS name) fails
    without enqueuing anything; None disarms."""
    _check(LIB.ff_fail_next_launch(-1 if kind is None else KERNEL_KINDS.index(kind)))


_profile_capacity = [0]  # max_launches of the active profile


def ff_profile_start(max_launches: int = 65536, kinds=None):
    """kinds: names from KERNEL_KINDS to time (None: every kind)."""
    mask = 0 if kinds is None else sum(1 << KERNEL_KINDS.index(k) for k in kinds)
    _check(LIB.ff_profile_start(max_launches, mask))
    _profile_capacity[0] = max_launches


def ff_profile_stop(launches: bool = False):
    """Per kernel kind: launches, total_ms, flops, bytes (event-timed on each launch's stream).
    With launches=True also the list of timed launches in enqueue order, each a dict of
    kind (name), m, n, k, aux, ms, flops, bytes: returns (stats, launches)."""
    arr = (ff_kernel_stats * len(KERNEL_KINDS))()
    if not launches:
        _check(LIB.ff_profile_stop(arr))
    else:
        cap = max(_profile_capacity[0], 1)  # no more launches are timed than that
        recs = (ff_launch_record * cap)()
        n = c_int32(0)
        _check(LIB.ff_profile_stop_launches(arr, recs, cap, ctypes.byref(n)))
    stats = {k: dict(launches=a.launches, total_ms=a.total_ms, flops=a.flops, bytes=a.bytes)
             for k, a in zip(KERNEL_KINDS, arr)}
    if not launches:
        return stats
    out = [dict(kind=KERNEL_KINDS[r.kind], m=r.m, n=r.n, k=r.k, aux=r.aux, ms=r.ms,
                flops=r.flops, bytes=r.bytes) for r in recs[:n.value]]
    return stats, out
