"""ctypes binding of libpointid (include/pointid.h), argument marshalling only.

Each function carries the name of the C entry point it calls.  Tensors are
torch tensors on the handle's device; the binding checks dtype, shape and
contiguity, passes raw device pointers and the current HIP stream, and raises
``PointIdError`` on a non-OK status.  Every step of the computation runs in the
library's HIP kernels; if the library is not built this module fails to import.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
# POINTID_LIB selects another build of the same library (the sanitized host
# builds, libpointid_asan.so / libpointid_tsan.so, for checking runs)
LIB_PATH = os.environ.get("POINTID_LIB") or os.path.join(_PKG, "libpointid.so")

POINTID_OK = 0
POINTID_EINVAL = -1
POINTID_ENOMEM = -2
POINTID_EHIP = -3
POINTID_ENODEV = -4
POINTID_EUNSUPPORTED = -5
POINTID_EIO = -6
POINTID_FP32 = 0
POINTID_BF16 = 1
POINTID_FP16 = 2
POINTID_FP8 = 3
MAX_PLANES = 64

_STATUS = {0: "OK", -1: "EINVAL", -2: "ENOMEM", -3: "EHIP", -4: "ENODEV", -5: "EUNSUPPORTED",
           -6: "EIO"}
_WEIGHT_FIELDS = ("conv_w", "conv_b", "fc1_w", "fc1_b", "fc2_w", "fc2_b",
                  "cls_w", "cls_b", "mic_w", "mic_b")
_WEIGHT_SIZES = {"conv_w": 48 * 25, "conv_b": 48, "fc1_w": 92928 * 128, "fc1_b": 128,
                 "fc2_w": 128 * 32, "fc2_b": 32, "cls_w": 32 * 3, "cls_b": 3,
                 "mic_w": 32, "mic_b": 1}


class PointIdError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_STATUS.get(status, status)}: {message}")
        self.status = status


class _Weights(ctypes.Structure):
    _fields_ = [(name, ctypes.POINTER(ctypes.c_float)) for name in _WEIGHT_FIELDS]


class _Plane(ctypes.Structure):
    _fields_ = [("image", ctypes.c_void_p), ("n_wires", ctypes.c_int32),
                ("n_ticks", ctypes.c_int32)]


class _Request(ctypes.Structure):
    _fields_ = [("hits", ctypes.c_void_p), ("n_hits", ctypes.c_int64),
                ("plane", ctypes.c_int32), ("scores", ctypes.c_void_p)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built; run `python -m paper_2009_04509_amd.build` "
            "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, cint = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_int
    sig = {
        "pointid_create": (cint, [ctypes.POINTER(_Weights), cint, cint, ctypes.POINTER(vp)]),
        "pointid_destroy": (cint, [vp]),
        "pointid_trim": (cint, [vp, ctypes.c_uint64, ctypes.POINTER(ctypes.c_uint64)]),
        "pointid_precision": (cint, [vp]),
        "pointid_classify": (cint, [vp, vp, i32, i32, vp, i64, vp, vp]),
        "pointid_classify_planes": (cint, [vp, ctypes.POINTER(_Plane), i32, vp, i64, vp, vp]),
        "pointid_classify_patches": (cint, [vp, vp, i64, vp, vp]),
        "pointid_classify_planes_noalloc": (cint, [vp, ctypes.POINTER(_Plane), i32, vp, i64, vp,
                                                   vp]),
        "pointid_classify_planes_ds": (cint, [vp, ctypes.POINTER(_Plane), i32, i32, vp, i64, vp,
                                              vp]),
        "pointid_downsample": (cint, [vp, i32, i32, i32, vp, vp]),
        "pointid_classify_requests": (cint, [vp, ctypes.POINTER(_Plane), i32,
                                             ctypes.POINTER(_Request), i32, vp]),
        "pointid_batcher_create": (cint, [vp, ctypes.POINTER(_Plane), i32, i32, i32,
                                          ctypes.POINTER(vp)]),
        "pointid_batcher_destroy": (cint, [vp]),
        "pointid_batcher_submit": (cint, [vp, ctypes.POINTER(_Request), vp,
                                            ctypes.POINTER(ctypes.c_uint64)]),
        "pointid_batcher_wait": (cint, [vp, ctypes.c_uint64]),
        "pointid_gather": (cint, [vp, i32, i32, vp, i64, vp, cint, vp]),
        "pointid_gather_planes": (cint, [ctypes.POINTER(_Plane), i32, vp, i64, vp, cint, vp]),
        "pointid_find_hits": (cint, [vp, ctypes.POINTER(_Plane), i32, ctypes.c_float, vp, i64,
                                     vp, vp]),
        "pointid_server_start": (cint, [vp, ctypes.POINTER(_Plane), i32, ctypes.c_char_p, i32, i32,
                                        ctypes.POINTER(vp)]),
        "pointid_server_stop": (cint, [vp]),
        "pointid_client_connect": (cint, [ctypes.c_char_p, ctypes.POINTER(vp)]),
        "pointid_client_classify": (cint, [vp, i32, vp, i64, vp, ctypes.POINTER(i64)]),
        "pointid_client_classify_patches": (cint, [vp, vp, i64, vp, ctypes.POINTER(i64)]),
        "pointid_client_close": (cint, [vp]),
        "pointid_timing_enable": (cint, [cint]),
        "pointid_timing_reset": (cint, []),
        "pointid_timing_query": (cint, [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_int64)]),
        "pointid_last_error": (ctypes.c_char_p, []),
        "pointid_version": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()
EXPORTED = ("pointid_create", "pointid_destroy", "pointid_precision", "pointid_trim",
            "pointid_classify",
            "pointid_classify_planes", "pointid_classify_planes_noalloc", "pointid_classify_requests",
            "pointid_classify_patches",
            "pointid_batcher_create", "pointid_batcher_destroy", "pointid_batcher_submit",
            "pointid_batcher_wait",
            "pointid_gather",
            "pointid_gather_planes", "pointid_find_hits", "pointid_classify_planes_ds",
            "pointid_downsample", "pointid_server_start", "pointid_server_stop",
            "pointid_client_connect", "pointid_client_classify", "pointid_client_classify_patches",
            "pointid_client_close", "pointid_timing_enable", "pointid_timing_reset",
            "pointid_timing_query", "pointid_last_error", "pointid_version")


def _check(status: int):
    if status != POINTID_OK:
        raise PointIdError(status, lib.pointid_last_error().decode())
    return status


def pointid_last_error() -> str:
    return lib.pointid_last_error().decode()


def pointid_version() -> str:
    return lib.pointid_version().decode()


def pointid_timing_enable(on: bool = True):
    _check(lib.pointid_timing_enable(1 if on else 0))


def pointid_timing_reset():
    _check(lib.pointid_timing_reset())


def pointid_timing_query(kernel: str):
    """(total_ms, launches) of `kernel` since the last reset."""
    ms = ctypes.c_double()
    n = ctypes.c_int64()
    _check(lib.pointid_timing_query(kernel.encode(), ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def _precision(p) -> int:
    if isinstance(p, str):
        return {"fp32": POINTID_FP32, "bf16": POINTID_BF16, "fp16": POINTID_FP16,
                "fp8": POINTID_FP8}[p]
    return int(p)


def _stream_ptr(stream, device=None):
    if stream is None:
        stream = torch.cuda.current_stream(device)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _need(t, dtype, name, device=None, tail_shape=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if device is not None and t.device.index != device:
        raise ValueError(f"{name} is on cuda:{t.device.index}, handle is on cuda:{device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if tail_shape is not None and tuple(t.shape[1:]) != tuple(tail_shape):
        raise ValueError(f"{name} must have shape [n, {', '.join(map(str, tail_shape))}]")


class Handle:
    """A created classifier; frees itself on garbage collection."""

    def __init__(self, raw: ctypes.c_void_p, device: int, precision: int):
        self._raw = raw
        self.device = device
        self.precision = precision

    @property
    def raw(self):
        if not self._raw:
            raise ValueError("handle was destroyed")
        return self._raw

    def close(self):
        if self._raw:
            _check(lib.pointid_destroy(self._raw))
            self._raw = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def pointid_create(weights: dict, precision="fp32", device: int = 0) -> Handle:
    """Upload ``weights`` (dict of float32 arrays, layouts of include/pointid.h)."""
    arrays = {}
    for name in _WEIGHT_FIELDS:
        a = np.ascontiguousarray(np.asarray(weights[name], dtype=np.float32))
        if a.size != _WEIGHT_SIZES[name]:
            raise ValueError(f"{name} has {a.size} values, expected {_WEIGHT_SIZES[name]}")
        arrays[name] = a
    w = _Weights(**{n: arrays[n].ctypes.data_as(ctypes.POINTER(ctypes.c_float))
                    for n in _WEIGHT_FIELDS})
    raw = ctypes.c_void_p()
    prec = _precision(precision)
    _check(lib.pointid_create(ctypes.byref(w), prec, int(device), ctypes.byref(raw)))
    return Handle(raw, int(device), prec)


def pointid_destroy(h: Handle):
    h.close()


def pointid_trim(h: Handle, keep_bytes: int = 0) -> int:
    """Free the handle's idle cached scratch buffers down to keep_bytes;
    returns the bytes still cached."""
    cached = ctypes.c_uint64()
    _check(lib.pointid_trim(h.raw, ctypes.c_uint64(int(keep_bytes)), ctypes.byref(cached)))
    return int(cached.value)


def pointid_classify(h: Handle, image: torch.Tensor, hits: torch.Tensor,
                     scores: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Scores [n][4] for int32 hits [n][2] = (wire, tick) on fp32 image [W][T]."""
    _need(image, torch.float32, "image", h.device)
    if image.dim() != 2:
        raise ValueError("image must be [n_wires][n_ticks]")
    _need(hits, torch.int32, "hits", h.device, (2,))
    n = hits.shape[0]
    if scores is None:
        scores = torch.empty((n, 4), dtype=torch.float32, device=image.device)
    _need(scores, torch.float32, "scores", h.device, (4,))
    _check(lib.pointid_classify(h.raw, _ptr(image), image.shape[0], image.shape[1], _ptr(hits),
                                n, _ptr(scores), _stream_ptr(stream, image.device)))
    return scores


def _plane_array(images):
    if len(images) < 1 or len(images) > MAX_PLANES:
        raise ValueError("between 1 and 64 planes")
    arr = (_Plane * len(images))()
    for i, im in enumerate(images):
        _need(im, torch.float32, f"images[{i}]")
        if im.dim() != 2:
            raise ValueError("each image must be [n_wires][n_ticks]")
        arr[i] = _Plane(im.data_ptr(), im.shape[0], im.shape[1])
    return arr


def pointid_classify_planes(h: Handle, images, hits: torch.Tensor,
                            scores: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Scores for int32 hits [n][3] = (plane, wire, tick) over a list of plane images."""
    arr = _plane_array(images)
    _need(hits, torch.int32, "hits", h.device, (3,))
    n = hits.shape[0]
    if scores is None:
        scores = torch.empty((n, 4), dtype=torch.float32, device=hits.device)
    _need(scores, torch.float32, "scores", h.device, (4,))
    _check(lib.pointid_classify_planes(h.raw, arr, len(images), _ptr(hits), n, _ptr(scores),
                                       _stream_ptr(stream, hits.device)))
    return scores


def pointid_classify_planes_noalloc(h: Handle, images, hits: torch.Tensor,
                                    scores: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """pointid_classify_planes with its scratch in the library's fixed device
    array (at most 8192 hits; calls on one GPU must not overlap)."""
    _need(hits, torch.int32, "hits", h.device, (3,))
    n = hits.shape[0]
    if scores is None:
        scores = torch.empty((n, 4), dtype=torch.float32, device=hits.device)
    _need(scores, torch.float32, "scores", h.device, (4,))
    arr = _plane_array(images)
    _check(lib.pointid_classify_planes_noalloc(h.raw, arr, len(images), _ptr(hits), n, _ptr(scores),
                                               _stream_ptr(stream, hits.device)))
    return scores


def pointid_classify_planes_ds(h: Handle, images, hits: torch.Tensor, ticks_per_column: int,
                               scores: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Scores with patches of ``ticks_per_column`` ticks per column; hits are
    (plane, wire, tick) in unbinned ticks over the unbinned plane images."""
    arr = _plane_array(images)
    _need(hits, torch.int32, "hits", h.device, (3,))
    n = hits.shape[0]
    if scores is None:
        scores = torch.empty((n, 4), dtype=torch.float32, device=hits.device)
    _need(scores, torch.float32, "scores", h.device, (4,))
    _check(lib.pointid_classify_planes_ds(h.raw, arr, len(images), int(ticks_per_column),
                                          _ptr(hits), n, _ptr(scores),
                                          _stream_ptr(stream, hits.device)))
    return scores


def pointid_downsample(image: torch.Tensor, ticks_per_column: int,
                       out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """fp32 image [W][T] binned into [W][ceil(T / D)] columns of D ticks."""
    _need(image, torch.float32, "image")
    if image.dim() != 2:
        raise ValueError("image must be [n_wires][n_ticks]")
    D = int(ticks_per_column)
    W, T = image.shape
    J = -(-T // D) if D >= 1 else 0
    if out is None:
        out = torch.empty((W, max(J, 1)), dtype=torch.float32, device=image.device)
    _need(out, torch.float32, "out")
    if tuple(out.shape) != (W, J):
        raise ValueError(f"out must be [{W}, {J}]")
    _check(lib.pointid_downsample(_ptr(image), W, T, D, _ptr(out),
                                  _stream_ptr(stream, image.device)))
    return out


def pointid_classify_requests(h: Handle, images, requests, stream=None):
    """Classify several requests in one batched call.

    ``requests`` is a list of ``(plane, hits, scores)``: ``plane`` an index into
    ``images`` with int32 hits [n][2] = (wire, tick), or -1 with hits [n][3] =
    (plane, wire, tick); ``scores`` a float32 [n][4] output, or None to allocate
    one.  Returns the list of score tensors."""
    arr = _plane_array(images)
    reqs = (_Request * max(len(requests), 1))()
    outs = []
    dev = None
    for i, (plane, hits, scores) in enumerate(requests):
        plane = int(plane)
        _need(hits, torch.int32, f"requests[{i}].hits", h.device, (2,) if plane >= 0 else (3,))
        n = hits.shape[0]
        if scores is None:
            scores = torch.empty((n, 4), dtype=torch.float32, device=hits.device)
        _need(scores, torch.float32, f"requests[{i}].scores", h.device, (4,))
        reqs[i] = _Request(hits.data_ptr(), n, plane, scores.data_ptr())
        outs.append(scores)
        dev = hits.device
    _check(lib.pointid_classify_requests(h.raw, arr, len(images), reqs, len(requests),
                                         _stream_ptr(stream, dev)))
    return outs


class Batcher:
    """Dynamic batcher over a handle and resident plane images (see
    pointid_batcher_create).  submit() returns a ticket; wait(ticket) blocks
    until that request's scores are written.  The hits and scores tensors of a
    request are kept alive here until its wait returns."""

    def __init__(self, h: Handle, images, max_requests: int = 64, max_delay_us: int = 200):
        self._arr = _plane_array(images)
        self._images = list(images)
        self._h = h
        raw = ctypes.c_void_p()
        _check(lib.pointid_batcher_create(h.raw, self._arr, len(images), int(max_requests),
                                          int(max_delay_us), ctypes.byref(raw)))
        self.raw = raw
        self._live = {}

    def submit(self, plane: int, hits: torch.Tensor, scores: torch.Tensor | None = None,
               stream=None) -> int:
        """Queue a request; the batch that classifies it starts after the work
        enqueued on `stream` (the current stream by default) before this call,
        so `hits` may still be in production there and `scores` may be a fresh
        allocation of that stream."""
        plane = int(plane)
        _need(hits, torch.int32, "hits", self._h.device, (2,) if plane >= 0 else (3,))
        n = hits.shape[0]
        if scores is None:
            scores = torch.empty((n, 4), dtype=torch.float32, device=hits.device)
        _need(scores, torch.float32, "scores", self._h.device, (4,))
        req = _Request(hits.data_ptr(), n, plane, scores.data_ptr())
        ticket = ctypes.c_uint64()
        _check(lib.pointid_batcher_submit(self.raw, ctypes.byref(req),
                                          _stream_ptr(stream, hits.device), ctypes.byref(ticket)))
        self._live[ticket.value] = (hits, scores)
        return ticket.value

    def wait(self, ticket: int) -> torch.Tensor:
        """Blocks until the request is classified; returns its scores tensor."""
        try:
            _check(lib.pointid_batcher_wait(self.raw, ctypes.c_uint64(ticket)))
        finally:
            pair = self._live.pop(ticket, None)
        return pair[1] if pair else None

    def close(self):
        if self.raw:
            _check(lib.pointid_batcher_destroy(self.raw))
            self.raw = None
            self._live.clear()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def pointid_classify_patches(h: Handle, patches: torch.Tensor,
                             scores: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Scores for fp32 patches [n][48][48]."""
    _need(patches, torch.float32, "patches", h.device, (48, 48))
    n = patches.shape[0]
    if scores is None:
        scores = torch.empty((n, 4), dtype=torch.float32, device=patches.device)
    _need(scores, torch.float32, "scores", h.device, (4,))
    _check(lib.pointid_classify_patches(h.raw, _ptr(patches), n, _ptr(scores),
                                        _stream_ptr(stream, patches.device)))
    return scores


def pointid_gather(image: torch.Tensor, hits: torch.Tensor, out_dtype="fp32",
                   out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Patches [n][48][48]: float32, or bf16 / fp16 bit patterns as int16."""
    _need(image, torch.float32, "image")
    _need(hits, torch.int32, "hits", None, (2,))
    code = _precision(out_dtype)
    n = hits.shape[0]
    tdt = torch.float32 if code == POINTID_FP32 else torch.int16
    if out is None:
        out = torch.empty((n, 48, 48), dtype=tdt, device=image.device)
    _check(lib.pointid_gather(_ptr(image), image.shape[0], image.shape[1], _ptr(hits), n,
                              _ptr(out), code, _stream_ptr(stream, image.device)))
    return out


def pointid_gather_planes(images, hits: torch.Tensor, out_dtype="fp32",
                          out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    arr = _plane_array(images)
    _need(hits, torch.int32, "hits", None, (3,))
    code = _precision(out_dtype)
    n = hits.shape[0]
    tdt = torch.float32 if code == POINTID_FP32 else torch.int16
    if out is None:
        out = torch.empty((n, 48, 48), dtype=tdt, device=hits.device)
    _check(lib.pointid_gather_planes(arr, len(images), _ptr(hits), n, _ptr(out), code,
                                     _stream_ptr(stream, hits.device)))
    return out


def pointid_find_hits(h: Handle, images, threshold: float, capacity: int | None = None,
                      hits_out: torch.Tensor | None = None, n_found: torch.Tensor | None = None,
                      stream=None):
    """Hits (plane, wire, tick) of fp32 plane images, found on the device.

    Returns ``(hits_out, n_found)``: int32 [capacity][3], of which the first
    min(n_found, capacity) rows are written, and a device int64 [1] holding the
    number of hits found (read it after the stream has passed the call).
    ``capacity`` defaults to ``hits_out``'s length, else to 65,536.
    """
    arr = _plane_array(images)
    dev = images[0].device
    if hits_out is None:
        cap = 65536 if capacity is None else int(capacity)
        hits_out = torch.empty((cap, 3), dtype=torch.int32, device=dev)
    _need(hits_out, torch.int32, "hits_out", h.device, (3,))
    cap = hits_out.shape[0] if capacity is None else int(capacity)
    if cap > hits_out.shape[0]:
        raise ValueError("capacity exceeds hits_out")
    if n_found is None:
        n_found = torch.empty((1,), dtype=torch.int64, device=dev)
    _need(n_found, torch.int64, "n_found", h.device)
    _check(lib.pointid_find_hits(h.raw, arr, len(images), float(threshold),
                                 _ptr(hits_out) if cap > 0 else ctypes.c_void_p(0), cap,
                                 _ptr(n_found), _stream_ptr(stream, dev)))
    return hits_out, n_found


class Server:
    """pointid_server_start / pointid_server_stop: a local request server over
    resident device planes (the handle and the planes must outlive it)."""

    def __init__(self, h: Handle, images, socket_path: str, max_requests: int = 0,
                 max_delay_us: int = 200):
        self._images = list(images)
        arr = _plane_array(self._images) if self._images else None
        raw = ctypes.c_void_p()
        _check(lib.pointid_server_start(h.raw, arr, len(self._images), socket_path.encode(),
                                        int(max_requests), int(max_delay_us), ctypes.byref(raw)))
        self._raw = raw
        self._h = h
        self.path = socket_path

    def close(self):
        if self._raw:
            _check(lib.pointid_server_stop(self._raw))
            self._raw = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Client:
    """pointid_client_*: host arrays in, host scores out (numpy; no GPU)."""

    def __init__(self, socket_path: str):
        raw = ctypes.c_void_p()
        _check(lib.pointid_client_connect(socket_path.encode(), ctypes.byref(raw)))
        self._raw = raw
        self.server_ns = 0

    def classify(self, hits: np.ndarray, plane: int = -1) -> np.ndarray:
        """Scores [n][4] of int32 hits [n][2] on `plane`, or [n][3] when plane < 0."""
        hits = np.ascontiguousarray(hits, dtype=np.int32)
        width = 2 if plane >= 0 else 3
        if hits.ndim != 2 or hits.shape[1] != width:
            raise ValueError(f"hits must be [n][{width}]")
        out = np.empty((hits.shape[0], 4), np.float32)
        ns = ctypes.c_int64()
        _check(lib.pointid_client_classify(self._raw, int(plane), hits.ctypes.data_as(ctypes.c_void_p),
                                           hits.shape[0], out.ctypes.data_as(ctypes.c_void_p),
                                           ctypes.byref(ns)))
        self.server_ns = ns.value
        return out

    def classify_patches(self, patches: np.ndarray) -> np.ndarray:
        patches = np.ascontiguousarray(patches, dtype=np.float32)
        if patches.ndim != 3 or patches.shape[1:] != (48, 48):
            raise ValueError("patches must be [n][48][48]")
        out = np.empty((patches.shape[0], 4), np.float32)
        ns = ctypes.c_int64()
        _check(lib.pointid_client_classify_patches(self._raw,
                                                   patches.ctypes.data_as(ctypes.c_void_p),
                                                   patches.shape[0],
                                                   out.ctypes.data_as(ctypes.c_void_p),
                                                   ctypes.byref(ns)))
        self.server_ns = ns.value
        return out

    def close(self):
        if self._raw:
            _check(lib.pointid_client_close(self._raw))
            self._raw = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
