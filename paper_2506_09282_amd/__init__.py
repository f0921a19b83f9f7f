"""Python binding of the MI355X batched HDC inference library (``libhd.so``).

Argument marshalling only: every step of inference runs in the library's HIP
kernels, called through the C ABI declared in ``include/hd.h``. PyTorch is
used for device memory and streams. There is no fallback: if the compiled
library is missing, importing a function raises.

Operation (ScalableHD, Alg. 1): H = HardSign(X B) (Eq. 7, Eq. 1),
S = H C^T (Eq. 8), labels = argmax_k S (Eq. 9). Single-pass training
(Sec. II-C): C = HardSign of the per-class sums of HardSign(X B).
"""
from __future__ import annotations

import ctypes
import os
import threading

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libhd.so")

HD_OK, HD_ERR_ARG, HD_ERR_UNSUPPORTED, HD_ERR_WORKSPACE, HD_ERR_HIP = range(5)
HD_F32, HD_BF16, HD_I8 = 0, 1, 2
HD_DETERMINISTIC = 0x100  # flag OR-ed into act: bit-identical results from call to call
ACTS = {"hardsign": 0, "identity": 1}

SYMBOLS = (
    "hd_status_str",
    "hd_encode",
    "hd_similarity",
    "hd_infer_workspace_bytes",
    "hd_infer",
    "hd_model_packed_bytes",
    "hd_pack_model",
    "hd_infer_packed_workspace_bytes",
    "hd_infer_packed",
    "hd_infer_kernel",
    "hd_noalloc_scratch_bytes",
    "hd_infer_packed_noalloc",
    "hd_infer_stream_workspace_bytes",
    "hd_infer_stream",
    "hd_bundle_classes",
    "hd_class_hardsign",
    "hd_bundle_classes_packed",
    "hd_bundle_kernel",
)

_lib = None
_lock = threading.Lock()


class HDError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = lib().hd_status_str(status).decode() if _lib is not None else str(status)
        super().__init__(f"{where}: {msg}")


def lib():
    """The loaded ``libhd.so`` with argument types set (raises if absent)."""
    global _lib
    if _lib is not None:
        return _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(LIB_PATH):
            raise ImportError(
                f"{LIB_PATH} is not built; run paper_2506_09282_amd/build.py "
                "(or __graft_entry__.build()) first")
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_size_t
        L.hd_status_str.argtypes = [i32]
        L.hd_status_str.restype = ctypes.c_char_p
        L.hd_encode.argtypes = [vp, vp, vp, i64, i64, i64, i32, i32, vp]
        L.hd_encode.restype = i32
        L.hd_similarity.argtypes = [vp, vp, vp, vp, i64, i64, i64, i32, vp]
        L.hd_similarity.restype = i32
        L.hd_infer_workspace_bytes.argtypes = [i64, i64, i64, i64, i32]
        L.hd_infer_workspace_bytes.restype = sz
        L.hd_infer.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64, i32, i32, vp, sz, vp]
        L.hd_infer.restype = i32
        L.hd_model_packed_bytes.argtypes = [i64, i64, i64, i32]
        L.hd_model_packed_bytes.restype = sz
        L.hd_pack_model.argtypes = [vp, vp, i64, i64, i64, i32, vp, sz, vp]
        L.hd_pack_model.restype = i32
        L.hd_infer_packed_workspace_bytes.argtypes = [i64, i64, i64, i64, i32]
        L.hd_infer_packed_workspace_bytes.restype = sz
        L.hd_infer_packed.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, i32, i32, vp, sz, vp]
        L.hd_infer_packed.restype = i32
        L.hd_infer_kernel.argtypes = [i64, i64, i64, i64, i32, i32]
        L.hd_infer_kernel.restype = ctypes.c_char_p
        L.hd_noalloc_scratch_bytes.argtypes = []
        L.hd_noalloc_scratch_bytes.restype = sz
        L.hd_infer_packed_noalloc.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, i32, i32, vp]
        L.hd_infer_packed_noalloc.restype = i32
        L.hd_infer_stream_workspace_bytes.argtypes = [i64, i64, i64, i64, i64, i32]
        L.hd_infer_stream_workspace_bytes.restype = sz
        L.hd_infer_stream.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, i32, i32,
                                      vp, sz, vp]
        L.hd_infer_stream.restype = i32
        L.hd_bundle_classes.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, i32, vp]
        L.hd_bundle_classes.restype = i32
        L.hd_class_hardsign.argtypes = [vp, vp, i64, i64, vp]
        L.hd_class_hardsign.restype = i32
        L.hd_bundle_classes_packed.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, i32, vp]
        L.hd_bundle_classes_packed.restype = i32
        L.hd_bundle_kernel.argtypes = [i64, i64, i64, i64, i32, i32]
        L.hd_bundle_kernel.restype = ctypes.c_char_p
        _lib = L
        return L


def _torch():
    import torch
    return torch


def _dt_of(dtype) -> int:
    torch = _torch()
    if dtype == torch.float32:
        return HD_F32
    if dtype == torch.bfloat16:
        return HD_BF16
    if dtype == torch.int8:
        return HD_I8
    raise TypeError(f"unsupported dtype {dtype}; use float32, bfloat16 or int8")


def _dt(t) -> int:
    return _dt_of(t.dtype)


def _check_dev(*ts):
    for t in ts:
        if not t.is_cuda:
            raise ValueError("tensors must be on the GPU")
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous (row-major)")


def _stream_ptr(device) -> int:
    torch = _torch()
    return torch.cuda.current_stream(device).cuda_stream


def _raise(st: int, where: str):
    if st != HD_OK:
        raise HDError(st, where)


# Workspaces are cached per (device, stream, size); the library leaves the
# parts that must start at zero zeroed after every call of the same shape,
# so a cached buffer is only zeroed when first allocated for that key.
_ws_cache: dict = {}


def _workspace(device, nbytes: int, key):
    torch = _torch()
    if nbytes == 0:
        return None
    k = (device.index, _stream_ptr(device), key, nbytes)
    ws = _ws_cache.get(k)
    if ws is None:
        ws = torch.zeros(nbytes, dtype=torch.uint8, device=device)
        _ws_cache[k] = ws
    return ws


def encode(X, B, act: str = "hardsign"):
    """Stage I alone: H[N, D] float32 = act(X B)."""
    torch = _torch()
    _check_dev(X, B)
    if X.dtype != B.dtype:
        raise TypeError("X and B must have the same dtype")
    N, F = X.shape
    F2, D = B.shape
    if F2 != F:
        raise ValueError("shape mismatch")
    H = torch.empty((N, D), dtype=torch.float32, device=X.device)
    st = lib().hd_encode(X.data_ptr(), B.data_ptr(), H.data_ptr(), N, F, D, _dt(X), ACTS[act],
                         _stream_ptr(X.device))
    _raise(st, "hd_encode")
    return H


def similarity(H, C, return_scores: bool = False):
    """Stage II alone: labels[N] int32 (and scores[N, K] float32)."""
    torch = _torch()
    _check_dev(H, C)
    if H.dtype != torch.float32:
        raise TypeError("H must be float32")
    N, D = H.shape
    K, D2 = C.shape
    if D2 != D:
        raise ValueError("shape mismatch")
    labels = torch.empty(N, dtype=torch.int32, device=H.device)
    scores = torch.empty((N, K), dtype=torch.float32, device=H.device) if return_scores else None
    st = lib().hd_similarity(H.data_ptr(), C.data_ptr(), labels.data_ptr(),
                             scores.data_ptr() if scores is not None else None, N, D, K, _dt(C),
                             _stream_ptr(H.device))
    _raise(st, "hd_similarity")
    return (labels, scores) if return_scores else labels


def infer_workspace_bytes(N: int, F: int, D: int, K: int, dtype) -> int:
    dt = _dt_of(dtype)
    return int(lib().hd_infer_workspace_bytes(N, F, D, K, dt))


def infer_kernel(N: int, F: int, D: int, K: int, dtype, packed: bool = True) -> str:
    """Name of the main kernel hd_infer / hd_infer_packed launches for these sizes."""
    dt = _dt_of(dtype)
    return lib().hd_infer_kernel(N, F, D, K, dt, 1 if packed else 0).decode()


def _act(act: str, deterministic: bool) -> int:
    return ACTS[act] | (HD_DETERMINISTIC if deterministic else 0)


def infer(X, B, C, act: str = "hardsign", return_scores: bool = False, out=None,
          workspace=None, deterministic: bool = False):
    """Alg. 1 fused: labels[N] int32 (and scores[N, K] float32).

    ``deterministic``: bit-identical scores and labels from call to call
    (fixed-order reduction of the partial scores).

    ``out`` may be a (labels, scores-or-None) pair of preallocated tensors.
    ``workspace`` may be a zeroed uint8 device tensor of at least
    ``infer_workspace_bytes(...)`` bytes; otherwise a cached one is used.
    """
    torch = _torch()
    _check_dev(X, B, C)
    if not (X.dtype == B.dtype == C.dtype):
        raise TypeError("X, B and C must share a dtype")
    N, F = X.shape
    F2, D = B.shape
    K, D2 = C.shape
    if F2 != F or D2 != D:
        raise ValueError("shape mismatch")
    dt = _dt(X)
    L = lib()
    if out is not None:
        labels, scores = out
    else:
        labels = torch.empty(N, dtype=torch.int32, device=X.device)
        scores = (torch.empty((N, K), dtype=torch.float32, device=X.device)
                  if return_scores else None)
    need = int(L.hd_infer_workspace_bytes(N, F, D, K, dt))
    ws = workspace if workspace is not None else _workspace(X.device, need, ("infer", N, F, D, K, dt))
    st = L.hd_infer(X.data_ptr(), B.data_ptr(), C.data_ptr(), labels.data_ptr(),
                    scores.data_ptr() if scores is not None else None, N, F, D, K, dt,
                    _act(act, deterministic),
                    ws.data_ptr() if ws is not None else None,
                    ws.numel() if ws is not None else 0, _stream_ptr(X.device))
    _raise(st, "hd_infer")
    return (labels, scores) if (return_scores or out is not None) else labels


class PackedModel:
    """A model tiled once by ``hd_pack_model`` (opaque device image)."""

    def __init__(self, image, F: int, D: int, K: int, dt: int):
        self.image, self.F, self.D, self.K, self.dt = image, F, D, K, dt


def pack_model(B, C=None, K: int = 1) -> PackedModel:
    """Tile B and C once (Sec. III-D). ``C=None`` packs B alone (the class
    part of the image is zero, sized for ``K`` classes): a model for
    ``bundle_classes_packed`` before the class hypervectors exist."""
    torch = _torch()
    _check_dev(B)
    F, D = B.shape
    if C is not None:
        _check_dev(C)
        if B.dtype != C.dtype:
            raise TypeError("B and C must share a dtype")
        K, D2 = C.shape
        if D2 != D:
            raise ValueError("shape mismatch")
    dt = _dt(B)
    L = lib()
    nbytes = int(L.hd_model_packed_bytes(F, D, K, dt))
    image = torch.empty(nbytes, dtype=torch.uint8, device=B.device)
    st = L.hd_pack_model(B.data_ptr(), C.data_ptr() if C is not None else None, F, D, K, dt,
                         image.data_ptr(), nbytes, _stream_ptr(B.device))
    _raise(st, "hd_pack_model")
    return PackedModel(image, F, D, K, dt)


def infer_packed(X, model: PackedModel, act: str = "hardsign", return_scores: bool = False,
                 out=None, workspace=None, deterministic: bool = False):
    """Alg. 1 fused from a packed model: labels[N] (and scores[N, K])."""
    torch = _torch()
    _check_dev(X)
    if _dt(X) != model.dt:
        raise TypeError("X dtype differs from the packed model's")
    N, F = X.shape
    if F != model.F:
        raise ValueError("shape mismatch")
    D, K, dt = model.D, model.K, model.dt
    L = lib()
    if out is not None:
        labels, scores = out
    else:
        labels = torch.empty(N, dtype=torch.int32, device=X.device)
        scores = (torch.empty((N, K), dtype=torch.float32, device=X.device)
                  if return_scores else None)
    need = int(L.hd_infer_packed_workspace_bytes(N, F, D, K, dt))
    ws = workspace if workspace is not None else _workspace(X.device, need,
                                                            ("packed", N, F, D, K, dt))
    st = L.hd_infer_packed(X.data_ptr(), model.image.data_ptr(), labels.data_ptr(),
                           scores.data_ptr() if scores is not None else None, N, F, D, K, dt,
                           _act(act, deterministic), ws.data_ptr() if ws is not None else None,
                           ws.numel() if ws is not None else 0, _stream_ptr(X.device))
    _raise(st, "hd_infer_packed")
    return (labels, scores) if (return_scores or out is not None) else labels


def infer_packed_noalloc(X, model: PackedModel, act: str = "hardsign", return_scores: bool = False,
                         out=None, deterministic: bool = False):
    """``infer_packed`` on the library's fixed scratch (no workspace argument;
    calls on one GPU must not overlap in time)."""
    torch = _torch()
    _check_dev(X)
    if _dt(X) != model.dt:
        raise TypeError("X dtype differs from the packed model's")
    N, F = X.shape
    if F != model.F:
        raise ValueError("shape mismatch")
    D, K, dt = model.D, model.K, model.dt
    if out is not None:
        labels, scores = out
    else:
        labels = torch.empty(N, dtype=torch.int32, device=X.device)
        scores = (torch.empty((N, K), dtype=torch.float32, device=X.device)
                  if return_scores else None)
    st = lib().hd_infer_packed_noalloc(X.data_ptr(), model.image.data_ptr(), labels.data_ptr(),
                                       scores.data_ptr() if scores is not None else None, N, F, D,
                                       K, dt, _act(act, deterministic), _stream_ptr(X.device))
    _raise(st, "hd_infer_packed_noalloc")
    return (labels, scores) if (return_scores or out is not None) else labels


def stream_workspace_bytes(nbatch: int, N: int, F: int, D: int, K: int, dtype) -> int:
    dt = _dt_of(dtype)
    return int(lib().hd_infer_stream_workspace_bytes(nbatch, N, F, D, K, dt))


def infer_stream(X, model: PackedModel, act: str = "hardsign", return_scores: bool = False,
                 ready=None, done=None, out=None, workspace=None):
    """Streaming inference: ``X`` is [nbatch, N, F] (a queue of batches); one
    persistent launch returns labels [nbatch, N] (and scores [nbatch, N, K]).

    ``ready``/``done``: optional int32 tensors of one element (device memory
    or pinned host memory) for the queue counter and the batches-done counter.
    ``workspace``: a zeroed uint8 device tensor of at least
    ``stream_workspace_bytes(...)`` bytes; otherwise a cached one is used."""
    torch = _torch()
    _check_dev(X)
    if _dt(X) != model.dt:
        raise TypeError("X dtype differs from the packed model's")
    if X.dim() != 3:
        raise ValueError("X must be [nbatch, N, F]")
    nbatch, N, F = X.shape
    if F != model.F:
        raise ValueError("shape mismatch")
    D, K, dt = model.D, model.K, model.dt
    L = lib()
    if out is not None:
        labels, scores = out
    else:
        labels = torch.empty((nbatch, N), dtype=torch.int32, device=X.device)
        scores = (torch.empty((nbatch, N, K), dtype=torch.float32, device=X.device)
                  if return_scores else None)
    need = int(L.hd_infer_stream_workspace_bytes(nbatch, N, F, D, K, dt))
    if need == 0 and nbatch > 0:
        raise HDError(HD_ERR_UNSUPPORTED, "hd_infer_stream")
    ws = workspace if workspace is not None else _workspace(X.device, need,
                                                            ("stream", nbatch, N, F, D, K, dt))
    st = L.hd_infer_stream(X.data_ptr(), model.image.data_ptr(),
                           ready.data_ptr() if ready is not None else None, labels.data_ptr(),
                           scores.data_ptr() if scores is not None else None,
                           done.data_ptr() if done is not None else None, nbatch, N, F, D, K, dt,
                           ACTS[act], ws.data_ptr() if ws is not None else None,
                           ws.numel() if ws is not None else 0, _stream_ptr(X.device))
    _raise(st, "hd_infer_stream")
    return (labels, scores) if (return_scores or out is not None) else labels


def bundle_classes(X, B, y, K: int, counts=None):
    """Single-pass training, accumulation step (Sec. II-C): adds
    HardSign(X_n B) into ``counts[y[n]]`` for every sample with 0 <= y[n] < K
    and returns ``counts`` ([K, D] int32; a new zeroed tensor when None).
    Calls with the same ``counts`` accumulate, so a training set can be fed
    in chunks."""
    torch = _torch()
    _check_dev(X, B, y)
    if X.dtype != B.dtype:
        raise TypeError("X and B must have the same dtype")
    if y.dtype != torch.int32:
        raise TypeError("y must be int32")
    N, F = X.shape
    F2, D = B.shape
    if F2 != F or y.shape != (N,):
        raise ValueError("shape mismatch")
    if counts is None:
        counts = torch.zeros((K, D), dtype=torch.int32, device=X.device)
    else:
        _check_dev(counts)
        if counts.dtype != torch.int32 or tuple(counts.shape) != (K, D):
            raise ValueError("counts must be int32 [K, D]")
    st = lib().hd_bundle_classes(X.data_ptr(), B.data_ptr(), y.data_ptr(), counts.data_ptr(), N,
                                 F, D, K, _dt(X), _stream_ptr(X.device))
    _raise(st, "hd_bundle_classes")
    return counts


def bundle_classes_packed(X, model: PackedModel, y, K: int, counts=None):
    """``bundle_classes`` on the matrix cores, reading B from a packed model
    (``pack_model(B)`` or ``pack_model(B, C)``; the class part is not read)."""
    torch = _torch()
    _check_dev(X, y)
    if _dt(X) != model.dt:
        raise TypeError("X dtype differs from the packed model's")
    if y.dtype != torch.int32:
        raise TypeError("y must be int32")
    N, F = X.shape
    if F != model.F or y.shape != (N,):
        raise ValueError("shape mismatch")
    D = model.D
    if counts is None:
        counts = torch.zeros((K, D), dtype=torch.int32, device=X.device)
    else:
        _check_dev(counts)
        if counts.dtype != torch.int32 or tuple(counts.shape) != (K, D):
            raise ValueError("counts must be int32 [K, D]")
    st = lib().hd_bundle_classes_packed(X.data_ptr(), model.image.data_ptr(), y.data_ptr(),
                                        counts.data_ptr(), N, F, D, K, model.dt,
                                        _stream_ptr(X.device))
    _raise(st, "hd_bundle_classes_packed")
    return counts


def bundle_kernel(N: int, F: int, D: int, K: int, dtype, packed: bool = True) -> str:
    """Name of the kernel bundle_classes(_packed) launches for these sizes."""
    dt = _dt_of(dtype)
    return lib().hd_bundle_kernel(N, F, D, K, dt, 1 if packed else 0).decode()


def class_hardsign(counts, out=None):
    """Normalisation step (Eq. 1): the class hypervectors M [K, D] float32,
    +1 where counts >= 0 (ties and empty classes) and -1 elsewhere."""
    torch = _torch()
    _check_dev(counts)
    if counts.dtype != torch.int32 or counts.dim() != 2:
        raise ValueError("counts must be int32 [K, D]")
    K, D = counts.shape
    M = out if out is not None else torch.empty((K, D), dtype=torch.float32,
                                                device=counts.device)
    _check_dev(M)
    if M.dtype != torch.float32 or tuple(M.shape) != (K, D):
        raise ValueError("out must be float32 [K, D]")
    st = lib().hd_class_hardsign(counts.data_ptr(), M.data_ptr(), K, D,
                                 _stream_ptr(counts.device))
    _raise(st, "hd_class_hardsign")
    return M


def train(X, B, y, K: int):
    """Single-pass training in one call: M [K, D] float32 = class_hardsign(
    bundle_classes(X, B, y, K))."""
    return class_hardsign(bundle_classes(X, B, y, K))
