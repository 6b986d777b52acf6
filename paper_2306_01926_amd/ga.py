"""Python binding of libga.so: argument marshalling only.

Every function takes torch CUDA tensors, allocates outputs (and a cached
workspace) with torch, and calls the C ABI declared in include/ga.h on the
current torch stream.  All computation happens in the HIP kernels; there is no
CPU fallback: if the library is missing the call raises.
"""
from __future__ import annotations

import ctypes
import math
import os

import torch

# GA_LIB lets the sanitizer test load an instrumented build of the same sources.
_LIB_PATH = os.environ.get("GA_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "libga.so")

GA_F32, GA_BF16 = 0, 1
STATUS = {0: "GA_OK", 1: "GA_ERR_INVALID_ARG", 2: "GA_ERR_UNSUPPORTED", 3: "GA_ERR_WORKSPACE", 4: "GA_ERR_HIP"}
SYMBOLS = ("ga_workspace_bytes", "ga_cluster", "ga_aggregate", "ga_attend", "ga_forward",
           "ga_block_workspace_bytes", "ga_project_qkv", "ga_project_out", "ga_attention_block",
           "ga_merge_plan", "ga_next_group_count", "ga_backward_workspace_bytes", "ga_backward",
           "ga_timing_enable", "ga_timing_collect", "ga_status_string", "ga_last_error", "ga_workspace_check",
           "ga_forward_noalloc")


class Shape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("H", ctypes.c_int32), ("n", ctypes.c_int32),
                ("d", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class KernelTime(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("launches", ctypes.c_int32), ("total_ms", ctypes.c_double)]


class GAError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded libga.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(_LIB_PATH)
        P, i32 = ctypes.c_void_p, ctypes.c_int32
        L.ga_workspace_bytes.argtypes = [Shape, i32]
        L.ga_workspace_bytes.restype = ctypes.c_size_t
        L.ga_cluster.argtypes = [Shape, P, i32, i32, P, P, P, P, P, ctypes.c_size_t, P]
        L.ga_aggregate.argtypes = [Shape, P, P, i32, P, P, ctypes.c_size_t, P]
        L.ga_attend.argtypes = [Shape, P, P, P, P, i32, ctypes.c_float, P, P, ctypes.c_size_t, P]
        L.ga_forward.argtypes = [Shape, P, P, P, i32, i32, ctypes.c_float, P, P, P, P, P, ctypes.c_size_t, P]
        L.ga_forward_noalloc.argtypes = [Shape, P, P, P, i32, i32, ctypes.c_float, P, P, P, P, P]
        L.ga_block_workspace_bytes.argtypes = [Shape, i32]
        L.ga_block_workspace_bytes.restype = ctypes.c_size_t
        L.ga_project_qkv.argtypes = [Shape, P, P, P, P, P, P]
        L.ga_project_out.argtypes = [Shape, P, P, P, P]
        L.ga_attention_block.argtypes = [Shape, P, P, P, i32, i32, ctypes.c_float, P, P, ctypes.c_size_t, P]
        L.ga_merge_plan.argtypes = [Shape, P, P, P, P, P, i32, ctypes.c_float, ctypes.c_double, P, P, P, P, P]
        L.ga_backward_workspace_bytes.argtypes = [Shape, i32]
        L.ga_backward_workspace_bytes.restype = ctypes.c_size_t
        L.ga_backward.argtypes = [Shape, P, P, P, P, P, P, i32, ctypes.c_float, P, P, P, P, ctypes.c_size_t, P]
        L.ga_next_group_count.argtypes = [i32, P, ctypes.c_int64, ctypes.c_double]
        L.ga_next_group_count.restype = i32
        for f in ("ga_cluster", "ga_aggregate", "ga_attend", "ga_forward", "ga_forward_noalloc", "ga_project_qkv",
                  "ga_project_out",
                  "ga_attention_block", "ga_merge_plan", "ga_backward"):
            getattr(L, f).restype = ctypes.c_int
        L.ga_workspace_check.argtypes = [Shape, i32, P, ctypes.c_size_t, P]
        L.ga_workspace_check.restype = ctypes.c_int
        L.ga_timing_enable.argtypes = [ctypes.c_int]
        L.ga_timing_enable.restype = ctypes.c_int
        L.ga_timing_collect.argtypes = [ctypes.POINTER(KernelTime), i32, ctypes.POINTER(i32)]
        L.ga_timing_collect.restype = ctypes.c_int
        L.ga_status_string.argtypes = [ctypes.c_int]
        L.ga_status_string.restype = ctypes.c_char_p
        L.ga_last_error.argtypes = []
        L.ga_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return GA_BF16
    if t.dtype == torch.float32:
        return GA_F32
    raise TypeError(f"unsupported dtype {t.dtype} (bf16 or fp32)")


def shape_of(X: torch.Tensor) -> Shape:
    if X.dim() != 4:
        raise ValueError("expected a [B, H, n, d] tensor")
    B, H, n, d = X.shape
    return Shape(B, H, n, d, _dtype_code(X))


def _p(t):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _expect(t, name: str, device, dtype, shape=None, optional: bool = False):
    """Check a tensor handed to the C ABI, which cannot check buffer sizes:
    it must live on `device` (a CUDA device), have `dtype`, be contiguous and
    (if given) have exactly `shape`.  Raises ValueError otherwise, before any
    pointer reaches a kernel."""
    if t is None:
        if optional:
            return
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch tensor")
    if t.device.type != "cuda" or t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _device_of(X: torch.Tensor):
    if X.device.type != "cuda":
        raise ValueError(f"tensors must be on a CUDA device (got {X.device})")
    return X.device


def _qkv_like(X: torch.Tensor, name: str):
    """Shape [B, H, n, d] and the device of the first operand of a call."""
    if not isinstance(X, torch.Tensor) or X.dim() != 4:
        raise ValueError(f"{name} must be a [B, H, n, d] tensor")
    return _device_of(X)


def _check(rc: int):
    if rc != 0:
        raise GAError(rc, lib().ga_last_error().decode())


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


_ws_cache: dict = {}


def workspace_bytes(shape: Shape, N: int) -> int:
    return int(lib().ga_workspace_bytes(shape, int(N)))


def workspace(shape: Shape, N: int, device, stream=None) -> tuple:
    """A cached device workspace (uint8 tensor) large enough for (shape, N).

    One buffer per (device, stream): the workspace carries state between the
    launches of one call, and calls on one stream run one after another, so
    calls without ws on different streams never share a buffer.  The buffer
    is allocated on (and its memory ordered by) that stream.
    """
    device = torch.device(device)
    if stream is None:
        stream = torch.cuda.current_stream(device)
    nbytes = max(workspace_bytes(shape, N), 256)
    key = (device, stream.cuda_stream)
    ws = _ws_cache.get(key)
    if ws is None or ws.numel() < nbytes:
        with torch.cuda.stream(stream):
            ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
        _ws_cache[key] = ws
    return ws, ws.numel()


def _ws_args(shape, N, device, ws):
    if ws is None:
        ws, nb = workspace(shape, N, device)
    else:
        _expect(ws, "ws", device, torch.uint8)
        nb = ws.numel() * ws.element_size()
    return _p(ws), nb


def cluster(K: torch.Tensor, N: int, iters: int, init: torch.Tensor | None = None, ws=None):
    """Grouping of the keys: returns (belong [B,H,n] int32, count [B,H,N] int32,
    centroid [B,H,N,d] fp32)."""
    dev = _qkv_like(K, "K")
    s = shape_of(K)
    B, H, n, d = K.shape
    _expect(init, "init", dev, torch.float32, (B, H, N, d), optional=True)
    belong = torch.empty(K.shape[:3], dtype=torch.int32, device=dev)
    count = torch.empty((*K.shape[:2], N), dtype=torch.int32, device=dev)
    centroid = torch.empty((*K.shape[:2], N, K.shape[3]), dtype=torch.float32, device=dev)
    wp, nb = _ws_args(s, N, dev, ws)
    _check(lib().ga_cluster(s, _p(K), int(N), int(iters), _p(init), _p(belong), _p(count), _p(centroid),
                            wp, nb, _stream(dev)))
    return belong, count, centroid


def aggregate(V: torch.Tensor, belong: torch.Tensor, N: int, ws=None) -> torch.Tensor:
    """Per-group fp32 sums of the values (fp64 accumulation)."""
    dev = _qkv_like(V, "V")
    s = shape_of(V)
    _expect(belong, "belong", dev, torch.int32, V.shape[:3])
    vsum = torch.empty((*V.shape[:2], N, V.shape[3]), dtype=torch.float32, device=dev)
    wp, nb = _ws_args(s, N, dev, ws)
    _check(lib().ga_aggregate(s, _p(V), _p(belong), int(N), _p(vsum), wp, nb, _stream(dev)))
    return vsum


def attend(Q: torch.Tensor, centroid: torch.Tensor, count: torch.Tensor, vsum: torch.Tensor, N: int,
           scale: float | None = None, ws=None) -> torch.Tensor:
    """Group softmax and combine; returns O [B,H,n,d] in Q's dtype."""
    dev = _qkv_like(Q, "Q")
    s = shape_of(Q)
    B, H, n, d = Q.shape
    _expect(centroid, "centroid", dev, torch.float32, (B, H, N, d))
    _expect(count, "count", dev, torch.int32, (B, H, N))
    _expect(vsum, "vsum", dev, torch.float32, (B, H, N, d))
    scale = 1.0 / math.sqrt(Q.shape[3]) if scale is None else float(scale)
    O = torch.empty_like(Q)
    wp, nb = _ws_args(s, N, dev, ws)
    _check(lib().ga_attend(s, _p(Q), _p(centroid), _p(count), _p(vsum), int(N), scale, _p(O), wp, nb,
                           _stream(dev)))
    return O


def forward(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, N: int, iters: int,
            scale: float | None = None, return_groups: bool = False, out: torch.Tensor | None = None,
            ws=None):
    """Whole group-attention forward; optionally also (belong, count, centroid)."""
    dev = _qkv_like(Q, "Q")
    s = shape_of(Q)
    for t, nm in ((K, "K"), (V, "V"), (out, "out")):
        _expect(t, nm, dev, Q.dtype, Q.shape, optional=nm == "out")
    scale = 1.0 / math.sqrt(Q.shape[3]) if scale is None else float(scale)
    O = torch.empty_like(Q) if out is None else out
    belong = count = centroid = None
    if return_groups:
        belong = torch.empty(K.shape[:3], dtype=torch.int32, device=dev)
        count = torch.empty((*K.shape[:2], N), dtype=torch.int32, device=dev)
        centroid = torch.empty((*K.shape[:2], N, K.shape[3]), dtype=torch.float32, device=dev)
    wp, nb = _ws_args(s, N, dev, ws)
    _check(lib().ga_forward(s, _p(Q), _p(K), _p(V), int(N), int(iters), scale, _p(O), _p(belong), _p(count),
                            _p(centroid), wp, nb, _stream(dev)))
    return (O, belong, count, centroid) if return_groups else O


def forward_noalloc(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, N: int, iters: int,
                    scale: float | None = None, return_groups: bool = False, out: torch.Tensor | None = None):
    """forward() through ga_forward_noalloc: no workspace, the library's static
    scratch instead (bf16, shapes of the one-launch grouping only).  Calls that
    overlap in time on one GPU share that scratch and race."""
    dev = _qkv_like(Q, "Q")
    s = shape_of(Q)
    for t, nm in ((K, "K"), (V, "V"), (out, "out")):
        _expect(t, nm, dev, Q.dtype, Q.shape, optional=nm == "out")
    scale = 1.0 / math.sqrt(Q.shape[3]) if scale is None else float(scale)
    O = torch.empty_like(Q) if out is None else out
    belong = count = centroid = None
    if return_groups:
        belong = torch.empty(K.shape[:3], dtype=torch.int32, device=dev)
        count = torch.empty((*K.shape[:2], N), dtype=torch.int32, device=dev)
        centroid = torch.empty((*K.shape[:2], N, K.shape[3]), dtype=torch.float32, device=dev)
    _check(lib().ga_forward_noalloc(s, _p(Q), _p(K), _p(V), int(N), int(iters), scale, _p(O), _p(belong),
                                    _p(count), _p(centroid), _stream(dev)))
    return (O, belong, count, centroid) if return_groups else O


def block_shape(X: torch.Tensor, H: int) -> Shape:
    """Shape of the attention block for token embeddings X [B, n, 64 H]."""
    if X.dim() != 3 or X.shape[2] != 64 * H:
        raise ValueError(f"expected X of shape [B, n, {64 * H}]")
    return Shape(X.shape[0], H, X.shape[1], 64, _dtype_code(X))


def project_qkv(X: torch.Tensor, Wqkv: torch.Tensor, H: int):
    """(Q, K, V) [B, H, n, 64] = per-head slices of X Wqkv^T (Wqkv [3D, D], rows = outputs)."""
    s = block_shape(X, H)
    dev = _device_of(X)
    B, n, D = X.shape
    _expect(Wqkv, "Wqkv", dev, X.dtype, (3 * D, D))
    Q, K, V = (torch.empty((B, H, n, 64), dtype=X.dtype, device=X.device) for _ in range(3))
    _check(lib().ga_project_qkv(s, _p(X), _p(Wqkv), _p(Q), _p(K), _p(V), _stream(X.device)))
    return Q, K, V


def project_out(O: torch.Tensor, Wo: torch.Tensor) -> torch.Tensor:
    """Y [B, n, D] = heads of O [B, H, n, 64] concatenated, times Wo^T (Wo [D, D])."""
    dev = _qkv_like(O, "O")
    B, H, n, d = O.shape
    _expect(Wo, "Wo", dev, O.dtype, (H * d, H * d))
    Y = torch.empty((B, n, H * d), dtype=O.dtype, device=O.device)
    _check(lib().ga_project_out(Shape(B, H, n, d, _dtype_code(O)), _p(O), _p(Wo), _p(Y), _stream(O.device)))
    return Y


def block_workspace_bytes(shape: Shape, N: int) -> int:
    return int(lib().ga_block_workspace_bytes(shape, int(N)))


def attention_block(X: torch.Tensor, Wqkv: torch.Tensor, Wo: torch.Tensor, H: int, N: int, iters: int,
                    scale: float | None = None, out: torch.Tensor | None = None, ws=None) -> torch.Tensor:
    """Attention block: projections, group-attention forward, output projection.
    ws: a uint8 device tensor of block_workspace_bytes(shape, N) (allocated if None)."""
    s = block_shape(X, H)
    dev = _device_of(X)
    D = X.shape[2]
    _expect(Wqkv, "Wqkv", dev, X.dtype, (3 * D, D))
    _expect(Wo, "Wo", dev, X.dtype, (D, D))
    _expect(out, "out", dev, X.dtype, X.shape, optional=True)
    scale = 1.0 / 8.0 if scale is None else float(scale)
    Y = torch.empty_like(X) if out is None else out
    if ws is None:
        ws = torch.empty(max(block_workspace_bytes(s, N), 256), dtype=torch.uint8, device=X.device)
    _expect(ws, "ws", dev, torch.uint8)
    _check(lib().ga_attention_block(s, _p(X), _p(Wqkv), _p(Wo), int(N), int(iters), scale, _p(Y), _p(ws),
                                    ws.numel(), _stream(dev)))
    return Y


def merge_plan(Q: torch.Tensor, K: torch.Tensor, belong: torch.Tensor, centroid: torch.Tensor,
               count: torch.Tensor, N: int, scale: float | None = None, eps: float = 2.0) -> dict:
    """Merge plan of the adaptive group count (Lemma 1 threshold, Eq. 5 rule):
    dict(radius [B,H,N] fp64, dthr [B,H] fp64, partner [B,H,N] int32, merges [B,H] int32)."""
    dev = _qkv_like(K, "K")
    s = shape_of(K)
    B, H, n, d = K.shape
    _expect(Q, "Q", dev, K.dtype, K.shape)
    _expect(belong, "belong", dev, torch.int32, (B, H, n))
    _expect(centroid, "centroid", dev, torch.float32, (B, H, N, d))
    _expect(count, "count", dev, torch.int32, (B, H, N))
    scale = 1.0 / math.sqrt(K.shape[3]) if scale is None else float(scale)
    radius = torch.empty((B, H, N), dtype=torch.float64, device=dev)
    dthr = torch.empty((B, H), dtype=torch.float64, device=dev)
    partner = torch.empty((B, H, N), dtype=torch.int32, device=dev)
    merges = torch.empty((B, H), dtype=torch.int32, device=dev)
    _check(lib().ga_merge_plan(s, _p(Q), _p(K), _p(belong), _p(centroid), _p(count), int(N), scale, float(eps),
                               _p(radius), _p(dthr), _p(partner), _p(merges), _stream(dev)))
    return dict(radius=radius, dthr=dthr, partner=partner, merges=merges)


def next_group_count(N: int, merges, alpha: float) -> int:
    """Momentum update of N from per-slice merge counts (copied to the host)."""
    m = torch.as_tensor(merges).to("cpu", torch.int32).contiguous().reshape(-1)
    r = lib().ga_next_group_count(int(N), ctypes.c_void_p(m.data_ptr()) if m.numel() else None, m.numel(),
                                  float(alpha))
    if r == 0:
        raise GAError(1, lib().ga_last_error().decode())
    return int(r)


def backward_workspace_bytes(shape: Shape, N: int) -> int:
    return int(lib().ga_backward_workspace_bytes(shape, int(N)))


def backward(Q: torch.Tensor, dO: torch.Tensor, belong: torch.Tensor, centroid: torch.Tensor, count: torch.Tensor,
             vsum: torch.Tensor, N: int, scale: float | None = None, ws=None):
    """Gradient of the forward with the grouping fixed: (dQ, dK, dV) [B,H,n,d] bf16."""
    dev = _qkv_like(Q, "Q")
    s = shape_of(Q)
    B, H, n, d = Q.shape
    _expect(dO, "dO", dev, Q.dtype, Q.shape)
    _expect(belong, "belong", dev, torch.int32, (B, H, n))
    _expect(centroid, "centroid", dev, torch.float32, (B, H, N, d))
    _expect(count, "count", dev, torch.int32, (B, H, N))
    _expect(vsum, "vsum", dev, torch.float32, (B, H, N, d))
    scale = 1.0 / math.sqrt(Q.shape[3]) if scale is None else float(scale)
    dQ, dK, dV = (torch.empty_like(Q) for _ in range(3))
    if ws is None:
        ws = torch.empty(max(backward_workspace_bytes(s, N), 256), dtype=torch.uint8, device=dev)
    _expect(ws, "ws", dev, torch.uint8)
    _check(lib().ga_backward(s, _p(Q), _p(dO), _p(belong), _p(centroid), _p(count), _p(vsum), int(N), scale, _p(dQ),
                             _p(dK), _p(dV), _p(ws), ws.numel(), _stream(dev)))
    return dQ, dK, dV


def workspace_check(X: torch.Tensor, N: int, ws=None) -> None:
    """Wait for the current stream and raise GAError if the last grouping
    launch that used this workspace (the cached one if ws is None) gave up a
    cross-workgroup wait."""
    dev = _qkv_like(X, "X")
    s = shape_of(X)
    wp, nb = _ws_args(s, N, dev, ws)
    _check(lib().ga_workspace_check(s, int(N), wp, nb, _stream(dev)))


def timing_enable(on: bool = True) -> None:
    """Bracket every kernel launch (this thread) with hipEvents on its stream."""
    _check(lib().ga_timing_enable(1 if on else 0))


def timing_collect() -> dict:
    """{kernel: (launches, total_ms)} since the last collect; waits for the events."""
    buf = (KernelTime * 64)()
    n = ctypes.c_int32(0)
    _check(lib().ga_timing_collect(buf, 64, ctypes.byref(n)))
    return {buf[i].name.decode(): (int(buf[i].launches), float(buf[i].total_ms)) for i in range(n.value)}
