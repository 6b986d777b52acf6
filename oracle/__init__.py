"""CPU oracle for RITA group attention -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The GPU library never loads it, and the
two share no code: the oracle is plain fp64 C (``ga_oracle.c``) written from
the paper's definitions, wrapped here with ctypes.

Functions take/return numpy arrays; inputs may be any float array holding the
exact values of the bf16 / fp32 tensors (they are widened to float64 here).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ga_oracle.c")
# GA_ORACLE_LIB lets the mutation test point the wrapper at a deliberately
# broken build of the same source.
_LIB = os.environ.get("GA_ORACLE_LIB") or os.path.join(_HERE, "libga_oracle.so")

DTYPES = {"f32": 0, "bf16": 1}


def build(force: bool = True, src: str = _SRC, out: str | None = None) -> str:
    """Compile the oracle with gcc (strict IEEE: no fast-math, no x87)."""
    out = out or _LIB
    if force or not os.path.exists(out):
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
               "-fno-fast-math", "-o", out + ".tmp", src, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(out + ".tmp", out)
    return out


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32, i64, f64 = ctypes.c_int, ctypes.c_int64, ctypes.c_double
        lib.ga_oracle_cluster.argtypes = [i32, i32, i32, i32, i32, P, i32, i32, P, P, P, P, P, P, P]
        lib.ga_oracle_cluster.restype = i64
        lib.ga_oracle_aggregate.argtypes = [i32, i32, i32, i32, P, P, i32, P]
        lib.ga_oracle_aggregate.restype = i64
        lib.ga_oracle_attend.argtypes = [i32, i32, i32, i32, i32, P, P, P, P, i32, f64, P]
        lib.ga_oracle_attend.restype = None
        lib.ga_oracle_merge_plan.argtypes = [i32, i32, i32, i32, P, P, P, P, P, i32, f64, f64, P, P, P, P]
        lib.ga_oracle_merge_plan.restype = None
        lib.ga_oracle_threads.argtypes = [i32]
        lib.ga_oracle_threads.restype = i32
        _lib = lib
    return _lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def _f64(x):
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def threads(n: int = 0) -> int:
    """Set (n > 0) and return the OpenMP thread count the oracle uses."""
    return _load().ga_oracle_threads(int(n))


def cluster(K, N: int, iters: int, dtype: str, init=None, trace: bool = False):
    """Lloyd grouping of the keys of every (b, h) slice (Section 4.4).

    K: [B, H, n, d].  Returns dict with belong [B,H,n] int32, count [B,H,N]
    int32, centroid [B,H,N,d] float32, inexact (count of inexact fp64 adds in
    the centroid sums) and, if trace, per-iteration belong / margin (second
    best minus best canonical score) / centroid, each with a leading iters axis.
    """
    K = _f64(K)
    B, H, n, d = K.shape
    belong = np.empty((B, H, n), np.int32)
    count = np.empty((B, H, N), np.int32)
    centroid = np.empty((B, H, N, d), np.float32)
    init_a = None if init is None else np.ascontiguousarray(np.asarray(init, np.float32))
    tb = tm = tc = None
    if trace:
        tb = np.empty((iters, B, H, n), np.int32)
        tm = np.empty((iters, B, H, n), np.float64)
        tc = np.empty((iters, B, H, N, d), np.float32)
    inexact = _load().ga_oracle_cluster(B, H, n, d, DTYPES[dtype], _ptr(K), N, iters, _ptr(init_a),
                                        _ptr(belong), _ptr(count), _ptr(centroid), _ptr(tb), _ptr(tm),
                                        _ptr(tc))
    out = dict(belong=belong, count=count, centroid=centroid, inexact=int(inexact))
    if trace:
        out.update(trace_belong=tb, trace_margin=tm, trace_centroid=tc)
    return out


def aggregate(V, belong, N: int):
    """Per-group fp64 sums of the value vectors (embedding aggregation)."""
    V = _f64(V)
    B, H, n, d = V.shape
    bel = np.ascontiguousarray(np.asarray(belong, np.int32))
    vsum = np.empty((B, H, N, d), np.float64)
    inexact = _load().ga_oracle_aggregate(B, H, n, d, _ptr(V), _ptr(bel), N, _ptr(vsum))
    return vsum, int(inexact)


def attend(Q, centroid, count, vsum, N: int, scale: float, dtype: str):
    """Group softmax (Eq. 3) and output combine; returns O [B,H,n,d] float64."""
    Q = _f64(Q)
    B, H, n, d = Q.shape
    cen = np.ascontiguousarray(np.asarray(centroid, np.float32))
    cnt = np.ascontiguousarray(np.asarray(count, np.int32))
    vs = _f64(vsum)
    O = np.empty((B, H, n, d), np.float64)
    _load().ga_oracle_attend(B, H, n, d, DTYPES[dtype], _ptr(Q), _ptr(cen), _ptr(cnt), _ptr(vs), N,
                             float(scale), _ptr(O))
    return O


def forward(Q, K, V, N: int, iters: int, scale: float, dtype: str, init=None):
    """Whole group-attention forward: grouping, aggregation, attention."""
    cl = cluster(K, N, iters, dtype, init=init)
    vsum, inexact_v = aggregate(V, cl["belong"], N)
    O = attend(Q, cl["centroid"], cl["count"], vsum, N, scale, dtype)
    return dict(O=O, vsum=vsum, inexact_v=inexact_v, **cl)


def merge_plan(Q, K, belong, centroid, count, N: int, scale: float, eps: float):
    """Adaptive scheduler's merge plan (Section 5.1, Lemma 1, Eq. 5) of a
    grouping: per slice the group radii, the distance threshold
    dthr = ln(eps) / (2 |scale| max|q|), each S2 group's lowest S1 partner
    (-1 if not mergeable) and the number of mergeable groups."""
    import math

    Q, K = _f64(Q), _f64(K)
    B, H, n, d = K.shape
    bel = np.ascontiguousarray(np.asarray(belong, np.int32))
    cen = np.ascontiguousarray(np.asarray(centroid, np.float32))
    cnt = np.ascontiguousarray(np.asarray(count, np.int32))
    radius = np.empty((B, H, N), np.float64)
    dthr = np.empty((B, H), np.float64)
    partner = np.empty((B, H, N), np.int32)
    merges = np.empty((B, H), np.int32)
    _load().ga_oracle_merge_plan(B, H, n, d, _ptr(Q), _ptr(K), _ptr(bel), _ptr(cen), _ptr(cnt), N, float(scale),
                                 math.log(eps), _ptr(radius), _ptr(dthr), _ptr(partner), _ptr(merges))
    return dict(radius=radius, dthr=dthr, partner=partner, merges=merges)


def next_group_count(N: int, merges, alpha: float) -> int:
    """Momentum update of the group count (Section 5.1):
    N_new = alpha (N - D) + (1 - alpha) N, with D the fewest mergeable groups
    over the slices (so that every slice keeps its bound), rounded to the
    nearest integer (halves up) and kept in [1, N]."""
    D = int(np.min(np.asarray(merges))) if np.size(merges) else 0
    x = alpha * (N - D) + (1.0 - alpha) * N
    return int(min(N, max(1, np.floor(x + 0.5))))


def round_bf16(x):
    """bf16 RNE of float32 values, as float32 (numpy, for test expectations)."""
    u = np.ascontiguousarray(np.asarray(x, np.float32)).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def round_bf16_f64(x):
    """bf16 round-to-nearest-even of float64 values in ONE rounding (no
    intermediate float32), as float64.  Normal bf16 range only."""
    m, e = np.frexp(np.asarray(x, np.float64))  # x = m 2^e, 0.5 <= |m| < 1
    return np.ldexp(np.rint(m * 256.0), e - 8)  # 8 significant bits; rint ties to even


def project_qkv(X, Wqkv, H: int):
    """Eq. 1 projections Q = X W_Q, K = X W_K, V = X W_V of token embeddings
    X [B, n, D] with Wqkv [3D, D] holding one output feature per row (Q rows,
    then K, then V; row 64 h + c = feature c of head h): exact fp64 products,
    each rounded once to bf16.  Returns Q, K, V as [B, H, n, 64] float64."""
    X, W = _f64(X), _f64(Wqkv)
    B, n, D = X.shape
    P = round_bf16_f64(X @ W.T)  # [B, n, 3D]
    heads = P.reshape(B, n, 3, H, 64).transpose(2, 0, 3, 1, 4)  # [3, B, H, n, 64]
    return tuple(np.ascontiguousarray(heads[i]) for i in range(3))


def project_out(O, Wo):
    """Output projection of the Transformer encoder's multi-head attention:
    the heads' outputs O [B, H, n, 64] concatenated per token (feature 64 h + c)
    times Wo^T (Wo [D, D], one output feature per row), rounded once to bf16."""
    O, W = _f64(O), _f64(Wo)
    B, H, n, d = O.shape
    cat = O.transpose(0, 2, 1, 3).reshape(B, n, H * d)
    return round_bf16_f64(cat @ W.T)


def attention_block(X, Wqkv, Wo, H: int, N: int, iters: int, scale: float):
    """RITA encoder attention block (Section 3: a Transformer encoder whose
    self-attention is group attention): projections (Eq. 1), the group
    attention forward of every (b, h) slice in bf16 storage, its output rounded
    to bf16, then the output projection.  Returns dict(Y, Q, K, V, O, belong,
    count, centroid)."""
    Q, K, V = project_qkv(X, Wqkv, H)
    r = forward(Q, K, V, N, iters, scale, "bf16")
    O = round_bf16_f64(r["O"])
    Y = project_out(O, Wo)
    return dict(Y=Y, Q=Q, K=K, V=V, O=O, belong=r["belong"], count=r["count"], centroid=r["centroid"])


def backward(Q, dO, belong, centroid, count, vsum, N: int, scale: float, dtype: str):
    """Gradient of the group-attention forward (Eq. 3, Algorithm 1) with the
    grouping held fixed (BELONG / COUNT are piecewise constant in the keys).
    r_j = round_dt(centroid_j) with the rounding passed straight through, so
    dr_j reaches every member key as dr_j / c_j (r_j is the member mean);
    mu_j = vsum_j / c_j reaches every member value as dmu_j / c_j.  fp64.
    Returns (dQ, dK, dV), each [B, H, n, d]."""
    Q, G = _f64(Q), _f64(dO)
    B, H, n, d = Q.shape
    C = _f64(centroid)
    R = round_bf16_f64(C) if dtype == "bf16" else C
    c = np.asarray(count, np.float64)
    cs = np.where(c > 0, c, 1.0)
    mu = np.where((c > 0)[..., None], _f64(vsum) / cs[..., None], 0.0)
    p = scale * np.einsum("bhid,bhjd->bhij", Q, R)
    live = (c > 0)[:, :, None, :]
    m = np.max(np.where(live, p, -np.inf), axis=-1, keepdims=True)
    m = np.where(np.isfinite(m), m, 0.0)
    e = np.where(live, c[:, :, None, :] * np.exp(p - m), 0.0)
    S = e.sum(-1, keepdims=True)
    w = np.where(S > 0, e / np.where(S > 0, S, 1.0), 0.0)
    dw = np.einsum("bhid,bhjd->bhij", G, mu)
    D = (w * dw).sum(-1, keepdims=True)
    dp = w * (dw - D)
    dQ = scale * np.einsum("bhij,bhjd->bhid", dp, R)
    dr = scale * np.einsum("bhij,bhid->bhjd", dp, Q)
    dmu = np.einsum("bhij,bhid->bhjd", w, G)
    idx = np.asarray(belong, np.int64)[..., None]
    per_k = np.take_along_axis(cs, idx[..., 0], axis=2)[..., None]
    dK = np.take_along_axis(dr, idx, axis=2) / per_k
    dV = np.take_along_axis(dmu, idx, axis=2) / per_k
    return dQ, dK, dV
