"""Host-side checks of the C ABI (no GPU needed).

libga.so must load and export every function include/ga.h declares.  Every
argument check runs on the host before any HIP call, so each error status can
be forced here with fake (never dereferenced) device pointers.
"""
import ctypes
import os
import re

import pytest

from paper_2306_01926_amd import ga

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x10000000  # 16-byte aligned, never dereferenced (validation returns first)


def header_functions():
    text = open(os.path.join(ROOT, "include", "ga.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ga_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = ga.lib()
    names = header_functions()
    assert set(names) == set(ga.SYMBOLS)
    for name in names:
        assert hasattr(L, name), name


def P(x=FAKE):
    return ctypes.c_void_p(x)


def shape(B=2, H=2, n=100, d=64, dtype=ga.GA_BF16):
    return ga.Shape(B, H, n, d, dtype)


def call_forward(s, N=8, iters=2, scale=0.125, Q=FAKE, K=FAKE, V=FAKE, O=FAKE, belong=None, ws=FAKE,
                 ws_bytes=None):
    L = ga.lib()
    if ws_bytes is None:
        ws_bytes = max(L.ga_workspace_bytes(s, N), 1)
    return L.ga_forward(s, P(Q), P(K), P(V), N, iters, scale, P(O), None if belong is None else P(belong), None,
                        None, P(ws) if ws else None, ws_bytes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(s=shape(dtype=7)), 1),
    (dict(s=shape(B=-1)), 1),
    (dict(s=shape(n=0)), 1),
    (dict(s=shape(d=32)), 2),
    (dict(s=shape(), N=0), 1),
    (dict(s=shape(n=10), N=11), 1),
    (dict(s=shape(n=5000), N=1025), 1),
    (dict(s=shape(), iters=0), 1),
    (dict(s=shape(), scale=float("inf")), 1),
    (dict(s=shape(), scale=float("nan")), 1),
    (dict(s=shape(), Q=0), 1),
    (dict(s=shape(), K=FAKE + 4), 1),
    (dict(s=shape(), belong=FAKE + 8), 1),
    (dict(s=shape(), ws=0), 3),
    (dict(s=shape(), ws=FAKE + 16), 3),
    (dict(s=shape(), ws_bytes=1000), 3),
    (dict(s=shape(B=300, H=300)), 2),
    (dict(s=shape(n=1000), N=300), 2),  # bf16 attention keeps N <= 256 groups on chip
])
def test_forward_argument_errors(kw, status):
    rc = call_forward(**kw)
    assert rc == status, ga.lib().ga_last_error().decode()
    assert ga.lib().ga_last_error().decode() != ""
    assert ga.lib().ga_status_string(rc).decode() == ga.STATUS[status]


def call_forward_noalloc(s, N=8, iters=2, scale=0.125, Q=FAKE, K=FAKE, V=FAKE, O=FAKE, belong=None):
    return ga.lib().ga_forward_noalloc(s, P(Q), P(K), P(V), N, iters, scale, P(O),
                                       None if belong is None else P(belong), None, None, None)


@pytest.mark.parametrize("kw,status,msg", [
    (dict(s=shape(dtype=7)), 1, "dtype"),
    (dict(s=shape(n=10), N=11), 1, "N"),
    (dict(s=shape(), iters=0), 1, "iters"),
    (dict(s=shape(), scale=float("nan")), 1, "scale"),
    (dict(s=shape(), Q=0), 1, "Q"),
    (dict(s=shape(), belong=FAKE + 8), 1, "belong"),
    (dict(s=shape(d=32)), 2, ""),
    (dict(s=shape(dtype=ga.GA_F32)), 2, "bf16 only"),
    # 300 slices of 60000 keys need about 150 MB of scratch, beyond the 32 MiB array
    (dict(s=shape(B=300, H=1, n=60000), N=128), 3, "static scratch"),
])
def test_forward_noalloc_argument_errors(kw, status, msg):
    """ga_forward_noalloc checks everything it can on the host, before any HIP call."""
    rc = call_forward_noalloc(**kw)
    err = ga.lib().ga_last_error().decode()
    assert rc == status, err
    assert msg in err


def test_forward_noalloc_empty_batch_is_a_no_op():
    assert call_forward_noalloc(shape(B=0)) == 0


def test_empty_batch_is_a_no_op():
    assert call_forward(shape(B=0)) == 0
    assert call_forward(shape(H=0), ws=0) == 0


def test_other_entry_points_validate():
    L = ga.lib()
    s = shape()
    nb = L.ga_workspace_bytes(s, 8)
    assert L.ga_cluster(s, P(), 8, 0, None, P(), P(), P(), P(), nb, None) == 1          # iters
    assert L.ga_cluster(s, P(), 8, 3, P(FAKE + 4), P(), P(), P(), P(), nb, None) == 1   # init misaligned
    assert L.ga_cluster(s, P(), 8, 3, None, None, P(), P(), P(), nb, None) == 1          # belong NULL
    assert L.ga_cluster(s, P(), 8, 3, None, P(), P(), P(), P(), 10, None) == 3           # workspace
    assert L.ga_aggregate(s, P(), None, 8, P(), P(), nb, None) == 1
    assert L.ga_aggregate(shape(d=128), P(), P(), 8, P(), P(), nb, None) == 2
    assert L.ga_attend(s, P(), P(), P(), P(), 8, float("nan"), P(), P(), nb, None) == 1
    assert L.ga_attend(s, P(), P(), None, P(), 8, 1.0, P(), P(), nb, None) == 1
    assert L.ga_attend(shape(dtype=ga.GA_F32), P(), P(), P(), P(), 8, 1.0, P(), P(), 10, None) == 3


def test_workspace_bytes():
    L = ga.lib()
    assert L.ga_workspace_bytes(shape(d=32), 8) == 0
    assert L.ga_workspace_bytes(shape(), 0) == 0
    a = L.ga_workspace_bytes(shape(n=100), 8)
    b = L.ga_workspace_bytes(shape(n=200), 8)
    c = L.ga_workspace_bytes(shape(n=200), 64)
    assert 0 < a < b < c
    # the metric workload's workspace (about 112 MB, half of it the fused
    # update's per-partition sums) stays modest next to 288 GB of HBM
    big = L.ga_workspace_bytes(ga.Shape(16, 8, 8000, 64, ga.GA_BF16), 128)
    assert big < 256 * 2**20


def test_block_entry_points_validate():
    L = ga.lib()
    s = shape(B=2, H=8, n=300)
    nb = L.ga_block_workspace_bytes(s, 32)
    assert nb > 4 * 2 * 8 * 300 * 64 * 2  # Q, K, V, O plus the forward's workspace
    assert L.ga_block_workspace_bytes(shape(dtype=ga.GA_F32), 8) == 0
    assert L.ga_block_workspace_bytes(s, 0) == 0
    assert L.ga_project_qkv(shape(dtype=ga.GA_F32), P(), P(), P(), P(), P(), None) == 2
    assert L.ga_project_qkv(shape(d=32), P(), P(), P(), P(), P(), None) == 2
    assert L.ga_project_qkv(shape(H=65), P(), P(), P(), P(), P(), None) == 2
    assert L.ga_project_qkv(s, None, P(), P(), P(), P(), None) == 1
    assert L.ga_project_qkv(s, P(), P(FAKE + 2), P(), P(), P(), None) == 1
    assert L.ga_project_qkv(shape(B=0, H=8), P(), P(), P(), P(), P(), None) == 0
    assert L.ga_project_out(s, P(), None, P(), None) == 1
    assert L.ga_project_out(shape(n=0), P(), P(), P(), None) == 1
    assert L.ga_project_out(shape(B=0), P(), P(), P(), None) == 0
    blk = lambda s, N=32, iters=2, scale=0.125, ws=FAKE, nbytes=nb: L.ga_attention_block(
        s, P(), P(), P(), N, iters, scale, P(), P(ws) if ws else None, nbytes, None)
    assert blk(s, N=0) == 1
    assert blk(s, N=301) == 1
    assert blk(shape(B=2, H=8, n=1000), N=300) == 2
    assert blk(s, iters=0) == 1
    assert blk(s, scale=float("inf")) == 1
    assert blk(s, ws=0) == 3
    assert blk(s, ws=FAKE + 64) == 3
    assert blk(s, nbytes=nb - 1) == 3
    assert blk(shape(B=0, H=8), ws=0) == 0


def test_merge_plan_validates():
    L = ga.lib()
    s = shape(B=1, H=2, n=300)
    mp = lambda s=s, N=16, scale=0.125, eps=2.0, Q=FAKE, radius=FAKE: L.ga_merge_plan(
        s, P(Q), P(), P(), P(), P(), N, scale, eps, P(radius) if radius else None, P(), P(), P(), None)
    assert mp(eps=1.0) == 1
    assert mp(eps=0.5) == 1
    assert mp(eps=float("inf")) == 1
    assert mp(eps=float("nan")) == 1
    assert mp(scale=float("nan")) == 1
    assert mp(N=0) == 1
    assert mp(s=shape(n=1000), N=300) == 2
    assert mp(Q=0) == 1
    assert mp(radius=0) == 1
    assert mp(radius=FAKE + 8) == 1
    assert mp(s=shape(B=0)) == 0


def test_next_group_count_matches_the_definition(oracle_mod):
    import numpy as np

    L = ga.lib()
    rng = np.random.default_rng(0)
    for _ in range(300):
        N = int(rng.integers(1, 1025))
        m = rng.integers(0, N + 3, size=int(rng.integers(1, 40))).astype(np.int32)
        alpha = float(rng.choice([0.0, 1.0, rng.uniform()]))
        got = L.ga_next_group_count(N, m.ctypes.data_as(ctypes.c_void_p), m.size, alpha)
        assert got == oracle_mod.next_group_count(N, m, alpha), (N, m, alpha)
    assert L.ga_next_group_count(10, None, 0, 0.5) == 10
    assert L.ga_next_group_count(0, None, 0, 0.5) == 0
    assert L.ga_next_group_count(10, None, 0, 1.5) == 0
    assert L.ga_next_group_count(10, None, 3, 0.5) == 0
    assert ga.lib().ga_last_error().decode() != ""


def test_backward_validates():
    L = ga.lib()
    s = shape(B=1, H=2, n=300)
    nb = L.ga_backward_workspace_bytes(s, 64)
    assert nb > 0
    assert L.ga_backward_workspace_bytes(shape(dtype=ga.GA_F32), 8) == 0
    assert L.ga_backward_workspace_bytes(s, 257) == 0
    bw = lambda s=s, N=64, scale=0.125, dQ=FAKE, ws=FAKE, nbytes=nb: L.ga_backward(
        s, P(), P(), P(), P(), P(), P(), N, scale, P(dQ) if dQ else None, P(), P(), P(ws) if ws else None, nbytes,
        None)
    assert bw(s=shape(dtype=ga.GA_F32)) == 2
    assert bw(N=257) == 2
    assert bw(N=0) == 1
    assert bw(scale=float("inf")) == 1
    assert bw(dQ=0) == 1
    assert bw(ws=0) == 3
    assert bw(nbytes=nb - 1) == 3
    assert bw(s=shape(B=0)) == 0


# ---------------------------------------------------------------- binding checks
# ga.py refuses tensors the C ABI could not check (a host pointer, a wrong
# dtype or a short buffer would reach a kernel) before any library call.

def _cpu(shape, dtype=None):
    import torch

    return torch.zeros(shape, dtype=dtype or torch.bfloat16)


@pytest.mark.parametrize("call", ["forward", "cluster", "aggregate", "attend", "backward", "merge_plan",
                                  "project_qkv", "project_out", "attention_block"])
def test_binding_rejects_host_tensors(call):
    import torch

    B, H, n, N = 1, 2, 40, 4
    X = _cpu((B, H, n, 64))
    i32, f32 = torch.int32, torch.float32
    calls = {
        "forward": lambda: ga.forward(X, X, X, N, 2),
        "cluster": lambda: ga.cluster(X, N, 2),
        "aggregate": lambda: ga.aggregate(X, _cpu((B, H, n), i32), N),
        "attend": lambda: ga.attend(X, _cpu((B, H, N, 64), f32), _cpu((B, H, N), i32), _cpu((B, H, N, 64), f32), N),
        "backward": lambda: ga.backward(X, X, _cpu((B, H, n), i32), _cpu((B, H, N, 64), f32), _cpu((B, H, N), i32),
                                        _cpu((B, H, N, 64), f32), N),
        "merge_plan": lambda: ga.merge_plan(X, X, _cpu((B, H, n), i32), _cpu((B, H, N, 64), f32),
                                            _cpu((B, H, N), i32), N),
        "project_qkv": lambda: ga.project_qkv(_cpu((B, n, 128)), _cpu((384, 128)), 2),
        "project_out": lambda: ga.project_out(X, _cpu((128, 128))),
        "attention_block": lambda: ga.attention_block(_cpu((B, n, 128)), _cpu((384, 128)), _cpu((128, 128)), 2, N, 2),
    }
    with pytest.raises(ValueError, match="CUDA|cuda"):
        calls[call]()


def test_expect_checks_dtype_shape_and_device():
    import torch

    cpu = torch.device("cpu")
    t = torch.zeros((2, 3), dtype=torch.int32)
    with pytest.raises(ValueError, match="on cpu"):
        ga._expect(t, "x", cpu, torch.int32, (2, 3))  # not a CUDA tensor
    with pytest.raises(ValueError, match="required"):
        ga._expect(None, "x", cpu, torch.int32)
    ga._expect(None, "x", cpu, torch.int32, optional=True)
    with pytest.raises(ValueError, match="\\[B, H, n, d\\]"):
        ga.forward(torch.zeros((2, 3)), None, None, 2, 1)
