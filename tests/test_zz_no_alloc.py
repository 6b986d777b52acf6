"""The allocation-free forward (ga_forward_noalloc, static device scratch)
against the workspace forward (ga_forward) through the C ABI.

Both run the same kernels, so groups, counts and centroids must agree bit for
bit and the outputs too (the bf16 bar would be 2e-2 relative; the kernels are
deterministic, so equality is asserted).  Two calls in a row, the second on a
smaller input, check that what the first call leaves in the shared scratch
does not leak into the second.
"""
import ctypes

import pytest
import torch

from paper_2306_01926_amd import ga, inputs

pytestmark = pytest.mark.gpu


def say(msg):
    print(f"\n[case] {msg}", flush=True)


def qkv(B, H, n, seed, dev):
    w = inputs.WORKLOADS["n8000_N128_bf16"]
    Q, K, V = inputs.make_qkv(B, H, n, 64, "bf16", seed, w.M, w.sigma_lo, w.sigma_hi)
    return Q.to(dev), K.to(dev), V.to(dev)


def test_noalloc_matches_workspace_forward_on_two_calls():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    dev = torch.device("cuda:0")
    ga.lib()
    # first call: several workgroups per slice and a ragged key tail; second call smaller
    for B, H, n, N, seed in ((2, 4, 3001, 128, 11), (1, 3, 700, 40, 12)):
        say(f"ga_forward_noalloc B={B} H={H} n={n} N={N} seed={seed}")
        Q, K, V = qkv(B, H, n, seed, dev)
        O, bel, cnt, cen = ga.forward_noalloc(Q, K, V, N, 10, 0.125, return_groups=True)
        Ow, belw, cntw, cenw = ga.forward(Q, K, V, N, 10, 0.125, return_groups=True)
        torch.cuda.synchronize()
        assert torch.equal(bel, belw)
        assert torch.equal(cnt, cntw)
        assert torch.equal(cen.view(torch.int32), cenw.view(torch.int32))
        assert torch.equal(O.view(torch.int16), Ow.view(torch.int16))
        assert int(cnt.sum()) == B * H * n


def test_noalloc_internal_groups_and_rejections():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    dev = torch.device("cuda:0")
    say("ga_forward_noalloc without group outputs, then rejected shapes")
    Q, K, V = qkv(1, 2, 900, 21, dev)
    O = ga.forward_noalloc(Q, K, V, 64, 5, 0.125)
    Ow = ga.forward(Q, K, V, 64, 5, 0.125)
    torch.cuda.synchronize()
    assert torch.equal(O.view(torch.int16), Ow.view(torch.int16))
    L = ga.lib()
    P = ctypes.c_void_p
    p = P(Q.data_ptr())
    # N above the one-launch grouping's limit
    Q2, K2, V2 = qkv(1, 1, 600, 22, dev)
    with pytest.raises(ga.GAError, match="one-launch grouping"):
        ga.forward_noalloc(Q2, K2, V2, 200, 3, 0.125)
    # scratch beyond the static array: B*H = 300 slices of n = 60000 need far more than 32 MiB
    s = ga.Shape(300, 1, 60000, 64, ga.GA_BF16)
    rc = L.ga_forward_noalloc(s, p, p, p, 128, 3, 0.125, p, None, None, None, None)
    assert rc == 3 and b"static scratch" in L.ga_last_error()
    # fp32 is not served
    s = ga.Shape(1, 1, 600, 64, ga.GA_F32)
    rc = L.ga_forward_noalloc(s, p, p, p, 32, 3, 0.125, p, None, None, None, None)
    assert rc == 2 and b"bf16" in L.ga_last_error()
