"""GPU parity of the attention block: projections around group attention.

Projections (ga_project_qkv, ga_project_out): the kernel accumulates the bf16
products in fp32 on the matrix cores and rounds once to bf16, so each output
is RNE_bf16(y^) with |y^ - y| <= g * sum_k |a_k w_k| for the exact dot product
y; the bar is |out - y| <= ulp_bf16/2 + g * sum_k |a_k w_k| with
g = 2 (D + 16) 2^-24 (twice the recursive-summation bound over D terms), and
nearly every output must equal the exactly rounded oracle value.

Whole block (ga_attention_block): within 2e-2 relative of the fp64 oracle
(per batch max |err| / max |ref| and per token ||err|| / ||ref||).  The
grouping inside sees keys that can differ from the oracle's by one bf16 step
where a projection lies next to a rounding boundary, so the block is compared
on its output only; the grouping itself is bit-exact given the same keys
(test_gpu_parity.py).
"""
import math

import numpy as np
import pytest
import torch

from paper_2306_01926_amd import ga, inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ga.lib()
    return torch.device("cuda:0")


def say(msg):
    print(f"\n[case] {msg}", flush=True)


def f64(t):
    return inputs.as_float64(t)


def ulp_bf16(x):
    return np.ldexp(1.0, np.frexp(np.abs(x))[1] - 8)


def check_projection(got, exact, absdot, D, oracle_mod):
    got = got.float().cpu().numpy().astype(np.float64)
    g = 2.0 * (D + 16) * 2.0 ** -24
    bound = 0.5 * ulp_bf16(np.maximum(np.abs(got), np.abs(exact))) + g * absdot
    err = np.abs(got - exact)
    assert np.all(err <= bound), f"{(err > bound).sum()} outputs outside the fp32-accumulation bound"
    same = (got == oracle_mod.round_bf16_f64(exact)).mean()
    assert same >= 0.99, f"only {same:.4f} of the outputs equal the exactly rounded product"
    return same


def heads(P, B, n, H):
    """[B, n, 3D] -> three [B, H, n, 64]."""
    h = P.reshape(B, n, 3, H, 64).transpose(2, 0, 3, 1, 4)
    return [h[i] for i in range(3)]


@pytest.mark.parametrize("B,n,H", [(2, 300, 8), (1, 77, 3), (3, 513, 1), (1, 256, 2)])
def test_project_qkv(oracle_mod, dev, B, n, H):
    say(f"project_qkv B={B} n={n} H={H}")
    X, Wqkv, _ = inputs.block_inputs(B, n, H, seed=1)
    Q, K, V = ga.project_qkv(X.to(dev), Wqkv.to(dev), H)
    torch.cuda.synchronize()
    x, w = f64(X), f64(Wqkv)
    exact = heads(x @ w.T, B, n, H)
    absdot = heads(np.abs(x) @ np.abs(w).T, B, n, H)
    for got, e, a in zip((Q, K, V), exact, absdot):
        check_projection(got, e, a, 64 * H, oracle_mod)


@pytest.mark.parametrize("B,n,H", [(2, 300, 8), (1, 77, 3), (2, 1000, 1)])
def test_project_out(oracle_mod, dev, B, n, H):
    say(f"project_out B={B} n={n} H={H}")
    rng = np.random.default_rng(2)
    O = inputs.to_storage(rng.standard_normal((B, H, n, 64)).astype(np.float32), "bf16")
    _, _, Wo = inputs.block_inputs(1, 8, H, seed=3)
    Y = ga.project_out(O.to(dev), Wo.to(dev))
    torch.cuda.synchronize()
    cat = f64(O).transpose(0, 2, 1, 3).reshape(B, n, 64 * H)
    w = f64(Wo)
    check_projection(Y, cat @ w.T, np.abs(cat) @ np.abs(w).T, 64 * H, oracle_mod)


def check_block(Y, Yref, tol=2e-2):
    Yg = Y.float().cpu().numpy().astype(np.float64)
    worst = 0.0
    for b in range(Yref.shape[0]):
        r = np.abs(Yg[b] - Yref[b]).max() / np.abs(Yref[b]).max()
        worst = max(worst, r)
        assert r <= tol, f"batch {b}: max relative error {r:.3g}"
        rows = np.linalg.norm(Yg[b] - Yref[b], axis=-1) / np.linalg.norm(Yref[b], axis=-1)
        assert rows.max() <= tol, f"batch {b}: {(rows > tol).sum()} tokens above {tol}"
    return worst


@pytest.mark.parametrize("B,n,H,N,iters", [(2, 700, 4, 32, 4), (1, 300, 8, 16, 3), (1, 96, 2, 96, 2)])
def test_attention_block_matches_oracle(oracle_mod, dev, B, n, H, N, iters):
    say(f"attention_block B={B} n={n} H={H} N={N} iters={iters}")
    X, Wqkv, Wo = inputs.block_inputs(B, n, H, seed=5)
    Y = ga.attention_block(X.to(dev), Wqkv.to(dev), Wo.to(dev), H, N, iters)
    torch.cuda.synchronize()
    ref = oracle_mod.attention_block(f64(X), f64(Wqkv), f64(Wo), H, N, iters, 0.125)
    check_block(Y, ref["Y"])


def test_block_is_its_steps_composed(dev):
    B, n, H, N, iters = 2, 500, 4, 24, 3
    say(f"attention_block vs its steps B={B} n={n} H={H} N={N}")
    X, Wqkv, Wo = (t.to(dev) for t in inputs.block_inputs(B, n, H, seed=6))
    Y = ga.attention_block(X, Wqkv, Wo, H, N, iters)
    Q, K, V = ga.project_qkv(X, Wqkv, H)
    O = ga.forward(Q, K, V, N, iters, 0.125)
    Y2 = ga.project_out(O, Wo)
    torch.cuda.synchronize()
    assert torch.equal(Y, Y2)


def test_full_size_encoder_sampled_batches(oracle_mod, dev):
    w = inputs.BLOCK_WORKLOADS["encoder_n4000_N128_bf16"]
    say(f"full size {w.name} (B={w.B} n={w.n} H={w.H} N={w.N}), batches 0 and {w.B - 1} against the oracle")
    X, Wqkv, Wo = inputs.block_inputs(w.B, w.n, w.H, seed=0)
    Y = ga.attention_block(X.to(dev), Wqkv.to(dev), Wo.to(dev), w.H, w.N, w.iters)
    torch.cuda.synchronize()
    for b in (0, w.B - 1):
        ref = oracle_mod.attention_block(f64(X[b:b + 1]), f64(Wqkv), f64(Wo), w.H, w.N, w.iters, 0.125)
        check_block(Y[b:b + 1], ref["Y"])
