"""GPU parity of the merge plan (adaptive group count, Section 5.1).

The grouping fed to both sides comes from the oracle (belong, count,
centroid), so the GPU and the CPU definition see identical inputs.  Bar:
bit-exact for everything: the fp64 radii and thresholds (same operations in
the same order, IEEE square roots), the partner indices and the merge counts.
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


def both(oracle_mod, dev, Q, K, N, iters, dtype, scale, eps):
    cl = oracle_mod.cluster(inputs.as_float64(K), N, iters, dtype)
    g = ga.merge_plan(Q.to(dev), K.to(dev), torch.from_numpy(cl["belong"]).to(dev),
                      torch.from_numpy(cl["centroid"]).to(dev), torch.from_numpy(cl["count"]).to(dev), N, scale, eps)
    torch.cuda.synchronize()
    ref = oracle_mod.merge_plan(inputs.as_float64(Q), inputs.as_float64(K), cl["belong"], cl["centroid"], cl["count"],
                                N, scale, eps)
    return {k: v.cpu().numpy() for k, v in g.items()}, ref


def assert_plan_equal(got, ref):
    assert np.array_equal(got["radius"].view(np.uint64), ref["radius"].view(np.uint64)), "radii differ"
    assert np.array_equal(got["dthr"].view(np.uint64), ref["dthr"].view(np.uint64)), "thresholds differ"
    assert np.array_equal(got["partner"], ref["partner"]), "partners differ"
    assert np.array_equal(got["merges"], ref["merges"]), "merge counts differ"


CASES = [
    # dtype, B, H, n, N, iters, M, sigma range, q scale, eps
    ("bf16", 1, 4, 1000, 64, 4, 24, (0.01, 0.05), 0.3, 1.5),
    ("bf16", 1, 2, 1000, 64, 4, 24, (0.01, 0.05), 0.3, 8.0),
    ("bf16", 2, 2, 777, 33, 3, 12, (0.02, 0.02), 0.2, 2.0),    # N odd: S1 one larger than S2
    ("bf16", 1, 1, 500, 1, 2, 4, (0.05, 0.05), 1.0, 2.0),      # one group: nothing to merge
    ("bf16", 1, 1, 300, 256, 2, 300, (0.05, 0.3), 1.0, 4.0),   # largest N, many tiny groups
    ("f32", 1, 2, 512, 32, 5, 32, (0.05, 0.05), 0.1, 2.0),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "-".join(map(str, c[:5])) + f"-eps{c[-1]}")
def test_merge_plan_bit_exact(oracle_mod, dev, case):
    dtype, B, H, n, N, iters, M, (lo, hi), qs, eps = case
    say(f"merge plan {case}")
    Q, K, _ = inputs.make_qkv(B, H, n, 64, dtype, 7, M, lo, hi)
    Q = inputs.to_storage(inputs.as_float64(Q).astype(np.float32) * qs, dtype)
    got, ref = both(oracle_mod, dev, Q, K, N, iters, dtype, 0.125, eps)
    assert_plan_equal(got, ref)


def test_merge_plan_zero_queries_give_infinite_threshold(oracle_mod, dev):
    say("merge plan with all-zero queries")
    _, K, _ = inputs.make_qkv(1, 1, 400, 64, "bf16", 3, 8, 0.05, 0.05)
    Q = torch.zeros_like(K)
    got, ref = both(oracle_mod, dev, Q, K, 16, 3, "bf16", 0.125, 2.0)
    assert_plan_equal(got, ref)
    assert np.isinf(got["dthr"]).all()
    assert got["merges"][0, 0] == 16 - 8  # every non-empty S2 group merges
    # ... provided all groups are non-empty, which the strided init on 8 tight clusters gives
    assert (ref["partner"][0, 0, 8:] >= 0).all()


def test_full_size_slices_and_the_group_count_update(oracle_mod, dev):
    w = inputs.WORKLOADS["n8000_N128_bf16"]
    say(f"merge plan on 3 full-size slices of {w.name}")
    Q, K, _ = inputs.make_qkv(1, 3, w.n, 64, "bf16", 0, w.M, w.sigma_lo, w.sigma_hi)
    got, ref = both(oracle_mod, dev, Q, K, w.N, w.iters, "bf16", 0.125, 2.0)
    assert_plan_equal(got, ref)
    assert ga.next_group_count(w.N, got["merges"], 0.5) == oracle_mod.next_group_count(w.N, ref["merges"], 0.5)


def test_scheduler_loop_on_the_gpu(dev):
    # forward, merge plan, next N, repeated: N never grows and stays >= 1
    say("scheduler loop: forward -> merge plan -> next N")
    Q, K, V = (t.to(dev) for t in inputs.make_qkv(1, 4, 2000, 64, "bf16", 5, 16, 0.01, 0.03))
    Q = Q * 0.25
    N = 128
    seen = [N]
    for _ in range(4):
        O, bel, cnt, cen = ga.forward(Q, K, V, N, 4, return_groups=True)
        plan = ga.merge_plan(Q, K, bel, cen, cnt, N, 0.125, 3.0)
        N = ga.next_group_count(N, plan["merges"], 0.5)
        seen.append(N)
    torch.cuda.synchronize()
    assert all(b <= a for a, b in zip(seen, seen[1:])) and seen[-1] >= 1
    assert seen[-1] < seen[0], f"no merge happened: {seen}"
