"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bars: group assignments, counts and fp32 centroids bit-exact; value sums equal
to the fp32 rounding of the oracle's fp64 sums; outputs within 1e-4 (fp32) or
2e-2 (bf16) relative, both per (b, h) slice (max |err| / max |ref|) and per
row (||err_i|| / ||ref_i||).
"""
import math

import numpy as np
import pytest
import torch

from paper_2306_01926_amd import ga, inputs

pytestmark = pytest.mark.gpu
TOL = {"f32": 1e-4, "bf16": 2e-2}


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ga.lib()
    return torch.device("cuda:0")


@pytest.fixture(params=["persistent", "rounds"])
def path(request, monkeypatch):
    """The grouping path under test: the persistent kernel (every round in one
    launch; the default where it applies) or one launch per round (the
    GA_GROUPING=rounds switch of the library)."""
    if request.param == "rounds":
        monkeypatch.setenv("GA_GROUPING", "rounds")
    else:
        monkeypatch.delenv("GA_GROUPING", raising=False)
    return request.param


def uses_persistent(path, dtype, N):
    return path == "persistent" and dtype == "bf16" and N <= 128


def say(msg):
    print(f"\n[case] {msg}", flush=True)


def f64(t):
    return inputs.as_float64(t)


def check_close(O_gpu, O_ref, tol):
    Og = O_gpu.float().cpu().numpy().astype(np.float64)
    err = np.abs(Og - O_ref)
    B, H = O_ref.shape[:2]
    worst = 0.0
    for b in range(B):
        for h in range(H):
            den = np.abs(O_ref[b, h]).max()
            r = err[b, h].max() / den if den > 0 else err[b, h].max()
            worst = max(worst, r)
            assert r <= tol, f"slice ({b},{h}) max relative error {r:.3g} > {tol}"
    rn = np.linalg.norm(O_ref, axis=-1)
    en = np.linalg.norm(Og - O_ref, axis=-1)
    scale = np.abs(O_ref).max()
    bad = en > tol * np.where(rn > 0, rn, scale)
    assert not bad.any(), f"{bad.sum()} rows exceed relative error {tol}"
    return worst


def cluster_both(oracle_mod, K, N, iters, dtype, dev, init=None, trace=False):
    Kd = K.to(dev)
    bel, cnt, cen = ga.cluster(Kd, N, iters, init=None if init is None else init.to(dev))
    torch.cuda.synchronize()
    ga.workspace_check(Kd, N)
    ref = oracle_mod.cluster(f64(K), N, iters, dtype, init=None if init is None else init.numpy(), trace=trace)
    return (bel.cpu().numpy(), cnt.cpu().numpy(), cen.cpu().numpy()), ref


def assert_groups_equal(got, ref):
    bel, cnt, cen = got
    mism = (bel != ref["belong"]).sum()
    assert mism == 0, f"{mism} assignments differ"
    assert np.array_equal(cnt, ref["count"]), "counts differ"
    assert np.array_equal(cen.view(np.uint32), ref["centroid"].view(np.uint32)), "centroids differ"


CLUSTER_CASES = [
    # dtype, B, H, n, N, iters, M (mixture components), sigma range
    ("bf16", 1, 2, 300, 16, 3, 12, (0.05, 0.3)),
    ("bf16", 2, 2, 1000, 64, 5, 64, (0.05, 0.3)),
    ("bf16", 1, 1, 97, 32, 4, 8, (0.1, 0.1)),        # ragged tail, n < 4 tiles
    ("bf16", 1, 2, 31, 31, 2, 4, (0.3, 0.3)),        # N = n < 32
    ("bf16", 1, 1, 64, 64, 2, 8, (0.2, 0.2)),        # N = n, full tiles
    ("bf16", 1, 1, 600, 1, 2, 8, (0.2, 0.2)),        # one group
    ("bf16", 1, 1, 2000, 256, 3, 256, (0.05, 0.3)),
    ("bf16", 1, 1, 1500, 1024, 2, 256, (0.05, 0.3)), # largest N
    ("bf16", 1, 1, 4000, 100, 4, 300, (0.3, 0.3)),   # N not a multiple of 32, heavy overlap
    ("bf16", 1, 2, 700, 50, 4, 64, (0.05, 0.3)),    # 3 ranks per slice on the one-launch path
    ("bf16", 1, 1, 1200, 70, 4, 96, (0.05, 0.3)),   # 5 ranks
    ("bf16", 1, 1, 1700, 128, 4, 160, (0.05, 0.3)), # 7 ranks, N = 128
    ("f32", 1, 1, 512, 32, 5, 32, (0.05, 0.05)),     # the fp32 workload at full size
    ("f32", 1, 2, 200, 20, 4, 30, (0.05, 0.3)),
    ("f32", 1, 1, 130, 130, 2, 8, (0.1, 0.1)),
]


@pytest.mark.parametrize("case", CLUSTER_CASES, ids=lambda c: "-".join(map(str, c[:6])))
def test_cluster_bit_exact(oracle_mod, dev, case, path):
    dtype, B, H, n, N, iters, M, (slo, shi) = case
    say(f"cluster {case}")
    _, K, _ = inputs.make_qkv(B, H, n, 64, dtype, 1000 + n + N, M, slo, shi)
    got, ref = cluster_both(oracle_mod, K, N, iters, dtype, dev)
    assert_groups_equal(got, ref)


def test_cluster_fixed_point_ends_early(oracle_mod, dev, path):
    """Well separated clusters reach a fixed point (no key changes group) in
    round 5 or 6 of 12 (each slice its own); the persistent kernel stops a
    slice there.
    Groups, counts, centroids and the forward's output must still equal the
    oracle's 12 full rounds."""
    say(f"cluster: fixed point before the last round ({path})")
    Q, K, V = inputs.make_qkv(1, 3, 2500, 64, "bf16", 79, 32, 0.01, 0.01)
    got, ref = cluster_both(oracle_mod, K, 32, 12, "bf16", dev, trace=True)
    tb = ref["trace_belong"]  # [iters, B, H, n]
    for h in range(3):
        same = [bool(np.array_equal(tb[t, 0, h], tb[t - 1, 0, h])) for t in range(1, 12)]
        assert any(same[:9]), f"slice {h} reaches no fixed point before round 10: the case does not test the exit"
    assert_groups_equal(got, ref)
    O, bel, cnt, cen = ga.forward(Q.to(dev), K.to(dev), V.to(dev), 32, 12, 0.125, return_groups=True)
    torch.cuda.synchronize()
    fref = oracle_mod.forward(f64(Q), f64(K), f64(V), 32, 12, 0.125, "bf16")
    assert_groups_equal((bel.cpu().numpy(), cnt.cpu().numpy(), cen.cpu().numpy()), fref)
    check_close(O, fref["O"], TOL["bf16"])


EXACT_ALL_CASES = [
    # B, H, n, N, iters: ranks per slice 8 (n = 2000), 4 and 16 (the last with
    # N not a multiple of 32) on the one-launch path
    (1, 2, 2000, 64, 4),
    (2, 2, 1000, 128, 3),
    (1, 1, 4000, 100, 3),
]


@pytest.mark.parametrize("case", EXACT_ALL_CASES, ids=lambda c: "-".join(map(str, c)))
def test_cluster_exact_decision_for_every_key(oracle_mod, dev, case, path, monkeypatch):
    """With the certification bound widened 65536 times (GA_CERT_WIDEN) the
    MFMA scores certify almost no key, so nearly every key of every round
    takes the exact fp64 decision (and, after the first round, adds its own
    row if it moves, beside the sums of the few certain moved keys).  The
    groups, counts and centroids must still equal the oracle's bit for bit."""
    B, H, n, N, iters = case
    monkeypatch.setenv("GA_CERT_WIDEN", "65536")
    say(f"cluster, exact decision for every key: {case} ({path})")
    _, K, _ = inputs.make_qkv(B, H, n, 64, "bf16", 300 + n + N, max(8, N), 0.05, 0.3)
    got, ref = cluster_both(oracle_mod, K, N, iters, "bf16", dev)
    assert_groups_equal(got, ref)


def test_cluster_with_caller_init(oracle_mod, dev):
    say("cluster with caller init")
    _, K, _ = inputs.make_qkv(2, 1, 700, 64, "bf16", 5, 40, 0.05, 0.3)
    init = torch.from_numpy(np.random.default_rng(0).standard_normal((2, 1, 40, 64)).astype(np.float32) * 0.2)
    got, ref = cluster_both(oracle_mod, K, 40, 3, "bf16", dev, init=init)
    assert_groups_equal(got, ref)


def emptying_group_case(N=3, active=(0, 1, 2)):
    """Keys on the first axis: -1 x2, -0.5625 x18, -0.375, +0.3125, +0.5625 x18,
    +1 x2 (exact in bf16); caller init -1, 0, +1 for the groups `active`
    (any other group starts far away on its own axis and never gets a key).
    Round 1 gives the middle group the keys at -0.375 and +0.3125 (its
    centroid becomes -0.03125); the update moves the outer groups to -0.60625
    and +0.60625, so in round 2 both keys leave and the middle group is empty
    from then on, keeping -0.03125 (neither its initial value nor zero)."""
    xs = [-1.0] * 2 + [-0.5625] * 18 + [-0.375, 0.3125] + [0.5625] * 18 + [1.0] * 2
    K = np.zeros((1, 1, len(xs), 64), np.float32)
    K[0, 0, :, 0] = xs
    init = np.zeros((1, 1, N, 64), np.float32)
    for j in range(N):
        init[0, 0, j, 1 + j % 63] = 8.0  # far from every key
    for j, x in zip(active, (-1.0, 0.0, 1.0)):
        init[0, 0, j] = 0.0
        init[0, 0, j, 0] = x
    return inputs.to_storage(K, "bf16"), torch.from_numpy(init)


@pytest.mark.parametrize("N,active", [(3, (0, 1, 2)), (40, (0, 33, 39))], ids=["N3", "N40-block1"])
def test_cluster_group_empties_in_a_later_round(oracle_mod, dev, N, active):
    say(f"cluster: a group loses every member in round 2 (N={N}, groups {active})")
    K, init = emptying_group_case(N, active)
    mid = active[1]
    ref = oracle_mod.cluster(f64(K), N, 4, "bf16", init=init.numpy(), trace=True)
    counts = [np.bincount(b.ravel(), minlength=N)[mid] for b in ref["trace_belong"]]
    assert counts[0] == 2 and all(c == 0 for c in counts[1:]), counts  # the case does what it says
    got, ref = cluster_both(oracle_mod, K, N, 4, "bf16", dev, init=init)
    assert_groups_equal(got, ref)
    assert got[2][0, 0, mid, 0] == np.float32(-0.03125) and got[1][0, 0, mid] == 0


def test_cluster_stepwise_against_trace(oracle_mod, dev):
    """Round t fed the oracle's C^(t-1): isolates each round from earlier ones."""
    say("stepwise cluster rounds")
    _, K, _ = inputs.make_qkv(2, 2, 2000, 64, "bf16", 7, 128, 0.05, 0.3)
    T = 6
    ref = oracle_mod.cluster(f64(K), 128, T, "bf16", trace=True)
    Kd = K.to(dev)
    n, N = 2000, 128
    prev = np.ascontiguousarray(f64(K)[:, :, (np.arange(N) * n) // N, :].astype(np.float32))
    for t in range(T):
        bel, cnt, cen = ga.cluster(Kd, N, 1, init=torch.from_numpy(prev).to(dev))
        torch.cuda.synchronize()
        assert np.array_equal(bel.cpu().numpy(), ref["trace_belong"][t]), f"round {t}"
        assert np.array_equal(cen.cpu().numpy().view(np.uint32), ref["trace_centroid"][t].view(np.uint32))
        prev = ref["trace_centroid"][t]


# One slice, so every workgroup of the first round covers 4 tiles of 32 keys:
# n keys make ceil(ceil(n / 32) / 4) partitions of the first round's fused
# update, 1 to 8, then 9 (too many: the separate update runs instead).
PARTITION_CASES = [
    # n, N, partitions
    (100, 20, 1), (200, 50, 2), (380, 90, 3), (500, 128, 4), (620, 33, 5),
    (750, 64, 6), (890, 100, 7), (1000, 127, 8), (1030, 128, 9),
]


@pytest.mark.parametrize("case", PARTITION_CASES, ids=lambda c: "-".join(map(str, c)))
def test_first_round_partitions(oracle_mod, dev, case, monkeypatch):
    n, N, parts = case
    monkeypatch.setenv("GA_GROUPING", "rounds")  # the launch-per-round path's first round
    say(f"first-round partitions n={n} N={N} parts={parts}")
    _, K, _ = inputs.make_qkv(1, 1, n, 64, "bf16", 40 + n, max(4, N // 2), 0.05, 0.3)
    ga.timing_enable(True)
    try:
        got, ref = cluster_both(oracle_mod, K, N, 2, "bf16", dev)
    finally:
        ga.timing_enable(False)
        launches = ga.timing_collect()
    assert_groups_equal(got, ref)
    assert ("part_finish" in launches) == (parts <= 8), sorted(launches)


@pytest.mark.parametrize("n", [700, 3000])
def test_cluster_single_round_with_caller_init(oracle_mod, dev, n):
    """One round only: the fused first round (n = 700) and the separate update (n = 3000)."""
    say(f"single round with caller init n={n}")
    _, K, _ = inputs.make_qkv(1, 2, n, 64, "bf16", 6, 60, 0.05, 0.3)
    init = torch.from_numpy(np.random.default_rng(n).standard_normal((1, 2, 96, 64)).astype(np.float32) * 0.2)
    got, ref = cluster_both(oracle_mod, K, 96, 1, "bf16", dev, init=init)
    assert_groups_equal(got, ref)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_aggregate_bit_exact(oracle_mod, dev, dtype):
    say(f"aggregate {dtype}")
    rng = np.random.default_rng(3)
    B, H, n, N = 2, 3, 1500, 70
    _, _, V = inputs.make_qkv(B, H, n, 64, dtype, 9, 8, 0.1, 0.1)
    belong = rng.integers(0, N - 3, size=(B, H, n)).astype(np.int32)
    belong[0, 0, 5] = -1       # ignored
    belong[1, 2, 7] = N        # ignored
    vs = ga.aggregate(V.to(dev), torch.from_numpy(belong).to(dev), N)
    torch.cuda.synchronize()
    ref, _ = oracle_mod.aggregate(f64(V), belong, N)
    assert np.array_equal(vs.cpu().numpy().view(np.uint32), ref.astype(np.float32).view(np.uint32))


ATTEND_CASES = [
    ("bf16", 2, 2, 1000, 64, 0.125),
    ("bf16", 1, 2, 97, 33, 0.125),     # ragged tiles, partial group block
    ("bf16", 1, 1, 3000, 256, 0.125),
    ("bf16", 1, 2, 500, 40, -0.3),     # negative scale
    ("bf16", 1, 1, 300, 20, 0.0),      # zero scale: o_i = mean of values
    ("bf16", 1, 1, 400, 50, 2.0),      # sharp softmax
    ("f32", 1, 1, 512, 32, 0.125),
    ("f32", 2, 1, 333, 100, -0.7),
]


@pytest.mark.parametrize("case", ATTEND_CASES, ids=lambda c: "-".join(map(str, c)))
def test_attend_given_groups(oracle_mod, dev, case):
    """Random groupings with empty groups and non-representable centroids."""
    dtype, B, H, n, N, scale = case
    say(f"attend {case}")
    rng = np.random.default_rng(n + N)
    Q, _, V = inputs.make_qkv(B, H, n, 64, dtype, 11, 8, 0.1, 0.1)
    belong = rng.integers(0, max(N - 5, 1), size=(B, H, n)).astype(np.int32)   # last groups empty
    count = np.stack([[np.bincount(belong[b, h], minlength=N) for h in range(H)] for b in range(B)]).astype(np.int32)
    centroid = (0.3 * rng.standard_normal((B, H, N, 64))).astype(np.float32)
    vsum, _ = oracle_mod.aggregate(f64(V), belong, N)
    vsum32 = vsum.astype(np.float32)
    O = ga.attend(Q.to(dev), torch.from_numpy(centroid).to(dev), torch.from_numpy(count).to(dev),
                  torch.from_numpy(vsum32).to(dev), N, scale)
    torch.cuda.synchronize()
    ref = oracle_mod.attend(f64(Q), centroid, count, vsum32, N, scale, dtype)
    check_close(O, ref, TOL[dtype])


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_attend_all_groups_empty_gives_zeros(dev, dtype):
    say(f"attend all-empty {dtype}")
    Q, _, _ = inputs.make_qkv(1, 2, 100, 64, dtype, 1, 4, 0.1, 0.1)
    N = 8
    count = torch.zeros((1, 2, N), dtype=torch.int32)
    count[0, 1, 3] = 100
    cen = torch.randn(1, 2, N, 64)
    vs = torch.randn(1, 2, N, 64)
    O = ga.attend(Q.to(dev), cen.to(dev), count.to(dev), vs.to(dev), N, 0.125)
    torch.cuda.synchronize()
    O = O.float().cpu()
    assert (O[0, 0] == 0).all()
    want = (vs[0, 1, 3] / 100).to(Q.dtype).float()
    assert torch.allclose(O[0, 1], want.expand(100, 64), rtol=TOL[dtype], atol=1e-6)


FORWARD_CASES = [
    ("bf16", 2, 2, 1200, 64, 4),
    ("bf16", 1, 3, 555, 50, 3),
    ("bf16", 1, 1, 96, 96, 2),      # N = n: exact attention
    ("f32", 1, 1, 512, 32, 5),      # the fp32 workload at full size
    ("f32", 1, 2, 100, 100, 2),     # N = n
]


@pytest.mark.parametrize("case", FORWARD_CASES, ids=lambda c: "-".join(map(str, c)))
def test_forward_end_to_end(oracle_mod, dev, case, path):
    dtype, B, H, n, N, iters = case
    say(f"forward {case} ({path})")
    M = max(4, N // 2)
    Q, K, V = inputs.make_qkv(B, H, n, 64, dtype, 21 + n, M, 0.05, 0.3)
    Qd = Q.to(dev)
    ga.timing_enable(True)
    O, bel, cnt, cen = ga.forward(Qd, K.to(dev), V.to(dev), N, iters, return_groups=True)
    torch.cuda.synchronize()
    ga.timing_enable(False)
    launches = ga.timing_collect()
    ga.workspace_check(Qd, N)
    assert ("lloyd" in launches) == uses_persistent(path, dtype, N), sorted(launches)
    ref = oracle_mod.forward(f64(Q), f64(K), f64(V), N, iters, 1 / 8, dtype)
    assert_groups_equal((bel.cpu().numpy(), cnt.cpu().numpy(), cen.cpu().numpy()), ref)
    check_close(O, ref["O"], TOL[dtype])
    if N == n:  # every key its own group: Eq. 1 exactly
        Qd, Kd, Vd = f64(Q), f64(K), f64(V)
        P = np.einsum("bhid,bhjd->bhij", Qd, Kd) / 8
        A = np.exp(P - P.max(-1, keepdims=True))
        A /= A.sum(-1, keepdims=True)
        check_close(O, np.einsum("bhij,bhjd->bhid", A, Vd), TOL[dtype])


def test_forward_is_deterministic(dev):
    say("determinism")
    Q, K, V = inputs.make_qkv(2, 2, 3000, 64, "bf16", 3, 128, 0.05, 0.3)
    Qd, Kd, Vd = Q.to(dev), K.to(dev), V.to(dev)
    a = ga.forward(Qd, Kd, Vd, 128, 6, return_groups=True)
    b = ga.forward(Qd, Kd, Vd, 128, 6, return_groups=True)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x.view(torch.uint8) if x.dtype == torch.bfloat16 else x,
                           y.view(torch.uint8) if y.dtype == torch.bfloat16 else y)


def test_forward_single_round(oracle_mod, dev):
    say("forward, one grouping round")
    Q, K, V = inputs.make_qkv(2, 1, 900, 64, "bf16", 17, 50, 0.05, 0.3)
    O, bel, cnt, cen = ga.forward(Q.to(dev), K.to(dev), V.to(dev), 80, 1, return_groups=True)
    torch.cuda.synchronize()
    ref = oracle_mod.forward(f64(Q), f64(K), f64(V), 80, 1, 1 / 8, "bf16")
    assert_groups_equal((bel.cpu().numpy(), cnt.cpu().numpy(), cen.cpu().numpy()), ref)
    check_close(O, ref["O"], TOL["bf16"])


@pytest.mark.parametrize("explicit_ws", [True, False], ids=["ws", "cached-ws"])
def test_concurrent_forwards_separate_workspaces(dev, explicit_ws):
    """Two forwards overlapping on two streams, each with its own workspace
    (given, or the binding's cached one, which is kept per device and stream),
    give the results of the same forwards run one after the other."""
    say(f"concurrent forwards on two streams (explicit workspaces: {explicit_ws})")
    args = [(inputs.make_qkv(2, 2, 2500, 64, "bf16", s, 128, 0.05, 0.3), N) for s, N in ((31, 128), (32, 100))]
    args = [(tuple(t.to(dev) for t in qkv), N) for qkv, N in args]
    seq = [ga.forward(*qkv, N, 5, return_groups=True) for qkv, N in args]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(dev) for _ in args]
    wss = [torch.empty(ga.workspace_bytes(ga.shape_of(qkv[0]), N), dtype=torch.uint8, device=dev)
           for qkv, N in args]
    outs = [None, None]
    for r in range(3):
        for i, ((qkv, N), s) in enumerate(zip(args, streams)):
            s.wait_stream(torch.cuda.current_stream(dev))
            with torch.cuda.stream(s):
                outs[i] = ga.forward(*qkv, N, 5, return_groups=True, ws=wss[i] if explicit_ws else None)
        torch.cuda.synchronize()
        for a, b in zip(seq, outs):
            for x, y in zip(a, b):
                assert torch.equal(x.view(torch.uint8) if x.dtype == torch.bfloat16 else x,
                                   y.view(torch.uint8) if y.dtype == torch.bfloat16 else y), f"repeat {r}"


def _sampled_full_size(oracle_mod, dev, w, seed, N, slices, queries=512):
    """Full-size forward; oracle on a few (b, h) slices (assignments) and sampled queries."""
    Q, K, V = inputs.workload_inputs(w, seed)
    O, bel, cnt, cen = ga.forward(Q.to(dev), K.to(dev), V.to(dev), N, w.iters, return_groups=True)
    torch.cuda.synchronize()
    O, bel, cnt, cen = O.cpu(), bel.cpu().numpy(), cnt.cpu().numpy(), cen.cpu().numpy()
    rng = np.random.default_rng(seed)
    for (b, h) in slices:
        Ks = f64(K[b:b + 1, h:h + 1])
        ref = oracle_mod.cluster(Ks, N, w.iters, w.dtype)
        assert_groups_equal((bel[b:b + 1, h:h + 1], cnt[b:b + 1, h:h + 1], cen[b:b + 1, h:h + 1]), ref)
        vsum, _ = oracle_mod.aggregate(f64(V[b:b + 1, h:h + 1]), ref["belong"], N)
        qi = np.sort(rng.choice(w.n, size=queries, replace=False))
        Oref = oracle_mod.attend(f64(Q[b:b + 1, h:h + 1, qi]), ref["centroid"], ref["count"], vsum, N,
                                 1 / math.sqrt(w.d), w.dtype)
        check_close(O[b:b + 1, h:h + 1, qi], Oref, TOL[w.dtype])


def test_full_size_n2000_all_slices(oracle_mod, dev):
    w = inputs.WORKLOADS["n2000_N64_bf16"]
    say(f"full size {w.name}, every slice")
    Q, K, V = inputs.workload_inputs(w, 0)
    O, bel, cnt, cen = ga.forward(Q.to(dev), K.to(dev), V.to(dev), w.N, w.iters, return_groups=True)
    torch.cuda.synchronize()
    ref = oracle_mod.forward(f64(Q), f64(K), f64(V), w.N, w.iters, 1 / 8, w.dtype)
    assert_groups_equal((bel.cpu().numpy(), cnt.cpu().numpy(), cen.cpu().numpy()), ref)
    check_close(O, ref["O"], TOL[w.dtype])


def test_full_size_n8000_sampled_slices(oracle_mod, dev):
    w = inputs.WORKLOADS["n8000_N128_bf16"]
    say(f"full size {w.name}, sampled slices")
    _sampled_full_size(oracle_mod, dev, w, 0, w.N, [(0, 0), (7, 3), (15, 7)])


@pytest.mark.parametrize("N", [32, 64])
def test_full_size_n20000_small_group_counts(oracle_mod, dev, N):
    """The two smaller group counts of the n = 20000 workload (the draws of
    the varying-N test give 256 and 128) at full size."""
    w = inputs.WORKLOADS["n20000_Nvar_bf16"]
    say(f"full size {w.name}, N={N}")
    _sampled_full_size(oracle_mod, dev, w, 2 + N, N, [(1, 2), (2, 5)], queries=256)


def test_full_size_n20000_varying_groups(oracle_mod, dev):
    w = inputs.WORKLOADS["n20000_Nvar_bf16"]
    for call in range(2):
        N = inputs.draw_group_count(w, 0, call)
        say(f"full size {w.name}, call {call}, N={N}")
        _sampled_full_size(oracle_mod, dev, w, call, N, [(0, 0), (3, 7)], queries=256)
