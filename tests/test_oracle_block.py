"""Pins for the oracle of the attention block (projections around group attention).

The block is the RITA encoder's attention (Section 3: a Transformer encoder
whose self-attention is group attention) with the bias-free projections of
Eq. 1.  None of these re-types the oracle's formulas; they use:
  * the bf16 format itself (torch's float32 -> bf16 conversion, and a value
    whose correct single rounding differs from rounding through float32);
  * a closed form: with W_Q = 0 every score is 0, so group attention returns
    the mean of the values for every query whatever the grouping, and with
    permutation matrices for W_V and W_O the block output is a column
    permutation of the per-batch token mean of X;
  * exact multi-head softmax attention (Eq. 1) when every key is its own
    group (N = n);
  * invariance of the output under a relabelling of the heads.
"""
import numpy as np
import pytest
import torch

from paper_2306_01926_amd import inputs


def f64(t):
    return inputs.as_float64(t)


def test_round_bf16_f64_is_one_correct_rounding(oracle_mod):
    rng = np.random.default_rng(3)
    x = (rng.standard_normal(20000) * np.exp(rng.uniform(-20, 20, 20000))).astype(np.float32)
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(oracle_mod.round_bf16_f64(x.astype(np.float64)), want)
    # 1 + 2^-8 is the midpoint between bf16 1 and 1 + 2^-7: just above it the
    # correct rounding goes up, while rounding through float32 first would land
    # on the midpoint and then tie to even (down)
    above = 1.0 + 2.0 ** -8 + 2.0 ** -30
    assert oracle_mod.round_bf16_f64(np.array([above]))[0] == 1.0 + 2.0 ** -7
    assert oracle_mod.round_bf16_f64(np.array([1.0 + 2.0 ** -8]))[0] == 1.0
    assert oracle_mod.round_bf16_f64(np.array([1.0 + 3 * 2.0 ** -8]))[0] == 1.0 + 2.0 ** -6
    assert oracle_mod.round_bf16_f64(np.array([0.0, -0.0]))[0] == 0.0


def perm_matrix(p):
    D = len(p)
    W = np.zeros((D, D))
    W[np.arange(D), p] = 1.0  # row o picks input p[o]
    return W


@pytest.mark.parametrize("H,N,iters", [(2, 5, 2), (3, 1, 1)])
def test_zero_queries_give_permuted_token_mean(oracle_mod, H, N, iters):
    B, n = 2, 40
    D = 64 * H
    X, _, _ = inputs.block_inputs(B, n, H, seed=11)
    X = f64(X)
    rng = np.random.default_rng(5)
    pv, po = rng.permutation(D), rng.permutation(D)
    Wk = np.asarray(inputs.to_storage(rng.standard_normal((D, D)).astype(np.float32) / 8, "bf16").double())
    Wqkv = np.concatenate([np.zeros((D, D)), Wk, perm_matrix(pv)])
    r = oracle_mod.attention_block(X, Wqkv, perm_matrix(po), H, N, iters, 0.125)
    # V = X[:, :, pv] exactly; O = mean over tokens of V; Y[..., o] = O[..., po[o]]
    mean = X.mean(axis=1)  # [B, D]
    want = oracle_mod.round_bf16_f64(mean[:, pv][:, po])
    for t in range(n):
        assert np.array_equal(r["Y"][:, t, :], want), t


def mha_exact(X, Wqkv, Wo, H, scale, rnd):
    """Eq. 1 multi-head softmax attention with bf16 storage between the steps,
    written per head on the column-per-feature weights W_Q = Wqkv[:D].T etc."""
    B, n, D = X.shape
    WQ, WK, WV = (Wqkv[i * D:(i + 1) * D].T for i in range(3))  # [D_in, D_out]
    WO = Wo.T
    Y = np.zeros((B, n, D))
    for b in range(B):
        heads = []
        for h in range(H):
            cols = slice(64 * h, 64 * h + 64)
            q, k, v = (rnd(X[b] @ W[:, cols]) for W in (WQ, WK, WV))
            s = scale * q @ k.T
            a = np.exp(s - s.max(axis=1, keepdims=True))
            heads.append(rnd((a / a.sum(axis=1, keepdims=True)) @ v))
        Y[b] = np.concatenate(heads, axis=1) @ WO
    return rnd(Y)


def test_every_key_its_own_group_is_exact_multihead_attention(oracle_mod):
    B, n, H = 2, 48, 2
    X, Wqkv, Wo = (f64(t) for t in inputs.block_inputs(B, n, H, seed=4))
    r = oracle_mod.attention_block(X, Wqkv, Wo, H, n, 2, 0.125)
    want = mha_exact(X, Wqkv, Wo, H, 0.125, oracle_mod.round_bf16_f64)
    # the two differ only by fp64 rounding before each bf16 rounding: at most
    # one bf16 step anywhere, almost everywhere identical
    diff = np.abs(r["Y"] - want)
    ulp = np.ldexp(1.0, np.frexp(np.abs(want))[1] - 8)
    assert np.all(diff <= ulp + 1e-30)
    assert (diff == 0).mean() > 0.99
    # and the grouping really is one key per group (strided init with N = n)
    assert np.array_equal(r["belong"], np.broadcast_to(np.arange(n), (B, H, n)))


def test_relabelling_the_heads_leaves_the_output_unchanged(oracle_mod):
    B, n, H = 1, 64, 4
    D = 64 * H
    X, Wqkv, Wo = (f64(t) for t in inputs.block_inputs(B, n, H, seed=9))
    tau = np.array([2, 0, 3, 1])
    rows = np.concatenate([64 * tau[h] + np.arange(64) for h in range(H)])
    Wqkv2 = np.concatenate([Wqkv[i * D:(i + 1) * D][rows] for i in range(3)])
    Wo2 = Wo[:, rows]
    a = oracle_mod.attention_block(X, Wqkv, Wo, H, 8, 3, 0.125)
    b = oracle_mod.attention_block(X, Wqkv2, Wo2, H, 8, 3, 0.125)
    # the heads' groupings are the same, permuted
    assert np.array_equal(b["belong"][0], a["belong"][0][tau])
    diff = np.abs(a["Y"] - b["Y"])
    ulp = np.ldexp(1.0, np.frexp(np.abs(a["Y"]))[1] - 8)
    assert np.all(diff <= ulp)  # only the order of the fp64 sum over heads differs
    assert (diff == 0).mean() > 0.99


# planted mistakes in the block oracle: each must fail at least one pin above
MUTANTS = {
    "head_split_feature_major": ("heads = P.reshape(B, n, 3, H, 64).transpose(2, 0, 3, 1, 4)",
                                 "heads = P.reshape(B, n, 3, 64, H).transpose(2, 0, 4, 1, 3)"),
    "out_weights_not_transposed": ("return round_bf16_f64(cat @ W.T)", "return round_bf16_f64(cat @ W)"),
    "head_output_not_rounded": ('O = round_bf16_f64(r["O"])', 'O = r["O"]'),
    "concat_feature_major": ("cat = O.transpose(0, 2, 1, 3).reshape(B, n, H * d)",
                             "cat = O.transpose(0, 2, 3, 1).reshape(B, n, H * d)"),
    "rounding_ties_away": ("np.rint(m * 256.0)", "np.floor(m * 256.0 + 0.5)"),
}
PINS = [
    lambda m: test_round_bf16_f64_is_one_correct_rounding(m),
    lambda m: test_zero_queries_give_permuted_token_mean(m, 2, 5, 2),
    lambda m: test_every_key_its_own_group_is_exact_multihead_attention(m),
    lambda m: test_relabelling_the_heads_leaves_the_output_unchanged(m),
]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_fails_the_pins(oracle_mod, name):
    import types

    src = open(oracle_mod.__file__).read()
    a, b = MUTANTS[name]
    assert src.count(a) == 1
    mod = types.ModuleType("oracle_mutant")
    mod.__file__ = oracle_mod.__file__
    exec(compile(src.replace(a, b), oracle_mod.__file__, "exec"), mod.__dict__)
    failed = 0
    for pin in PINS:
        try:
            pin(mod)
        except AssertionError:
            failed += 1
    assert failed > 0, f"no pin caught {name}"
