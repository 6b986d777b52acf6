"""Pins for the oracle's backward pass (gradient with the grouping held fixed).

None of these re-types the oracle's formulas; they use:
  * central finite differences of a different formulation of the same forward:
    Section 4.2's naive restore (every key replaced by its group's mean, a
    plain n x n softmax, times V), which Lemma 3 proves equal to group
    attention, differentiated numerically in Q, K and V with the grouping
    fixed;
  * invariants: the value gradients add up to the output gradients
    (sum_k dV_k = sum_i dO_i, since each query's weights sum to 1) and the key
    gradients add up to 0 (the softmax is shift invariant).
"""
import types

import numpy as np
import pytest

D = 16


def restore_forward(Q, K, V, belong, N, scale):
    """Naive restore with the grouping fixed: keys -> member means."""
    n = K.shape[0]
    Kbar = np.zeros_like(K)
    for j in range(N):
        mem = belong == j
        if mem.any():
            Kbar[mem] = K[mem].mean(0)
    P = scale * Q @ Kbar.T
    A = np.exp(P - P.max(1, keepdims=True))
    A /= A.sum(1, keepdims=True)
    return A @ V


def grouping(rng, n, N, empty=()):
    live = [j for j in range(N) if j not in empty]
    belong = np.array(live + list(rng.choice(live, size=n - len(live))), np.int32)
    rng.shuffle(belong)
    return belong


def oracle_inputs(K, V, belong, N):
    count = np.bincount(belong, minlength=N).astype(np.int32)
    cen = np.zeros((N, K.shape[1]))
    vs = np.zeros((N, K.shape[1]))
    for j in range(N):
        if count[j]:
            cen[j] = K[belong == j].mean(0)
            vs[j] = V[belong == j].sum(0)
    return count, cen, vs


@pytest.mark.parametrize("seed,n,N,empty", [(0, 24, 5, ()), (1, 30, 7, (2, 5)), (2, 12, 12, ())])
def test_gradient_matches_finite_differences_of_the_naive_restore(oracle_mod, seed, n, N, empty):
    rng = np.random.default_rng(seed)
    Q, K, V, G = (rng.standard_normal((n, D)) for _ in range(4))
    belong = grouping(rng, n, N, empty)
    count, cen, vs = oracle_inputs(K, V, belong, N)
    scale = 0.7
    dQ, dK, dV = oracle_mod.backward(Q[None, None], G[None, None], belong[None, None], cen[None, None],
                                     count[None, None], vs[None, None], N, scale, "f32")
    f = lambda Q_, K_, V_: float((G * restore_forward(Q_, K_, V_, belong, N, scale)).sum())
    eps = 1e-6
    for name, X, grad in (("Q", Q, dQ), ("K", K, dK), ("V", V, dV)):
        for _ in range(25):
            i, c = rng.integers(n), rng.integers(D)
            Xp, Xm = X.copy(), X.copy()
            Xp[i, c] += eps
            Xm[i, c] -= eps
            args_p = {"Q": (Xp, K, V), "K": (Q, Xp, V), "V": (Q, K, Xp)}[name]
            args_m = {"Q": (Xm, K, V), "K": (Q, Xm, V), "V": (Q, K, Xm)}[name]
            num = (f(*args_p) - f(*args_m)) / (2 * eps)
            assert abs(num - grad[0, 0, i, c]) <= 1e-6 * max(1.0, abs(num)), (name, i, c, num, grad[0, 0, i, c])


def test_gradient_sums(oracle_mod):
    rng = np.random.default_rng(4)
    n, N = 200, 11
    Q, K, V, G = (rng.standard_normal((n, 64)) for _ in range(4))
    belong = grouping(rng, n, N, (3,))
    count, cen, vs = oracle_inputs(K, V, belong, N)
    dQ, dK, dV = oracle_mod.backward(Q[None, None], G[None, None], belong[None, None], cen[None, None],
                                     count[None, None], vs[None, None], N, 0.125, "f32")
    assert np.allclose(dV[0, 0].sum(0), G.sum(0), rtol=1e-10, atol=1e-10)
    assert np.allclose(dK[0, 0].sum(0), 0.0, atol=1e-10)


MUTANTS = {
    "key_gradient_not_divided_by_count": ("dK = np.take_along_axis(dr, idx, axis=2) / per_k",
                                          "dK = np.take_along_axis(dr, idx, axis=2)"),
    "value_gradient_not_divided_by_count": ("dV = np.take_along_axis(dmu, idx, axis=2) / per_k",
                                            "dV = np.take_along_axis(dmu, idx, axis=2)"),
    "softmax_backward_drops_the_mean_term": ("dp = w * (dw - D)", "dp = w * dw"),
    "query_gradient_unscaled": ("dQ = scale * np.einsum", "dQ = np.einsum"),
    "weights_without_count": ('e = np.where(live, c[:, :, None, :] * np.exp(p - m), 0.0)',
                              'e = np.where(live, np.exp(p - m), 0.0)'),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_fails_the_pins(oracle_mod, name):
    src = open(oracle_mod.__file__).read()
    a, b = MUTANTS[name]
    assert src.count(a) == 1
    mod = types.ModuleType("oracle_mutant")
    mod.__file__ = oracle_mod.__file__
    exec(compile(src.replace(a, b), oracle_mod.__file__, "exec"), mod.__dict__)
    failed = 0
    for pin in (lambda m: test_gradient_matches_finite_differences_of_the_naive_restore(m, 0, 24, 5, ()),
                lambda m: test_gradient_sums(m)):
        try:
            pin(mod)
        except AssertionError:
            failed += 1
    assert failed > 0, f"no pin caught {name}"
