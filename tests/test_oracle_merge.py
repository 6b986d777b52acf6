"""Pins for the oracle's merge plan (adaptive group count, Section 5.1).

None of these re-types the oracle's formulas; they use:
  * constructed geometry whose radii, threshold and marks are known in closed
    form (members at c +- r e_a, a query of norm 5, centres a known distance
    apart), on both sides of each of the two conditions of Eq. 5;
  * Lemma 2's conclusion checked by brute force: merging a marked group (and
    every other group marked with the same partner) into its partner keeps
    every member within the threshold of the merged centre;
  * Lemma 1's conclusion checked by brute force after the merge: every
    restored attention weight is within a factor eps of the exact one;
  * closed forms of the momentum update of N.
"""
import math

import numpy as np
import pytest

from paper_2306_01926_amd import inputs

D = 64


def unit(a):
    e = np.zeros(D)
    e[a] = 1.0
    return e


def slice_with_groups(centres, radii, qnorm=5.0, n_queries=8):
    """Keys c_g +- r_g e_(1 + g) and c_g itself, in that order, for each group
    g (three members, mean c_g, radius r_g exactly, the farthest member not
    the last); queries with largest norm qnorm."""
    K, belong = [], []
    for g, (c, r) in enumerate(zip(centres, radii)):
        for sgn in (1.0, -1.0, 0.0):
            K.append(c + sgn * r * unit(1 + g % (D - 1)))
            belong.append(g)
    Q = np.zeros((n_queries, D))
    Q[0, 0], Q[0, 1] = 0.6 * qnorm, 0.8 * qnorm  # norm qnorm (3-4-5 scaled)
    Q[1:, 2] = 0.5
    n = len(K)
    if n_queries < n:
        Q = np.vstack([Q, np.zeros((n - n_queries, D))])
    return Q[None, None, :n], np.array(K)[None, None], np.array(belong, np.int32)[None, None]


def plan(oracle_mod, centres, radii, eps, scale=0.125, counts=None):
    Q, K, bel = slice_with_groups(centres, radii)
    N = len(centres)
    cen = np.array(centres, np.float32)[None, None]
    cnt = np.array(counts if counts is not None else [3] * N, np.int32)[None, None]
    return oracle_mod.merge_plan(Q, K, bel, cen, cnt, N, scale, eps)


def test_radius_and_threshold_closed_form(oracle_mod):
    centres = [np.zeros(D), 2.0 * unit(0), -2.0 * unit(0), 4.0 * unit(0)]
    radii = [0.25, 0.5, 0.125, 1.0]
    eps = 2.0
    p = plan(oracle_mod, centres, radii, eps, scale=0.125)
    assert np.array_equal(p["radius"][0, 0], np.array(radii))
    # R' = |scale| max |q| = 0.125 * 5;  dthr = ln(eps) / (2 R')
    assert p["dthr"][0, 0] == pytest.approx(math.log(2.0) / 1.25, rel=1e-15)
    # a negative scale bounds the same scores
    q = plan(oracle_mod, centres, radii, eps, scale=-0.125)
    assert q["dthr"][0, 0] == p["dthr"][0, 0]


# two groups: S1 = {0} at the origin, S2 = {1} at distance delta along e_0
@pytest.mark.parametrize("delta,r0,r1,marked", [
    (0.1, 0.1, 0.05, True),    # delta + r0 = 0.2 <= t, delta + r1 = 0.15 <= t / 2
    (0.1, 0.5, 0.05, False),   # first condition fails (S1 group too wide)
    (0.1, 0.1, 0.3, False),    # second fails: delta + r1 = 0.4 > t / 2 although <= t
    (0.35, 0.05, 0.05, False), # centres too far apart for the S2 side
    (0.0, 0.0, 0.0, True),     # coincident point groups
])
def test_merge_rule_of_eq5(oracle_mod, delta, r0, r1, marked):
    # qnorm 5, scale 0.125, eps = e^0.625: t = 0.625 / 1.25 = 0.5, t / 2 = 0.25
    p = plan(oracle_mod, [np.zeros(D), delta * unit(0)], [r0, r1], math.exp(0.625))
    assert p["dthr"][0, 0] == pytest.approx(0.5, rel=1e-12)
    assert p["partner"][0, 0, 0] == -1  # S1 groups are never marked
    assert (p["partner"][0, 0, 1] == 0) == marked
    assert p["merges"][0, 0] == int(marked)


def test_lowest_partner_and_empty_groups(oracle_mod):
    # S1 = {0, 1, 2}, S2 = {3, 4, 5}; t = 0.5
    c = [np.zeros(D), 0.05 * unit(0), 3.0 * unit(0), 0.1 * unit(0), 3.05 * unit(0), 9.0 * unit(0)]
    r = [0.05, 0.05, 0.05, 0.05, 0.05, 0.05]
    p = plan(oracle_mod, c, r, math.exp(0.625))
    assert list(p["partner"][0, 0]) == [-1, -1, -1, 0, 2, -1]
    assert p["merges"][0, 0] == 2
    # group 0 empty: group 3 takes the next S1 group that qualifies
    p = plan(oracle_mod, c, [0.0] + r[1:], math.exp(0.625), counts=[0, 3, 3, 3, 3, 3])
    assert list(p["partner"][0, 0]) == [-1, -1, -1, 1, 2, -1]
    # group 4 empty: never marked
    p = plan(oracle_mod, c, r, math.exp(0.625), counts=[3, 3, 3, 3, 0, 3])
    assert p["partner"][0, 0, 4] == -1 and p["merges"][0, 0] == 1


def merged_groups(belong, partner):
    """Group of each key after merging every marked group into its partner."""
    target = np.where(partner >= 0, partner, np.arange(len(partner)))
    return target[belong]


@pytest.mark.parametrize("seed", [0, 1])
def test_lemma2_and_lemma1_hold_after_merging(oracle_mod, seed):
    # tight mixture keys and a large eps so that several groups merge
    n, N = 600, 48
    Q, K, V = inputs.make_qkv(1, 2, n, D, "f32", seed, 12, 0.01, 0.02)
    Q = inputs.as_float64(Q) * 0.2
    K = inputs.as_float64(K)
    cl = oracle_mod.cluster(K, N, 6, "f32")
    eps = 1.5
    p = oracle_mod.merge_plan(Q, K, cl["belong"], cl["centroid"], cl["count"], N, 0.125, eps)
    assert p["merges"].sum() > 0, "the case should merge something"
    for h in range(2):
        bel, cnt = cl["belong"][0, h], cl["count"][0, h].astype(np.float64)
        cen = cl["centroid"][0, h].astype(np.float64)
        t = p["dthr"][0, h]
        new = merged_groups(bel, p["partner"][0, h])
        # Lemma 2 (and the transfer-node argument): every member of a merged
        # group lies within t of the count-weighted mean of the merged centres
        rep = np.zeros((N, D))
        for g in np.unique(new):
            parts = np.unique(bel[new == g])
            rep[g] = (cnt[parts, None] * cen[parts]).sum(0) / cnt[parts].sum()
            dist = np.linalg.norm(K[0, h][new == g] - rep[g], axis=1)
            assert dist.max() <= t * (1 + 1e-6), (g, dist.max(), t)
        # Lemma 1: restored attention within a factor eps of the exact one
        s = 0.125 * Q[0, h] @ K[0, h].T
        sb = 0.125 * Q[0, h] @ rep[new].T
        A = np.exp(s - s.max(1, keepdims=True))
        A /= A.sum(1, keepdims=True)
        Ab = np.exp(sb - sb.max(1, keepdims=True))
        Ab /= Ab.sum(1, keepdims=True)
        ratio = Ab / A
        assert ratio.max() <= eps * (1 + 1e-9) and ratio.min() >= 1 / eps / (1 + 1e-9)


@pytest.mark.parametrize("N,merges,alpha,want", [
    (128, [5, 3, 7], 0.5, 127),   # D = 3: 126.5 rounds up
    (128, [5, 3, 7], 1.0, 125),
    (128, [5, 3, 7], 0.0, 128),
    (64, [10, 12], 0.3, 61),      # 64 - 3.0
    (4, [9], 1.0, 1),             # never below one group
    (32, [], 0.5, 32),
])
def test_momentum_update_of_the_group_count(oracle_mod, N, merges, alpha, want):
    assert oracle_mod.next_group_count(N, merges, alpha) == want
