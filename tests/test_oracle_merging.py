"""Pins of the oracle's layer-aware merging (Section 5): the per-layer budget of
Eq. 1, the PCA features of the experts and the fused cross-layer K-Means.
None of these re-types the oracle's formulas: a hand-worked example, a
brute-force search over integer budgets, scikit-learn's PCA, closed-form
geometry and brute force over partitions fix the results."""
import itertools
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle as O
from paper_2508_19078_amd import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden", "merge_budget_example.json")


# ------------------------------------------------------------- Eq. 1 budget --

def test_budget_hand_worked_example():
    g = json.load(open(GOLD))
    counts = np.array(g["counts"])
    tuning = np.array(g["tuning"], dtype=bool)
    for case in g["cases"]:
        B, share = O.merge_budget(counts, tuning, g["total_tokens"], case["B_non"])
        assert B.tolist() == case["budget"], case
        want = [float(Fraction(a, b)) for a, b in case["share"]]
        np.testing.assert_allclose(share, want, rtol=1e-14)


def _sq_err(share, B):
    return float(np.sum((np.asarray(share) - np.asarray(B)) ** 2))


@pytest.mark.parametrize("seed", range(12))
def test_budget_is_the_closest_feasible_integer_split(seed):
    """With a feasible total, the integer budgets minimise sum (share - B)^2
    over all vectors with sum B_non and min(1, n_l) <= B_l <= n_l (searched
    exhaustively); outside the feasible range every layer sits at a bound."""
    rng = np.random.default_rng(seed)
    L, E = int(rng.integers(2, 5)), 6
    counts = rng.integers(0, 40, size=(L, E))
    tuning = rng.random((L, E)) < 0.3
    tuning[0, :] = False
    n = (~tuning).sum(1)
    lo = np.minimum(1, n)
    for B_non in range(0, int(n.sum()) + 3):
        B, share = O.merge_budget(counts, tuning, 50.0, B_non)
        assert np.all(B >= lo) and np.all(B <= n)
        if B_non < lo.sum():
            assert np.array_equal(B, lo)
            continue
        if B_non > n.sum():
            assert np.array_equal(B, n)
            continue
        assert B.sum() == B_non
        best = min(_sq_err(share, c) for c in itertools.product(*[range(a, b + 1) for a, b in zip(lo, n)])
                   if sum(c) == B_non)
        assert _sq_err(share, B) <= best + 1e-12


def test_budget_largest_remainder_and_layer_order():
    """No clamp binding: each layer gets floor(share) or floor(share) + 1, the
    +1 going to the largest fractional parts; with equal variances the shares
    are proportional to L - l + 1, so earlier layers never get less."""
    L, E = 7, 64
    row = np.arange(E) % 5 + 1
    counts = np.tile(row, (L, 1))
    tuning = np.zeros((L, E), dtype=bool)
    B, share = O.merge_budget(counts, tuning, 100.0, 100)
    np.testing.assert_allclose(share, 100 * np.arange(L, 0, -1) / (L * (L + 1) / 2), rtol=1e-13)
    fl = np.floor(share)
    assert B.sum() == 100 and np.all((B == fl) | (B == fl + 1))
    extra = np.argsort(-(share - fl), kind="stable")[:100 - int(fl.sum())]
    assert sorted(np.nonzero(B == fl + 1)[0].tolist()) == sorted(extra.tolist())
    assert np.all(np.diff(B) <= 0)


def test_budget_scale_invariance_and_flat_layer():
    rng = np.random.default_rng(3)
    counts = rng.integers(0, 100, size=(5, 16))
    tuning = np.zeros((5, 16), dtype=bool)
    B1, s1 = O.merge_budget(counts, tuning, 77.0, 30)
    B2, s2 = O.merge_budget(counts * 3, tuning, 231.0, 30)
    assert np.array_equal(B1, B2)
    np.testing.assert_allclose(s1, s2, rtol=1e-12)
    # a layer whose experts are all equally active has v = 0 -> the eps floor
    # makes its weight dominate: it takes every slot it can hold
    counts[2] = 7
    B, _ = O.merge_budget(counts, tuning, 77.0, 30)
    assert B[2] == 16 and B.sum() == 30


# ------------------------------------------------------------ PCA features --

def _planted(n, D, K, rng, mix=0.7):
    protos = rng.standard_normal((K, D))
    cls = np.arange(n) % K
    X = np.sqrt(mix) * protos[cls] + np.sqrt(1 - mix) * rng.standard_normal((n, D))
    return X, cls


def test_pca_scores_match_scikit_learn():
    from sklearn.decomposition import PCA
    rng = np.random.default_rng(0)
    X, _ = _planted(12, 300, 4, rng)
    X += 5.0                                  # a large common offset
    for r in (1, 3, 6):
        Z = O.pca_features(X, r)
        S = PCA(n_components=r, svd_solver="full").fit_transform(X)
        # scores agree up to the sign of each component
        for j in range(r):
            sgn = np.sign(Z[:, j] @ S[:, j])
            np.testing.assert_allclose(Z[:, j], sgn * S[:, j], rtol=1e-9, atol=1e-9)


def test_pca_full_rank_and_invariances():
    rng = np.random.default_rng(1)
    X = rng.standard_normal((9, 200))
    Xc = X - X.mean(0)
    Z = O.pca_features(X, 12)                 # r beyond the rank: zero columns
    assert np.all(Z[:, 9:] == 0)
    np.testing.assert_allclose(Z @ Z.T, Xc @ Xc.T, rtol=1e-10, atol=1e-10)
    G = Z.T @ Z                               # scores are orthogonal, decreasing
    np.testing.assert_allclose(G - np.diag(np.diag(G)), 0, atol=1e-9)
    assert np.all(np.diff(np.diag(G)[:8]) <= 1e-9)
    Z2 = O.pca_features(X + rng.standard_normal(200), 4)   # same shift for all
    np.testing.assert_allclose(Z2 @ Z2.T, Z[:, :4] @ Z[:, :4].T, rtol=1e-9, atol=1e-9)


def test_expert_vectors_order():
    wg = np.arange(2 * 3 * 4).reshape(2, 3, 4)
    wu = 100 + np.arange(2 * 3 * 4).reshape(2, 3, 4)
    wd = 200 + np.arange(2 * 4 * 3).reshape(2, 4, 3)
    v = O.expert_vectors(wg, wu, wd)
    assert v.shape == (2, 36)
    assert v[1, 0] == wg[1, 0, 0] and v[1, 12] == wu[1, 0, 0] and v[1, 24] == wd[1, 0, 0]
    assert v[0, 35] == wd[0, 3, 2]


# ----------------------------------------------------------- K-Means seeds --

def test_maximin_seeds_geometry():
    ang = np.deg2rad([0.0, 10.0, 90.0, 180.0])
    rad = np.array([2.0, 1.0, 1.5, 1.0])
    Z = np.stack([rad * np.cos(ang), rad * np.sin(ang)], 1)
    # largest norm first (0 deg), then the opposite direction, then 90 deg
    assert O.maximin_seeds(Z, 4) == [0, 3, 2, 1]
    assert O.maximin_seeds(Z, 2) == [0, 3]
    # equal norms: the lower index starts
    assert O.maximin_seeds(np.eye(3), 1) == [0]


# --------------------------------------------------------- fused K-Means ----

def _objective(Zh, lab):
    tot = 0.0
    for c in np.unique(lab):
        m = Zh[lab == c].mean(0)
        tot += np.sum(Zh[lab == c] @ m) / np.linalg.norm(m)
    return tot


def _same_partition(a, b):
    a, b = np.asarray(a), np.asarray(b)
    return all(len(set(b[a == c])) == 1 for c in np.unique(a)) and \
        all(len(set(a[b == c])) == 1 for c in np.unique(b))


def _directions(n, K, r, rng, spread=0.05):
    centers = rng.standard_normal((K, r))
    cls = rng.permutation(np.arange(n) % K)
    Z = centers[cls] + spread * rng.standard_normal((n, r))
    Z *= rng.uniform(0.5, 3.0, size=(n, 1))          # norms do not matter
    return Z, cls


def test_kmeans_recovers_planted_clusters_per_layer():
    rng = np.random.default_rng(5)
    feats, cls, Bs = [], [], []
    for n, K in ((12, 3), (20, 5), (7, 2), (16, 4)):
        Z, c = _directions(n, K, 6, rng)
        feats.append(Z)
        cls.append(c)
        Bs.append(K)
    labels, passes = O.fused_kmeans(feats, Bs, max_iter=50)
    for l in range(4):
        assert _same_partition(labels[l], cls[l])
        assert set(labels[l].tolist()) == set(range(Bs[l]))
        assert 1 <= passes[l] < 50


def test_fused_equals_independent_layers():
    """Masking cross-layer distances makes the fused problem the union of the
    per-layer problems: same labels, same passes."""
    rng = np.random.default_rng(6)
    feats = [rng.standard_normal((n, 5)) for n in (10, 14, 9)]
    Bs = [3, 5, 2]
    labels, passes = O.fused_kmeans(feats, Bs, max_iter=40)
    for l in range(3):
        lab1, p1 = O.fused_kmeans([feats[l]], [Bs[l]], max_iter=40)
        assert np.array_equal(lab1[0], labels[l])
        assert p1[0] == passes[l]
    # an expert of layer 1 pointing exactly at a layer-0 seed stays in layer 1
    f2 = [feats[0], np.vstack([feats[1], feats[0][O.maximin_seeds(feats[0], 3)[0]]])]
    lab2, _ = O.fused_kmeans(f2, [3, 5], max_iter=40)
    assert 0 <= lab2[1][-1] < 5


def test_kmeans_fixed_point_and_monotone_objective():
    rng = np.random.default_rng(7)
    Z = rng.standard_normal((30, 4))
    Zh = O.unit_rows(Z)
    prev = -np.inf
    for it in range(1, 12):
        lab, _ = O.fused_kmeans([Z], [6], max_iter=it)
        J = _objective(Zh, lab[0])
        assert J >= prev - 1e-12
        prev = J
    lab, passes = O.fused_kmeans([Z], [6], max_iter=200)
    assert passes[0] < 200
    lab = lab[0]
    # converged: every expert's own centroid is its most similar one
    cents = {c: Zh[lab == c].mean(0) for c in np.unique(lab)}
    for e in range(30):
        sims = {c: Zh[e] @ m / np.linalg.norm(m) for c, m in cents.items()}
        assert sims[lab[e]] >= max(sims.values()) - 1e-12


def test_kmeans_brute_force_optimum_on_tiny_planted():
    rng = np.random.default_rng(8)
    for trial in range(5):
        Z, cls = _directions(7, 2, 3, rng, spread=0.1)
        lab, _ = O.fused_kmeans([Z], [2], max_iter=50)
        Zh = O.unit_rows(Z)
        best = max(_objective(Zh, np.array(p)) for p in itertools.product((0, 1), repeat=7)
                   if 0 < sum(p) < 7)
        assert _objective(Zh, lab[0]) >= best - 1e-12


def test_kmeans_degenerate_budgets():
    rng = np.random.default_rng(9)
    Z = rng.standard_normal((8, 3))
    lab, _ = O.fused_kmeans([Z, Z[:3]], [8, 1], max_iter=20)
    assert sorted(lab[0].tolist()) == list(range(8))
    assert lab[1].tolist() == [0, 0, 0]
    # one expert: its score is zero after centring; it forms the single group
    lab, _ = O.fused_kmeans([np.zeros((1, 3))], [1], max_iter=5)
    assert lab[0].tolist() == [0]


# ------------------------------------------------- planted expert weights ---

def test_pca_kmeans_recovers_planted_expert_classes():
    """End to end on synthetic expert weights: experts that share a class
    prototype (draw_planted_experts) end up in one group when the budget equals
    the number of classes present."""
    w = W.scaled(W.WORKLOADS["deepseek_stack"], d=64, I=96, E=16)
    feats, truth, Bs = [], [], []
    for layer in range(3):
        K = 4
        wg, wu, wd = W.draw_planted_experts(w, layer, K, 0.6)
        cls = W.expert_classes(w, layer, K)
        X = O.expert_vectors(wg.f64(), wu.f64(), wd.f64())
        feats.append(O.pca_features(X, K - 1))
        truth.append(cls)
        Bs.append(len(set(cls.tolist())))
    labels, _ = O.fused_kmeans(feats, Bs, max_iter=50)
    for l in range(3):
        assert _same_partition(labels[l], truth[l])
