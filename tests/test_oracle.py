"""Pins of the fp64 oracle against brute force, closed forms, library routines on
special cases and finite differences.  None of these re-types the oracle's own
formula; each is chosen so that a dropped term, a wrong sign or index, or a
transposed operand in the oracle fails at least one of them.
"""
import itertools
import json
import os

import numpy as np
import pytest
import scipy.special
import torch

import oracle as O

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def rng(seed):
    return np.random.default_rng(seed)


# ------------------------------------------------------------------ router --

def brute_topk_set(row, k):
    """The unique k-subset whose every member beats every non-member under
    (value desc, index asc), found by enumerating all subsets."""
    E = len(row)
    beats = lambda a, b: row[a] > row[b] or (row[a] == row[b] and a < b)
    found = [S for S in itertools.combinations(range(E), k)
             if all(beats(a, b) for a in S for b in range(E) if b not in S)]
    assert len(found) == 1
    return set(found[0])


@pytest.mark.parametrize("k", [1, 2, 3, 6])
def test_topk_matches_brute_force_with_ties(k):
    r = rng(1)
    logits = r.integers(-2, 3, size=(200, 6)).astype(float)  # many exact ties
    idx = O.topk_select(logits, k)
    for t in range(len(logits)):
        assert set(idx[t]) == brute_topk_set(logits[t], k)
        for a, b in zip(idx[t][:-1], idx[t][1:]):   # rank order
            assert logits[t, a] > logits[t, b] or (logits[t, a] == logits[t, b] and a < b)


def test_topk_signed_zero_is_a_tie():
    logits = np.array([[-0.0, 0.0, -1.0], [0.0, -0.0, -1.0]])
    np.testing.assert_array_equal(O.topk_select(logits, 2), [[0, 1], [0, 1]])


def test_gate_equals_renormalised_full_softmax():
    r = rng(2)
    X, Wr, b = r.normal(size=(64, 16)), r.normal(size=(10, 16)), r.normal(size=10)
    idx, gate, logits = O.route_topk(X, Wr, b, 3)
    full = scipy.special.softmax(X @ Wr.T + b, axis=1)
    sel = np.take_along_axis(full, idx, 1)
    np.testing.assert_allclose(gate, sel / sel.sum(1, keepdims=True), rtol=1e-13)
    np.testing.assert_allclose(gate.sum(1), 1.0, atol=1e-15)
    np.testing.assert_allclose(logits, X @ Wr.T + b, rtol=1e-13)


def test_gate_k_equals_E_is_full_softmax():
    r = rng(3)
    X, Wr = r.normal(size=(32, 8)), r.normal(size=(5, 8))
    idx, gate, _ = O.route_topk(X, Wr, None, 5)
    full = scipy.special.softmax(X @ Wr.T, axis=1)
    np.testing.assert_allclose(gate, np.take_along_axis(full, idx, 1), rtol=1e-13)


def test_equal_logits_choose_lowest_indices_uniformly():
    X, Wr = np.ones((4, 3)), np.zeros((7, 3))
    idx, gate, _ = O.route_topk(X, Wr, np.zeros(7), 3)
    np.testing.assert_array_equal(idx, np.tile([0, 1, 2], (4, 1)))
    np.testing.assert_allclose(gate, 1.0 / 3.0, rtol=1e-15)


def test_router_is_expert_permutation_equivariant():
    r = rng(4)
    X, Wr, b = r.normal(size=(50, 12)), r.normal(size=(9, 12)), r.normal(size=9)
    perm = r.permutation(9)
    idx, gate, _ = O.route_topk(X, Wr, b, 4)
    idx_p, gate_p, _ = O.route_topk(X, Wr[perm], b[perm], 4)
    np.testing.assert_array_equal(perm[idx_p], idx)   # no ties with normal data
    np.testing.assert_allclose(gate_p, gate, rtol=1e-14)


def _route_fd_setup(seed=21, T=5, d=4, E=6, k=3):
    r = rng(seed)
    X, Wr = r.normal(size=(T, d)), r.normal(size=(E, d))
    bias = 3.0 * r.normal(size=E)            # wide selection margins
    _, _, logits = O.route_topk(X, Wr, bias, k)
    assert np.all(O.topk_gap(logits, k) > 1e-3)
    return X, Wr, bias, r.normal(size=(T, k))


def test_route_backward_matches_central_differences():
    """dX of L(X) = <dgate, gate(X)> through top-k and the renormalised softmax
    (scipy's softmax, the selection re-made at every evaluation) against the
    closed-form router backward."""
    X, Wr, bias, dgate = _route_fd_setup()
    k = dgate.shape[1]
    idx, gate, _ = O.route_topk(X, Wr, bias, k)

    def loss():
        lg = X @ Wr.T + bias
        sel = np.argsort(-lg, axis=1, kind="stable")[:, :k]
        return float(np.sum(dgate * scipy.special.softmax(np.take_along_axis(lg, sel, 1), axis=1)))

    dlogit, dX = O.route_topk_backward(Wr, idx, gate, dgate)
    np.testing.assert_allclose(dX, _fd(loss, X), rtol=1e-7, atol=1e-9)
    # and with respect to the logits themselves (selection fixed by the margins)
    lg0 = X @ Wr.T + bias

    def loss_l():
        sel = np.argsort(-lg0, axis=1, kind="stable")[:, :k]
        return float(np.sum(dgate * scipy.special.softmax(np.take_along_axis(lg0, sel, 1), axis=1)))

    np.testing.assert_allclose(dlogit, _fd(loss_l, lg0), rtol=1e-7, atol=1e-9)


def test_route_backward_invariants():
    """Per token the logit gradient sums to 0 (the gates sum to 1); k = 1 and a
    dgate constant over a token's choices give no gradient."""
    X, Wr, bias, dgate = _route_fd_setup(seed=22, T=40, d=8, E=10, k=4)
    idx, gate, _ = O.route_topk(X, Wr, bias, 4)
    dlogit, _ = O.route_topk_backward(Wr, idx, gate, dgate)
    np.testing.assert_allclose(dlogit.sum(axis=1), 0.0, atol=1e-12)
    assert np.count_nonzero(dlogit) <= dlogit.shape[0] * 4
    const = np.repeat(dgate[:, :1], 4, axis=1)
    assert np.all(np.abs(O.route_topk_backward(Wr, idx, gate, const)[0]) < 1e-12)
    idx1, gate1, _ = O.route_topk(X, Wr, bias, 1)
    dl1, dx1 = O.route_topk_backward(Wr, idx1, gate1, dgate[:, :1])
    assert not dl1.any() and not dx1.any()


def test_topk_gap():
    logits = np.array([[3.0, 1.0, 2.0, 2.0], [0.0, 0.0, 0.0, 5.0]])
    np.testing.assert_array_equal(O.topk_gap(logits, 2), [0.0, 0.0])
    np.testing.assert_array_equal(O.topk_gap(logits, 1), [1.0, 5.0])
    assert np.isinf(O.topk_gap(logits, 4)).all()


# ------------------------------------------------------- int8 profiling ----

def test_quantize_golden():
    g = json.load(open(os.path.join(GOLD, "quantize_int8_rows.json")))
    q, s = O.quantize_int8_rows(np.array(g["W"], dtype=np.float32))
    np.testing.assert_array_equal(q, g["q"])
    np.testing.assert_allclose(s * 127.0, g["s_times_127"], rtol=1e-7)
    assert s.dtype == np.float32 and q.dtype == np.int8


def test_quantize_error_bound():
    W = rng(5).normal(size=(16, 300)).astype(np.float32)
    q, s = O.quantize_int8_rows(W)
    assert np.abs(q).max() <= 127
    assert (np.abs(q) == 127).any(axis=1).all()        # the row maximum maps to +-127
    err = np.abs(q.astype(np.float64) * s[:, None] - W)
    assert np.all(err <= 0.5 * s[:, None] * (1 + 1e-6))


def test_hist_totals_and_bruteforce():
    r = rng(6)
    T, d, E, k = 300, 24, 7, 3
    X = r.normal(size=(T, d))
    q, s = O.quantize_int8_rows(r.normal(size=(E, d)))
    b = r.normal(size=E)
    counts, idx, lg = O.profile_hist(X, q, s, b, k)
    assert counts.sum() == T * k and counts.max() <= T
    brute = [sum(e in set(idx[t]) for t in range(T)) for e in range(E)]
    np.testing.assert_array_equal(counts, brute)
    # dequantised logits: one independent recomputation per element
    t, e = 17, 4
    assert abs(lg[t, e] - (sum(X[t, i] * float(q[e, i]) for i in range(d)) * float(s[e]) + b[e])) < 1e-12


def test_hist_equals_full_precision_when_router_is_exactly_quantised():
    r = rng(7)
    T, d, E, k = 500, 32, 8, 2
    q_true = r.integers(-127, 128, size=(E, d))
    q_true[:, 0] = 127                         # make max |row| = 127 exactly
    scale = 2.0 ** -9
    Wr = q_true * scale                        # exactly representable
    X = r.normal(size=(T, d))
    q, s = O.quantize_int8_rows(Wr)
    np.testing.assert_array_equal(q, q_true)
    counts, idx8, _ = O.profile_hist(X, q, s, None, k)
    idx, _, _ = O.route_topk(X, Wr, None, k)
    np.testing.assert_array_equal(idx8, idx)
    np.testing.assert_array_equal(counts, np.bincount(idx.ravel(), minlength=E))


# ------------------------------------------------------------ merge plan ----

def test_frequency_plan_golden():
    g = json.load(open(os.path.join(GOLD, "merge_plan_example.json")))
    plan = O.frequency_merge_plan(g["counts"], g["n_merge"], g["group"])
    assert plan.kept == g["kept"] and plan.groups == g["groups"]
    np.testing.assert_array_equal(plan.expert_map, g["expert_map"])
    alpha = np.array(g["counts"], dtype=float)
    np.testing.assert_allclose(O.merge_weights(alpha, plan.groups[0]),
                               g["alpha_equals_counts_merge_coefficients"]["group0"])
    np.testing.assert_allclose(O.merge_weights(alpha, plan.groups[1]),
                               g["alpha_equals_counts_merge_coefficients"]["group1"])


def test_explicit_plan_golden():
    g = json.load(open(os.path.join(GOLD, "explicit_merge_plan_example.json")))
    for c in g["cases"]:
        plan = O.explicit_merge_plan(c["E"], c["groups"], tune_all=c["tune_all"])
        assert plan.kept == c["kept"], c["note"]
        assert plan.groups == c["groups"], c["note"]
        assert plan.S == c["S"], c["note"]
        np.testing.assert_array_equal(plan.expert_map, c["expert_map"], err_msg=c["note"])
        np.testing.assert_array_equal(plan.tuning, c["tuning"], err_msg=c["note"])


def test_frequency_plan_properties():
    r = rng(8)
    counts = r.integers(0, 50, size=64)
    plan = O.frequency_merge_plan(counts, 32, 4, n_tune=16)
    assert len(plan.kept) == 32 and len(plan.groups) == 8 and plan.S == 40
    merged = [e for g in plan.groups for e in g]
    assert sorted(plan.kept + merged) == list(range(64))
    assert min(counts[plan.kept]) >= max(counts[merged])
    assert plan.tuning.sum() == 16 and plan.tuning[:16].all()
    for e in range(64):
        s = plan.expert_map[e]
        assert (plan.kept[s] == e) if s < 32 else (e in plan.groups[s - 32])


# ------------------------------------------------------------------ merge ----

def test_merge_identity_copy_mean_closed_form():
    r = rng(9)
    W = r.normal(size=(5, 6, 7))
    same = np.stack([W[0]] * 3)
    np.testing.assert_allclose(O.merge_experts(same, [0, 1, 2], [0.1, 5.0, 2.0]), W[0], rtol=1e-14)
    np.testing.assert_array_equal(O.merge_experts(W, [3], [0, 0, 0, 4.0, 0]), W[3])
    np.testing.assert_allclose(O.merge_experts(W, [0, 2, 4], np.ones(5)), W[[0, 2, 4]].mean(0), rtol=1e-13)
    np.testing.assert_allclose(O.merge_experts(W, [0, 1], [1.0, 3.0]), 0.25 * W[0] + 0.75 * W[1], rtol=1e-14)
    np.testing.assert_allclose(O.merge_experts(W, [1, 3], np.zeros(5)), (W[1] + W[3]) / 2, rtol=1e-14)
    V = r.normal(size=W.shape)
    a = r.uniform(size=5)
    np.testing.assert_allclose(O.merge_experts(2 * W - 3 * V, [0, 1, 4], a),
                               2 * O.merge_experts(W, [0, 1, 4], a) - 3 * O.merge_experts(V, [0, 1, 4], a),
                               rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- permute ----

def test_permute_maps_properties():
    r = rng(10)
    T, E, k = 120, 8, 3
    logits = r.normal(size=(T, E))
    idx = O.topk_select(logits, k)
    gate = O.softmax_rows(np.take_along_axis(logits, idx, 1))
    plan = O.frequency_merge_plan(r.integers(0, 9, size=E), 4, 2)
    offsets, ptok, pgate, inv = O.permute_maps(idx, gate, plan.expert_map, plan.S)
    slot = plan.expert_map[idx]
    pairs = {(t, int(slot[t, j])) for t in range(T) for j in range(k)}
    counts = [sum(1 for (_, s) in pairs if s == c) for c in range(plan.S)]
    np.testing.assert_array_equal(offsets, np.concatenate([[0], np.cumsum(counts)]))
    assert len(ptok) == len(pairs) < T * k            # folding happened
    for s in range(plan.S):
        seg = ptok[offsets[s]:offsets[s + 1]]
        assert np.all(np.diff(seg) > 0)                # stable: ascending tokens
        assert all((int(t), s) in pairs for t in seg)
    for t in range(T):
        np.testing.assert_allclose(pgate[[p for p in inv[t] if p >= 0]].sum(), gate[t].sum(), rtol=1e-14)
        for j in range(k):
            p = inv[t, j] if inv[t, j] >= 0 else -2 - inv[t, j]
            assert ptok[p] == t and offsets[slot[t, j]] <= p < offsets[slot[t, j] + 1]
        firsts = [j for j in range(k) if inv[t, j] >= 0]
        assert len(firsts) == len({int(s) for s in slot[t]})
    # unpermute(permute(X)) with identity experts and unit gate sums returns X
    X = r.normal(size=(T, 5))
    Xp = X[ptok]
    Y = np.zeros_like(X)
    for t in range(T):
        for p in inv[t]:
            if p >= 0:
                Y[t] += pgate[p] * Xp[p]
    np.testing.assert_allclose(Y, X, rtol=1e-13)


# ------------------------------------------------------------ expert FFN ----

def torch_swiglu(x, Wg, Wu, Wd):
    x, Wg, Wu, Wd = (torch.from_numpy(np.asarray(a, dtype=np.float64)) for a in (x, Wg, Wu, Wd))
    h = torch.nn.functional.silu(x @ Wg.T) * (x @ Wu.T)
    return (h @ Wd.T).numpy()


def make_slots(r, S, d, I, n_shared=0, tuning=None):
    wg = [r.normal(size=(I, d)) for _ in range(S)]
    wu = [r.normal(size=(I, d)) for _ in range(S)]
    wd = [r.normal(size=(d, I)) for _ in range(S)]
    tuning = [True] * S if tuning is None else tuning
    return O.SlotWeights(wg, wu, wd, tuning, n_shared=n_shared)


def test_single_expert_is_dense_swiglu():
    r = rng(11)
    X = r.normal(size=(20, 6))
    slots = make_slots(r, 1, 6, 9)
    idx, gate, _ = O.route_topk(X, r.normal(size=(1, 6)), None, 1)
    np.testing.assert_array_equal(gate, 1.0)
    Y = O.moe_forward(X, idx, gate, np.array([0]), slots)
    np.testing.assert_allclose(Y, torch_swiglu(X, slots.wg[0], slots.wu[0], slots.wd[0]), rtol=1e-12)


def test_uniform_gate_all_experts_is_mean_of_experts():
    r = rng(12)
    E, X = 4, r.normal(size=(16, 5))
    slots = make_slots(r, E, 5, 7)
    idx, gate, _ = O.route_topk(X, np.zeros((E, 5)), np.zeros(E), E)
    Y = O.moe_forward(X, idx, gate, np.arange(E), slots)
    mean = np.mean([torch_swiglu(X, slots.wg[e], slots.wu[e], slots.wd[e]) for e in range(E)], axis=0)
    np.testing.assert_allclose(Y, mean, rtol=1e-12)


def test_shared_experts_add_dense_outputs():
    r = rng(13)
    X = r.normal(size=(10, 4))
    slots = make_slots(r, 3, 4, 6, n_shared=2)
    idx = np.zeros((10, 1), dtype=int)
    gate = np.full((10, 1), 0.5)
    Y = O.moe_forward(X, idx, gate, np.array([0]), slots)
    ref = 0.5 * torch_swiglu(X, slots.wg[0], slots.wu[0], slots.wd[0])
    ref += torch_swiglu(X, slots.wg[1], slots.wu[1], slots.wd[1])
    ref += torch_swiglu(X, slots.wg[2], slots.wu[2], slots.wd[2])
    np.testing.assert_allclose(Y, ref, rtol=1e-12)


def _fd_setup(n_shared=0, tuning=None):
    r = rng(14)
    T, d, E, k, I = 4, 3, 3, 2, 5
    X, dY = r.normal(size=(T, d)), r.normal(size=(T, d))
    idx, gate, _ = O.route_topk(X, r.normal(size=(E, d)), r.normal(size=E), k)
    slots = make_slots(r, E + n_shared, d, I, n_shared=n_shared, tuning=tuning)
    return X, dY, idx, gate, np.arange(E), slots


def _loss(X, dY, idx, gate, emap, slots):
    return float(np.sum(dY * O.moe_forward(X, idx, gate, emap, slots)))


def _fd(f, a, h=1e-6):
    g = np.zeros_like(a)
    for i in np.ndindex(a.shape):
        old = a[i]
        a[i] = old + h
        fp = f()
        a[i] = old - h
        fm = f()
        a[i] = old
        g[i] = (fp - fm) / (2 * h)
    return g


@pytest.mark.parametrize("n_shared", [0, 1])
def test_backward_matches_central_differences(n_shared):
    tuning = [True, False, True] + [True] * n_shared
    X, dY, idx, gate, emap, slots = _fd_setup(n_shared, tuning)
    dX, dW, dgate = O.moe_backward(X, dY, idx, gate, emap, slots)
    f = lambda: _loss(X, dY, idx, gate, emap, slots)
    np.testing.assert_allclose(dX, _fd(f, X), rtol=1e-7, atol=1e-8)
    np.testing.assert_allclose(dgate, _fd(f, gate), rtol=1e-7, atol=1e-8)
    assert set(dW) == {s for s in range(slots.S) if tuning[s]}
    for s, (dWg, dWu, dWd) in dW.items():
        np.testing.assert_allclose(dWg, _fd(f, slots.wg[s]), rtol=1e-7, atol=1e-8)
        np.testing.assert_allclose(dWu, _fd(f, slots.wu[s]), rtol=1e-7, atol=1e-8)
        np.testing.assert_allclose(dWd, _fd(f, slots.wd[s]), rtol=1e-7, atol=1e-8)


def test_adjoint_identity():
    X, dY, idx, gate, emap, slots = _fd_setup()
    dX, _, _ = O.moe_backward(X, dY, idx, gate, emap, slots)
    v = rng(15).normal(size=X.shape)
    h = 1e-6
    jv = (O.moe_forward(X + h * v, idx, gate, emap, slots)
          - O.moe_forward(X - h * v, idx, gate, emap, slots)) / (2 * h)
    assert abs(np.sum(dY * jv) - np.sum(dX * v)) < 1e-7 * max(1.0, abs(np.sum(dX * v)))


def test_empty_tuning_slot_gets_zero_dw():
    X, dY, idx, gate, _, slots = _fd_setup()
    emap = np.array([0, 0, 0])              # slots 1 and 2 receive no rows
    _, dW, _ = O.moe_backward(X, dY, idx, gate, emap, slots)
    for s in (1, 2):
        assert all(np.all(w == 0) for w in dW[s])


def test_expert_utility_per_token_gradients_and_folding():
    """Eq. 3 utility: (a) one routed expert with every token on it at gate 1:
    u^2 / n equals the sum over tokens of the squared norms of that token's
    weight gradient, taken by torch autograd (float64) through a dense SwiGLU
    with torch's silu; (b) a token whose two choices reach the same slot counts
    once, with the summed gate; (c) linear in dY; (d) an empty slot has 0."""
    r = rng(31)
    T, d, I = 7, 5, 6
    X, dY = r.normal(size=(T, d)), r.normal(size=(T, d))
    Wg, Wu, Wd = r.normal(size=(I, d)), r.normal(size=(I, d)), r.normal(size=(d, I))
    slots = O.SlotWeights([Wg, Wg], [Wu, Wu], [Wd, Wd], [True, True])
    emap = np.array([0, 1])
    idx = np.zeros((T, 1), dtype=np.int64)
    gate = np.ones((T, 1))
    u = O.expert_utility(X, dY, idx, gate, emap, slots)
    assert u[1] == 0.0
    tot = 0.0
    for t in range(T):
        ws = [torch.tensor(w, dtype=torch.float64, requires_grad=True) for w in (Wg, Wu, Wd)]
        x = torch.tensor(X[t], dtype=torch.float64)
        y = ws[2] @ (torch.nn.functional.silu(ws[0] @ x) * (ws[1] @ x))
        (y @ torch.tensor(dY[t], dtype=torch.float64)).backward()
        tot += sum(float((w.grad ** 2).sum()) for w in ws)
    np.testing.assert_allclose(u[0] ** 2 / T, tot, rtol=1e-12)
    g2 = r.uniform(0.1, 0.9, size=(T, 2))
    u2 = O.expert_utility(X, dY, np.zeros((T, 2), dtype=np.int64), g2, emap, slots)
    u1 = O.expert_utility(X, dY, idx, g2.sum(axis=1, keepdims=True), emap, slots)
    np.testing.assert_allclose(u2, u1, rtol=1e-12)
    np.testing.assert_allclose(O.expert_utility(X, 3 * dY, idx, gate, emap, slots), 3 * u, rtol=1e-12)


def test_grad_columns_match_central_differences():
    r = rng(16)
    n, d, I = 6, 4, 7
    x, dO = r.normal(size=(n, d)), r.normal(size=(n, d))
    Wg, Wu, Wd = r.normal(size=(I, d)), r.normal(size=(I, d)), r.normal(size=(d, I))
    f = lambda: float(np.sum(dO * O.swiglu_fwd(x, Wg, Wu, Wd)[3]))
    cols = [1, 4, 6]
    dWg, dWu, dWd = O.expert_grad_columns(x, Wg, Wu, Wd, dO, cols)
    np.testing.assert_allclose(dWg, _fd(f, Wg)[cols], rtol=1e-7, atol=1e-8)
    np.testing.assert_allclose(dWu, _fd(f, Wu)[cols], rtol=1e-7, atol=1e-8)
    np.testing.assert_allclose(dWd, _fd(f, Wd)[:, cols], rtol=1e-7, atol=1e-8)


def test_expert_utility_rank_one_route_equals_per_token_gradients():
    """The batched utility (norms of rank-one products) against the explicit
    per-token gradients of expert_utility, which the autograd test above pins:
    several routed slots with folded choices (two experts of a token in one
    merged slot), an empty slot, a frozen slot, two shared experts and unequal
    gates; then a random layer with ties of slots across many tokens."""
    r = rng(33)
    T, d, I, E, k = 40, 6, 7, 6, 3
    X, dY = r.normal(size=(T, d)), r.normal(size=(T, d))
    S_r, n_sh = 5, 2
    mats = [(r.normal(size=(I, d)), r.normal(size=(I, d)), r.normal(size=(d, I))) for _ in range(S_r + n_sh)]
    slots = O.SlotWeights([m[0] for m in mats], [m[1] for m in mats], [m[2] for m in mats],
                          [True, False, True, True, True, True, True], n_shared=n_sh)
    emap = np.array([0, 1, 2, 2, 0, 4])           # experts 2 and 3 share slot 2, 0 and 4 share slot 0
    idx = np.stack([r.choice(E, size=k, replace=False) for _ in range(T)])
    idx[idx == 5] = 4                            # nothing reaches slot 4... through expert 5
    idx[:, 0] = np.where(idx[:, 0] == 4, 1, idx[:, 0])
    z = r.normal(size=(T, k))
    gate = np.exp(z) / np.exp(z).sum(1, keepdims=True)
    u_ref = O.expert_utility(X, dY, idx, gate, emap, slots)
    u = O.expert_utility_rank_one(X, dY, idx, gate, emap, slots)
    folded = sum(len(set(emap[idx[t]])) < k for t in range(T))
    assert folded > 0
    np.testing.assert_allclose(u, u_ref, rtol=1e-12, atol=0)
    assert np.array_equal(u == 0, u_ref == 0)
    # a plain random layer
    idx2 = np.stack([r.choice(E, size=k, replace=False) for _ in range(T)])
    emap2 = np.array([0, 1, 2, 3, 4, 4])
    np.testing.assert_allclose(O.expert_utility_rank_one(X, dY, idx2, gate, emap2, slots),
                               O.expert_utility(X, dY, idx2, gate, emap2, slots), rtol=1e-12)
