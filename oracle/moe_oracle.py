"""fp64 CPU oracle for the MoE-layer hot path of Flux (federated MoE fine-tuning).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import this module.  The HIP library never
calls it, and it shares no code, constant or helper with the HIP library: it is
written from the paper's statement of the method, in plain NumPy, in float64.

What each function follows:

* Routing (Section 2.1, "MoE"): a gating network assigns each token to experts.
  The paper gives no formula; the reading used here is the usual softmax gate
  with top-k selection on the logits and renormalisation over the selected k,
  ties broken towards the lower expert index.
* Activation frequency (Section 2.2, Observation 2): tokens that activate an
  expert divided by all tokens.
* Quantisation-based profiling (Section 4.1): the same routing computed with a
  low-bit copy of the weights.  Here the router is int8 with one symmetric scale
  per expert row.
* Expert merging (Section 5.3, Eq. 2): a weighted average of the weights of the
  experts in a group, weights alpha_e normalised within the group.
* Gate re-routing (Section 7): original experts are remapped to the slot that
  now holds them, merged or not.
* Tuning and non-tuning experts (Section 1, Section 3): tuning experts receive
  weight gradients; non-tuning (merged, frozen) experts do not.
* Expert FFN: SwiGLU, out = W_down (silu(W_gate x) * (W_up x)).
* Expert utility (Section 6.1, Eq. 3): the gradient-norm utility of a slot.
* Quantised profiling of a layer stack (Section 4.1): int8 router and experts,
  each layer reading the RMS-normalised stream (the pre-norm of the paper's
  models), layers coupled by a residual stream.
* Layer-aware merging (Section 5): the per-layer budget of Eq. 1 (Section 5.1),
  then PCA features of the experts' parameters and K-Means with cosine
  distance over all layers at once, cross-layer pairs masked (Section 5.2).

Readings of silent or ambiguous points are listed in the design notes of the
repository and restated at each function.  Every function here is pinned by
tests that do not re-type its formula (brute force, closed forms, library
routines on special cases, finite differences).
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np

F64 = np.float64


def _f64(a) -> np.ndarray:
    a = np.asarray(a, dtype=F64)
    assert np.all(np.isfinite(a)), "oracle inputs must be finite"
    return a


# ------------------------------------------------------------------ router --

def router_logits(X, Wr, bias=None) -> np.ndarray:
    """logit[t, e] = <X[t], Wr[e]> + bias[e], exactly (fp64, inputs exact)."""
    X, Wr = _f64(X), _f64(Wr)
    logits = X @ Wr.T
    if bias is not None:
        logits = logits + _f64(bias)[None, :]
    return logits


def topk_select(logits, k: int) -> np.ndarray:
    """Indices of the k largest logits per row, in rank order.

    Order is (logit descending, expert index ascending): on equal logits the
    lower expert index ranks first.  A stable sort of the negated logits keeps
    equal keys in index order, and -0.0 compares equal to +0.0.
    """
    logits = _f64(logits)
    E = logits.shape[1]
    assert 1 <= k <= E
    order = np.argsort(-logits, axis=1, kind="stable")
    return order[:, :k].astype(np.int64)


def softmax_rows(z) -> np.ndarray:
    z = _f64(z)
    e = np.exp(z - z.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True)


def route_topk(X, Wr, bias, k: int):
    """Gate of one MoE layer: (idx [T,k], gate [T,k], logits [T,E]).

    gate is the softmax over the k selected logits, which equals the softmax
    over all E experts renormalised over the selected ones.
    """
    logits = router_logits(X, Wr, bias)
    idx = topk_select(logits, k)
    gate = softmax_rows(np.take_along_axis(logits, idx, axis=1))
    return idx, gate, logits


def route_topk_backward(Wr, idx, gate, dgate):
    """Router backward with the top-k selection held fixed (the selection is a
    piecewise-constant function of the logits).  The gate of a token is the
    softmax of its k selected logits, so a gradient dgate [T,k] on the gates
    gives the logits the softmax Jacobian-vector product
        dlogit[t, idx[t,j]] = gate[t,j] * (dgate[t,j] - sum_i gate[t,i] dgate[t,i])
    and 0 on the experts not selected; logit = X Wr^T + bias then gives
    dX = dlogit Wr.  Returns (dlogit [T,E], dX [T,d]).  (The router itself is
    frozen in expert-only tuning, so no weight or bias gradient is formed.)
    """
    Wr, gate, dgate = _f64(Wr), _f64(gate), _f64(dgate)
    idx = np.asarray(idx, dtype=np.int64)
    T, k = gate.shape
    inner = np.sum(gate * dgate, axis=1, keepdims=True)
    dsel = gate * (dgate - inner)
    dlogit = np.zeros((T, Wr.shape[0]), dtype=F64)
    np.put_along_axis(dlogit, idx, dsel, axis=1)
    return dlogit, dlogit @ Wr


def topk_gap(logits, k: int) -> np.ndarray:
    """logit_(k) - logit_(k+1) per row (inf when k == E): the selection margin."""
    logits = _f64(logits)
    s = -np.sort(-logits, axis=1)
    if k >= logits.shape[1]:
        return np.full(logits.shape[0], np.inf)
    return s[:, k - 1] - s[:, k]


# ------------------------------------------------------- int8 profiling ----

def quantize_int8_rows(W):
    """Per-row symmetric int8 quantisation of a router weight (Section 4.1).

    The section does not say how the low-bit copy is made; this is the
    definition of the int8 copy used throughout: s_e = max_i |W[e,i]| / 127 and
    q = clamp(round_half_even(W / s_e), -127, 127), a zero row getting s_e = 0
    and q = 0, with s_e, the division and the rounding in float32, the precision
    the copy's scales are stored in.  The division and the rounding decide an
    integer, so their precision is part of the definition, not an implementation
    detail (W is a bf16 or fp32 value, so max|W| is exact in float32 and the
    float32 quotient is the correctly rounded one).
    """
    W32 = np.asarray(W, dtype=np.float32)
    amax = np.max(np.abs(W32), axis=1)
    s = (amax / np.float32(127.0)).astype(np.float32)
    q = np.zeros(W32.shape, dtype=np.int8)
    nz = s > 0
    r = (W32[nz] / s[nz, None]).astype(np.float32)
    q[nz] = np.clip(np.rint(r), -127, 127).astype(np.int8)
    return q, s


def profile_logits(X, q, s, bias=None) -> np.ndarray:
    """Dequantised router logits: s_e * <X[t], q[e]> + bias[e] (fp64)."""
    logits = _f64(X) @ np.asarray(q, dtype=F64).T * _f64(s)[None, :]
    if bias is not None:
        logits = logits + _f64(bias)[None, :]
    return logits


def profile_hist(X, q, s, bias, k: int):
    """Activation histogram of the int8 profiling router: (counts [E], idx [T,k]).

    counts[e] = number of tokens whose top-k set under the dequantised logits
    contains e.  The activation frequency of Observation 2 is counts / T.
    """
    lg = profile_logits(X, q, s, bias)
    idx = topk_select(lg, k)
    counts = np.bincount(idx.ravel(), minlength=lg.shape[1]).astype(np.int64)
    return counts, idx, lg


# ------------------------------------------------------------ merge plan ----

class MergePlan:
    """Which slot holds which experts after merging (Sections 5.2 and 7).

    kept[j]     original expert held unchanged by routed slot j (j < K)
    groups[g]   original experts merged into routed slot K + g
    tuning[s]   slot s receives weight gradients
    expert_map  original expert -> routed slot (the re-routing table)
    """

    def __init__(self, E: int, kept: Sequence[int], groups: Sequence[Sequence[int]],
                 n_tune: Optional[int] = None, tune_groups: bool = False):
        self.E = E
        self.kept = [int(e) for e in kept]
        self.groups = [[int(e) for e in g] for g in groups]
        K, G = len(self.kept), len(self.groups)
        self.S = K + G
        n_tune = K if n_tune is None else n_tune
        self.tuning = np.array([j < n_tune for j in range(K)] + [tune_groups] * G)
        self.expert_map = np.full(E, -1, dtype=np.int64)
        for j, e in enumerate(self.kept):
            self.expert_map[e] = j
        for g, members in enumerate(self.groups):
            for e in members:
                self.expert_map[e] = K + g
        assert np.all(self.expert_map >= 0), "every expert needs a slot"


def frequency_merge_plan(counts, n_merge: int, group: int, n_tune: Optional[int] = None):
    """Merge the n_merge least-activated experts, in groups of ``group``.

    Experts are ranked by (count descending, index ascending).  The last n_merge
    in that ranking are merged: walked from the least activated upwards, they
    are cut into consecutive groups of ``group``.  Kept experts occupy the first
    routed slots in ranking order, so the n_tune most activated kept experts are
    slots 0..n_tune-1.  This rule stands in for the clustering of Section 5.2
    (similar experts share a group), which is a later stage of this work.
    """
    counts = np.asarray(counts)
    E = len(counts)
    assert 0 <= n_merge <= E and n_merge % group == 0
    rank = sorted(range(E), key=lambda e: (-int(counts[e]), e))
    kept = rank[:E - n_merge]
    tail = rank[E - n_merge:][::-1]
    groups = [tail[i:i + group] for i in range(0, n_merge, group)]
    return MergePlan(E, kept, groups, n_tune=n_tune)


def explicit_merge_plan(E: int, groups: Sequence[Sequence[int]], tune_all: bool = True):
    """Given groups; every other expert kept, in index order."""
    grouped = {e for g in groups for e in g}
    kept = [e for e in range(E) if e not in grouped]
    return MergePlan(E, kept, groups, tune_groups=tune_all)


# ------------------------------------------------------------------ merge ----

def merge_weights(alpha, members: Sequence[int]) -> np.ndarray:
    """Eq. 2 coefficients alpha_e / sum(alpha) over a group.

    A group whose alphas sum to zero (none of its experts was activated) takes
    the plain mean, the paper's "Avg." merging of Section 8.3.
    """
    a = _f64(alpha)[list(members)]
    tot = a.sum()
    if tot > 0:
        return a / tot
    return np.full(len(members), 1.0 / len(members))


def merge_experts(W, members: Sequence[int], alpha) -> np.ndarray:
    """Eq. 2: sum_e (alpha_e / sum alpha) W_e over the group, W stacked on axis 0."""
    w = merge_weights(alpha, members)
    out = np.zeros(np.shape(W)[1:], dtype=F64)
    for coef, e in zip(w, members):
        out += coef * _f64(W[e])
    return out


# ---------------------------------------------------------------- permute ----

def permute_maps(idx, gate, expert_map, S_routed: int):
    """Token -> slot buckets after gate re-routing (Section 7).

    Each (token t, choice j) is mapped to slot = expert_map[idx[t, j]].  Choices
    of one token that land on the same slot are one row of that slot, carrying
    the sum of their gates.  Rows of a slot are ordered by token; slots are laid
    out back to back (offsets = exclusive prefix sum of the row counts).

    Returns offsets [S+1], perm_token [N], perm_gate [N] and inv [T, k] where
    inv[t, j] = p for the choice that opened row p and -2 - p for a later choice
    of the same token folded into row p.
    """
    idx = np.asarray(idx)
    gate = _f64(gate)
    expert_map = np.asarray(expert_map)
    T, k = idx.shape
    rows: List[List[tuple]] = [[] for _ in range(S_routed)]   # (t, first j)
    owner = {}
    for t in range(T):
        for j in range(k):
            s = int(expert_map[idx[t, j]])
            assert 0 <= s < S_routed
            if (t, s) not in owner:
                owner[(t, s)] = j
                rows[s].append(t)
    counts = np.array([len(r) for r in rows], dtype=np.int64)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    N = int(offsets[-1])
    perm_token = np.zeros(N, dtype=np.int64)
    perm_gate = np.zeros(N, dtype=F64)
    pos = {}
    for s in range(S_routed):
        for r, t in enumerate(rows[s]):
            p = int(offsets[s]) + r
            perm_token[p] = t
            pos[(t, s)] = p
    inv = np.zeros((T, k), dtype=np.int64)
    for t in range(T):
        for j in range(k):
            s = int(expert_map[idx[t, j]])
            p = pos[(t, s)]
            perm_gate[p] += gate[t, j]
            inv[t, j] = p if owner[(t, s)] == j else -2 - p
    return offsets, perm_token, perm_gate, inv


# ------------------------------------------------------------ expert FFN ----

def sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


def swiglu_fwd(x, Wg, Wu, Wd):
    """One expert on rows x [n, d]: (a_g, a_u, h, o), o = h Wd^T, h = silu(a_g) a_u."""
    x = _f64(x)
    a_g = x @ _f64(Wg).T
    a_u = x @ _f64(Wu).T
    h = a_g * sigmoid(a_g) * a_u
    o = h @ _f64(Wd).T
    return a_g, a_u, h, o


def swiglu_bwd(x, Wg, Wu, Wd, dO, want_dw: bool):
    """Backward of one expert for output gradient dO [n, d].

    Returns dx [n, d] and, if want_dw, (dWg [I,d], dWu [I,d], dWd [d,I]) as sums
    over the rows (not means).
    """
    x, dO = _f64(x), _f64(dO)
    a_g, a_u, h, _ = swiglu_fwd(x, Wg, Wu, Wd)
    dh = dO @ _f64(Wd)
    sg = sigmoid(a_g)
    silu = a_g * sg
    da_u = dh * silu
    da_g = dh * a_u * sg * (1.0 + a_g * (1.0 - sg))
    dx = da_g @ _f64(Wg) + da_u @ _f64(Wu)
    if not want_dw:
        return dx, None
    return dx, (da_g.T @ x, da_u.T @ x, dO.T @ h)


class SlotWeights:
    """Per-slot expert weights of one layer: routed slots then shared experts."""

    def __init__(self, wg, wu, wd, tuning, n_shared: int = 0):
        self.wg, self.wu, self.wd = list(wg), list(wu), list(wd)
        self.tuning = np.asarray(tuning, dtype=bool)
        self.n_shared = n_shared
        self.S = len(self.wg)
        self.S_routed = self.S - n_shared
        assert len(self.tuning) == self.S


def _assignments(idx, expert_map, s):
    slot = np.asarray(expert_map)[np.asarray(idx)]
    return np.nonzero(slot == s)


def moe_forward(X, idx, gate, expert_map, slots: SlotWeights):
    """Y[t] = sum_j gate[t,j] FFN_{slot(t,j)}(X[t]) + sum_shared FFN_sh(X[t]).

    Each (t, j) is its own assignment here (no folding of equal slots), which by
    linearity equals the folded computation of the HIP path.
    """
    X, gate = _f64(X), _f64(gate)
    Y = np.zeros_like(X)
    for s in range(slots.S_routed):
        t, j = _assignments(idx, expert_map, s)
        if len(t) == 0:
            continue
        o = swiglu_fwd(X[t], slots.wg[s], slots.wu[s], slots.wd[s])[3]
        np.add.at(Y, t, gate[t, j][:, None] * o)
    for s in range(slots.S_routed, slots.S):
        Y += swiglu_fwd(X, slots.wg[s], slots.wu[s], slots.wd[s])[3]
    return Y


def moe_backward(X, dY, idx, gate, expert_map, slots: SlotWeights):
    """Expert-path gradients with the gates held constant.

    Returns dX [T, d], dW {slot: (dWg, dWu, dWd)} for tuning slots (zero arrays
    for a tuning slot with no rows) and dgate [T, k] = <dY[t], o_(t,j)>.
    """
    X, dY, gate = _f64(X), _f64(dY), _f64(gate)
    T, d = X.shape
    dX = np.zeros_like(X)
    dgate = np.zeros(np.shape(idx), dtype=F64)
    dW: Dict[int, tuple] = {}
    for s in range(slots.S):
        Wg, Wu, Wd = slots.wg[s], slots.wu[s], slots.wd[s]
        I = np.shape(Wg)[0]
        if s < slots.S_routed:
            t, j = _assignments(idx, expert_map, s)
            g = gate[t, j]
        else:
            t, j = np.arange(T), None
            g = np.ones(T)
        if len(t) == 0:
            if slots.tuning[s]:
                dW[s] = (np.zeros((I, d)), np.zeros((I, d)), np.zeros((d, I)))
            continue
        dO = g[:, None] * dY[t]
        dx, dw = swiglu_bwd(X[t], Wg, Wu, Wd, dO, bool(slots.tuning[s]))
        np.add.at(dX, t, dx)
        if dw is not None:
            dW[s] = dw
        if j is not None:
            o = swiglu_fwd(X[t], Wg, Wu, Wd)[3]
            dgate[t, j] = np.sum(dY[t] * o, axis=1)
    return dX, dW, dgate


def expert_utility(X, dY, idx, gate, expert_map, slots: SlotWeights, only: Optional[Sequence[int]] = None):
    """Utility of each slot's expert (Section 6.1, Eq. 3).  The summand printed
    there is garbled; read as the squared norm of the per-token gradient:
        u_s = |D_s| * sqrt((1/|D_s|) * sum_{t in D_s} ||g_{s,t}||^2),
    D_s the tokens that reach slot s and g_{s,t} the gradient of the slot's
    parameters (W_gate, W_up, W_down) from token t alone; u_s = 0 for an empty
    slot.  A token whose several choices map to the same slot reaches it once,
    with the gates of those choices summed (the gradient of one token is what
    its combined output contribution gives); shared experts take every token
    with gate 1.  Computed as the explicit per-token gradients of one expert,
    its weight gradient on a batch of one token.  With `only`, the other slots
    are left NaN.
    """
    X, dY, gate = _f64(X), _f64(dY), _f64(gate)
    T = X.shape[0]
    slot_of = np.asarray(expert_map)[np.asarray(idx)]
    u = np.zeros(slots.S, dtype=F64)
    if only is not None:
        u[:] = np.nan
    for s in (range(slots.S) if only is None else only):
        u[s] = 0.0
        if s < slots.S_routed:
            tokens = np.unique(np.nonzero(slot_of == s)[0])
            gsum = np.array([gate[t][slot_of[t] == s].sum() for t in tokens])
        else:
            tokens, gsum = np.arange(T), np.ones(T)
        if len(tokens) == 0:
            continue
        sq = 0.0
        for t, g in zip(tokens, gsum):
            _, (dWg, dWu, dWd) = swiglu_bwd(X[t:t + 1], slots.wg[s], slots.wu[s], slots.wd[s],
                                            g * dY[t:t + 1], True)
            sq += np.sum(dWg ** 2) + np.sum(dWu ** 2) + np.sum(dWd ** 2)
        n = len(tokens)
        u[s] = n * np.sqrt(sq / n)
    return u


def expert_utility_rank_one(X, dY, idx, gate, expert_map, slots: SlotWeights):
    """The utility of expert_utility (Eq. 3, same reading, same token sets and
    summed gates) without forming the per-token gradients: each of them is a
    sum of three rank-one matrices, dW_down = dO_t h_t^T, dW_gate = da_g,t x_t^T,
    dW_up = da_u,t x_t^T, and the Frobenius norm of an outer product a b^T is
    ||a|| ||b||, so ||g_t||^2 = ||dO_t||^2 ||h_t||^2 + (||da_g,t||^2 +
    ||da_u,t||^2) ||x_t||^2.  One batched pass per slot; for full-size layers,
    where forming T * k gradients of size 3 I d is out of reach.
    """
    X, dY, gate = _f64(X), _f64(dY), _f64(gate)
    T = X.shape[0]
    slot_of = np.asarray(expert_map)[np.asarray(idx)]
    u = np.zeros(slots.S, dtype=F64)
    for s in range(slots.S):
        if s < slots.S_routed:
            t_all, j_all = np.nonzero(slot_of == s)
            tokens = np.unique(t_all)
            gsum = np.zeros(T)
            np.add.at(gsum, t_all, gate[t_all, j_all])
            gsum = gsum[tokens]
        else:
            tokens, gsum = np.arange(T), np.ones(T)
        n = len(tokens)
        if n == 0:
            continue
        x = X[tokens]
        dO = gsum[:, None] * dY[tokens]
        a_g, a_u, h, _ = swiglu_fwd(x, slots.wg[s], slots.wu[s], slots.wd[s])
        dh = dO @ _f64(slots.wd[s])
        sg = sigmoid(a_g)
        da_u = dh * a_g * sg
        da_g = dh * a_u * sg * (1.0 + a_g * (1.0 - sg))
        sq = (np.sum(dO ** 2, axis=1) * np.sum(h ** 2, axis=1)
              + (np.sum(da_g ** 2, axis=1) + np.sum(da_u ** 2, axis=1)) * np.sum(x ** 2, axis=1))
        u[s] = n * np.sqrt(np.sum(sq) / n)
    return u


def expert_grad_columns(x, Wg, Wu, Wd, dO, cols):
    """Slices of one expert's weight gradients along the intermediate index:
    (dWg[cols, :], dWu[cols, :], dWd[:, cols]) for rows x [n, d] and output
    gradient dO [n, d].  Column c of the intermediate layer only needs
    a_g[:, c], a_u[:, c] and dH[:, c], so a few columns are cheap at any n.
    """
    x, dO = _f64(x), _f64(dO)
    cols = list(cols)
    Wg_c, Wu_c, Wd_c = _f64(Wg)[cols], _f64(Wu)[cols], _f64(Wd)[:, cols]
    a_g = x @ Wg_c.T
    a_u = x @ Wu_c.T
    sg = sigmoid(a_g)
    h = a_g * sg * a_u
    dh = dO @ Wd_c
    da_u = dh * a_g * sg
    da_g = dh * a_u * sg * (1.0 + a_g * (1.0 - sg))
    return da_g.T @ x, da_u.T @ x, dO.T @ h


# ------------------------------------- layer-aware merging (Section 5) ----

def merge_budget(counts, tuning, total_tokens, B_non: int, eps: float = 1e-12):
    """Merging budget of each layer, Section 5.1, Eq. 1.

    counts [L, E] activation counts of every layer, tuning [L, E] bool (True =
    tuning expert), B_non the participant's total number of non-tuning slots.
    Layer l (0-based here, the paper's l = l0 + 1) weighs
        b_l = (L - l0) / v_l,   v_l = max(Var_e f_e, eps),   f_e = counts / T
    (population variance over all E experts of the layer), and its share of the
    budget is B_non * b_l / sum_k b_k.  The paper floors the share and leaves the
    rest unassigned; here the floor is clamped to [min(1, n_l), n_l] (n_l the
    layer's non-tuning experts: a layer with any of them needs one group, and
    cannot have more groups than experts) and the difference to B_non is settled
    one slot at a time: while short, +1 to the layer with the largest
    share - B_l that is below n_l (ties: lower layer); while over, -1 to the
    layer with the smallest share - B_l that is above its floor (ties: higher
    layer).  With no clamp binding this is the largest-remainder rule.
    Returns (B [L] int64, share [L] float64).
    """
    counts = _f64(counts)
    tuning = np.asarray(tuning, dtype=bool)
    L, E = counts.shape
    f = counts / float(total_tokens)
    v = np.maximum(f.var(axis=1), eps)
    b = np.array([(L - l0) / v[l0] for l0 in range(L)])
    share = B_non * b / b.sum()
    n = (~tuning).sum(axis=1)
    lo = np.minimum(1, n)
    B = np.clip(np.floor(share).astype(np.int64), lo, n)
    while B.sum() < B_non:
        room = [l for l in range(L) if B[l] < n[l]]
        if not room:
            break
        best = room[0]
        for l in room[1:]:
            if share[l] - B[l] > share[best] - B[best]:
                best = l
        B[best] += 1
    while B.sum() > B_non:
        room = [l for l in range(L) if B[l] > lo[l]]
        if not room:
            break
        best = room[0]
        for l in room[1:]:
            if share[l] - B[l] <= share[best] - B[best]:
                best = l
        B[best] -= 1
    return B, share


def expert_vectors(wg, wu, wd) -> np.ndarray:
    """Each expert's parameters as one vector: W_gate, W_up, W_down row-major,
    concatenated in that order ([n, 3*I*d], float64)."""
    mats = [_f64(m) for m in (wg, wu, wd)]
    n = mats[0].shape[0]
    return np.concatenate([m.reshape(n, int(np.prod(m.shape[1:]))) for m in mats], axis=1)


def pca_features(vectors, r: int) -> np.ndarray:
    """Principal-component scores of experts, Section 5.2 (first step).

    The experts' parameter vectors are centred on their mean and decomposed,
    Xc = U S V^T (thin SVD); the scores on the r leading components are
    U[:, :r] * S[:r], components ordered by decreasing singular value.  Columns
    beyond the rank of Xc are zero.  Returns [n, r] float64.
    """
    X = _f64(vectors)
    Xc = X - X.mean(axis=0)
    U, S, _ = np.linalg.svd(Xc, full_matrices=False)
    n = X.shape[0]
    Z = np.zeros((n, r), dtype=F64)
    m = min(r, len(S))
    Z[:, :m] = U[:, :m] * S[:m]
    return Z


def unit_rows(Z) -> np.ndarray:
    """Rows scaled to unit length; a zero row stays zero."""
    Z = _f64(Z)
    nrm = np.sqrt(np.sum(Z * Z, axis=1))
    out = np.zeros_like(Z)
    nz = nrm > 0
    out[nz] = Z[nz] / nrm[nz, None]
    return out


def cosine_to_centroids(Zhat, C) -> np.ndarray:
    """cos(z, c) for unit rows z and centroids c; 0 where |c| = 0."""
    Zhat, C = _f64(Zhat), _f64(C)
    cn = np.sqrt(np.sum(C * C, axis=1))
    dots = Zhat @ C.T
    out = np.zeros_like(dots)
    nz = cn > 0
    out[:, nz] = dots[:, nz] / cn[nz]
    return out


def maximin_seeds(Z, B: int) -> List[int]:
    """Initial centroids of one layer: experts chosen by farthest-first
    traversal under cosine distance 1 - cos.  The first is the expert farthest
    from the mean (largest score norm |z|); each next one is the unchosen expert
    whose distance to its nearest chosen seed is largest.  Ties: lower index.
    (The paper initialises the centroids without saying how.)
    """
    Z = _f64(Z)
    n = Z.shape[0]
    if B == 0 or n == 0:
        return []
    Zhat = unit_rows(Z)
    nrm2 = np.sum(Z * Z, axis=1)
    first = 0
    for e in range(1, n):
        if nrm2[e] > nrm2[first]:
            first = e
    seeds = [first]
    mind = 1.0 - Zhat @ Zhat[first]
    while len(seeds) < B:
        best = -1
        for e in range(n):
            if e in seeds:
                continue
            if best < 0 or mind[e] > mind[best]:
                best = e
        seeds.append(best)
        mind = np.minimum(mind, 1.0 - Zhat @ Zhat[best])
    return seeds


def fused_kmeans(features: Sequence, budgets: Sequence[int], max_iter: int):
    """K-Means with cosine distance over every layer at once, Section 5.2.

    features[l] [n_l, r] are the layers' expert features, budgets[l] = B_l the
    number of clusters of layer l.  All sum_l B_l centroids are held together,
    each labelled with its layer; one matrix of cosine similarities between all
    experts and all centroids drives the assignment, with every expert-centroid
    pair from different layers masked out (similarity -inf: such a centroid is
    never chosen).  Features are compared as unit vectors; a centroid is the
    mean of its members' unit features (an empty cluster keeps its centroid).
    Each pass assigns every expert to its most similar centroid (ties: lower
    centroid) and stops when no label changes or after max_iter passes.
    Returns (labels: list of [n_l] int64 cluster ids within the layer,
    passes: [L] int64, the pass after which each layer's labels stopped
    changing, or max_iter).
    """
    L = len(features)
    Zh = [unit_rows(z) for z in features]
    layer_of_expert = np.concatenate([np.full(len(z), l) for l, z in enumerate(Zh)])
    first_c = np.concatenate([[0], np.cumsum(budgets)]).astype(np.int64)
    layer_of_centroid = np.concatenate([np.full(B, l) for l, B in enumerate(budgets)])
    Zall = np.concatenate(Zh, axis=0) if L else np.zeros((0, 0))
    r = Zall.shape[1] if Zall.size else 0
    C = np.zeros((int(first_c[-1]), r), dtype=F64)
    for l in range(L):
        for j, e in enumerate(maximin_seeds(features[l], int(budgets[l]))):
            C[first_c[l] + j] = Zh[l][e]
    mask = layer_of_expert[:, None] != layer_of_centroid[None, :]
    prev = None
    passes = np.full(L, max_iter, dtype=np.int64)
    it = 0
    while True:
        sim = cosine_to_centroids(Zall, C)
        sim[mask] = -np.inf
        lab = np.argmax(sim, axis=1) if sim.shape[1] else np.zeros(len(Zall), np.int64)
        it += 1
        if prev is not None:
            for l in range(L):
                sel = layer_of_expert == l
                if passes[l] == max_iter and np.array_equal(lab[sel], prev[sel]):
                    passes[l] = it
        if (prev is not None and np.array_equal(lab, prev)) or it >= max_iter:
            break
        for c in range(C.shape[0]):
            members = np.nonzero(lab == c)[0]
            if len(members):
                C[c] = Zall[members].mean(axis=0)
        prev = lab
    labels = [lab[layer_of_expert == l] - first_c[l] for l in range(L)]
    return labels, passes


# ------------------------------- quantised profiling of a layer stack ----

def dequantize_rows(q, s) -> np.ndarray:
    """q [..., rows, cols] int8 codes times their row scale s [..., rows]."""
    return _f64(q) * _f64(s)[..., None]


def rms_norm_rows(X, eps: float = 1e-6) -> np.ndarray:
    """The normalisation in front of every MoE layer of the paper's models
    (LLaMA-MoE and DeepSeek-MoE are pre-norm transformers with RMSNorm): each
    row divided by its root mean square, X / sqrt(mean(X^2) + eps), unit gain;
    a zero row stays zero (also with eps = 0)."""
    X = _f64(X)
    den = np.sqrt(np.mean(X * X, axis=1, keepdims=True) + eps)
    return X / np.where(den > 0, den, 1.0)


def quantized_stack_profile(X0, layers: Sequence[Dict], k: int, eps: float = 1e-6):
    """Profiling pass of Section 4.1 with a low-bit copy of a stack of MoE
    layers: each layer's router and expert matrices are quantised per row to
    int8 (quantize_int8_rows), and the layer runs on them — the int8 router's
    top-k and softmax gate, every routed expert (unmerged) with its dequantised
    weights q * s, and shared experts with gate 1.  The histogram of layer l
    counts its top-k selections.  A layer reads the RMS-normalised stream
    (rms_norm_rows), and layers are coupled by a residual stream,
    X_{l+1} = X_l + Y_l(rms_norm(X_l)) (the synthetic stack has no attention or
    other sublayers; without the normalisation the SwiGLU experts, quadratic in
    their input, make the stream grow without bound over a deep stack).
    layers[l]: dict with Wr [E,d], bias [E] or None, wg [E,I,d], wu [E,I,d],
    wd [E,d,I] and optionally sg, su, sd (shared experts).
    Returns (counts [L][E] int64, idx [L][T,k], gate [L][T,k], X [L+1][T,d]).
    """
    X = _f64(X0)
    counts, idxs, gates, Xs = [], [], [], [X]
    for lay in layers:
        Xn = rms_norm_rows(X, eps)
        q, s = quantize_int8_rows(lay["Wr"])
        lg = profile_logits(Xn, q, s, lay.get("bias"))
        idx = topk_select(lg, k)
        sel = np.take_along_axis(lg, idx, axis=1)
        gate = softmax_rows(sel)
        E = lg.shape[1]
        counts.append(np.bincount(idx.ravel(), minlength=E).astype(np.int64))

        def deq(W):
            W = np.asarray(W)
            n = W.shape[0]
            qq, ss = quantize_int8_rows(W.reshape(-1, W.shape[-1]))
            return dequantize_rows(qq, ss).reshape(W.shape) if n else W

        wg, wu, wd = deq(lay["wg"]), deq(lay["wu"]), deq(lay["wd"])
        n_sh = 0
        if lay.get("sg") is not None:
            sgq, suq, sdq = deq(lay["sg"]), deq(lay["su"]), deq(lay["sd"])
            n_sh = len(sgq)
            wg = list(wg) + list(sgq)
            wu = list(wu) + list(suq)
            wd = list(wd) + list(sdq)
        slots = SlotWeights(wg, wu, wd, [False] * (E + n_sh), n_shared=n_sh)
        Y = moe_forward(Xn, idx, gate, np.arange(E), slots)
        X = X + Y
        idxs.append(idx)
        gates.append(gate)
        Xs.append(X)
    return counts, idxs, gates, Xs
