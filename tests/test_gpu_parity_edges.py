"""Degenerate and limit cases of the hot path against the fp64 oracle, through
the C ABI: every token on one expert (the other slots empty), k = E, a single
token, all logits equal (including -0.0 against +0.0), a merged group none of
whose experts is activated (Eq. 2 falls back to the mean), the router at its
limits (E = 256, k = 16), empty calls, and bit-for-bit determinism of a whole
step."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2508_19078_amd import api
from paper_2508_19078_amd import workloads as W
from paper_2508_19078_amd.layer import LayerInputs, MoELayerRunner

from gpu_harness import GAP, TOL_FFN, TOL_MERGE, OracleLayer, compare_hist, compare_topk, host, log, rel_fro, rne_bf16

pytestmark = pytest.mark.gpu

BASE = W.LayerWorkload(name="edge", cid=201, T=300, d=128, E=8, k=2, I=192, dtype="bf16",
                       merge=("groups", ((6, 7),)))


def with_bias(inp, bias):
    inp.bias = np.asarray(bias, dtype=np.float32)
    return inp


def zero_x(inp):
    x = inp.X
    inp.X = W.Tensor(np.zeros_like(x.store), x.dtype, x.shape)
    return inp


def edge_cases():
    E = BASE.E
    one = np.full(E, -30.0, dtype=np.float32)
    one[3] = 30.0
    cold = np.zeros(E, dtype=np.float32)
    cold[6:] = -60.0                      # experts 6 and 7 never selected
    tie = np.zeros(E, dtype=np.float32)
    tie[1::2] = -0.0
    return {
        "one_expert": (W.scaled(BASE, name="one_expert", cid=202, k=1), lambda i: with_bias(i, one)),
        "k_equals_E": (W.scaled(BASE, name="k_equals_E", cid=203, k=E), None),
        "single_token": (W.scaled(BASE, name="single_token", cid=204, T=1), None),
        "all_ties": (W.scaled(BASE, name="all_ties", cid=205), lambda i: with_bias(zero_x(i), tie)),
        "cold_group": (W.scaled(BASE, name="cold_group", cid=206, k=2), lambda i: with_bias(i, cold)),
    }


CASES = edge_cases()


class EdgeRun:
    def __init__(self, name):
        w, mod = CASES[name]
        log(f"edge {name}: T={w.T} d={w.d} E={w.E} k={w.k} I={w.I}")
        inp = LayerInputs(w)
        if mod is not None:
            inp = mod(inp)
        self.w, self.name = w, name
        self.ref = ref = OracleLayer(w, inp)
        r = MoELayerRunner(w, inp)
        self.r = r
        idx8 = torch.full((w.T, w.k), -1, dtype=torch.int32, device="cuda")
        r.profile(idx8=idx8)
        api.moe_route_topk(r.X, r.Wr, r.bias, w.k, r.idx, r.gate, r.logits)
        self.idx_g, self.gate_g, self.logits_g = host(r.idx), host(r.gate), host(r.logits)
        self.counts_g, self.idx8_g = host(r.counts), host(idx8)
        r.merge(counts=torch.from_numpy(ref.counts.astype(np.int32)).cuda())
        r.forward(idx=torch.from_numpy(ref.idx.astype(np.int32)).cuda(),
                  gate=torch.from_numpy(ref.gate.astype(np.float32)).cuda())
        r.backward(dgate=True)
        torch.cuda.synchronize()


_runs = {}


@pytest.fixture(params=list(CASES))
def run(request):
    if request.param not in _runs:
        _runs[request.param] = EdgeRun(request.param)
    return _runs[request.param]


def test_edge_routing(run):
    ref, w = run.ref, run.w
    if run.name == "all_ties":
        # every logit equal: the lowest indices win, gates uniform
        np.testing.assert_array_equal(run.idx_g, np.tile(np.arange(w.k), (w.T, 1)))
        np.testing.assert_allclose(run.gate_g, 1.0 / w.k, rtol=1e-6)
        np.testing.assert_array_equal(ref.idx, run.idx_g)
        np.testing.assert_array_equal(run.counts_g, ref.counts)
        return
    excl, bad = compare_topk(run.idx_g, run.logits_g, ref.idx, ref.logits, w.k)
    assert bad == 0 and excl <= 1
    assert compare_hist(run.counts_g, run.idx8_g, ref, w.k, w.E) <= 1
    np.testing.assert_array_equal(run.counts_g, ref.counts)
    if run.name == "k_equals_E":
        sm = np.exp(ref.logits - ref.logits.max(1, keepdims=True))
        sm /= sm.sum(1, keepdims=True)
        np.testing.assert_allclose(np.take_along_axis(sm, run.idx_g, 1), run.gate_g, rtol=1e-5, atol=1e-7)


def test_edge_merge(run):
    ref, r = run.ref, run.r
    np.testing.assert_array_equal(host(r.expert_map), ref.plan.expert_map)
    for g in range(len(ref.plan.groups)):
        for got, exact in zip((r.Mg[g], r.Mu[g], r.Md[g]), ref.merged[g]):
            assert rel_fro(host(got), rne_bf16(exact)) <= TOL_MERGE
    if run.name == "cold_group":
        assert ref.counts[6] == 0 and ref.counts[7] == 0
        mean = 0.5 * (host(r.Wg[6]) + host(r.Wg[7]))
        assert rel_fro(host(r.Mg[0]), rne_bf16(mean)) <= TOL_MERGE


def test_edge_forward_backward(run):
    ref, r = run.ref, run.r
    Y = ref.forward()
    dX, dW, dgate = ref.backward()
    e_y, e_dx = rel_fro(host(r.Y), Y), rel_fro(host(r.dX), dX)
    slots = r.tuning_slots
    got = np.concatenate([np.concatenate([host(r.dWg[i]).ravel(), host(r.dWu[i]).ravel(), host(r.dWd[i]).ravel()])
                          for i in range(len(slots))])
    exp = np.concatenate([np.concatenate([dW[s][0].ravel(), dW[s][1].ravel(), dW[s][2].ravel()]) for s in slots])
    e_dw = rel_fro(got, exp)
    log(f"{run.name}: Y {e_y:.2e} dX {e_dx:.2e} dW {e_dw:.2e}")
    assert e_y <= TOL_FFN and e_dx <= TOL_FFN and e_dw <= TOL_FFN
    for i, s in enumerate(slots):                 # slots without rows: exactly zero
        if all(np.all(a == 0) for a in dW[s]):
            assert not r.dWg[i].any() and not r.dWu[i].any() and not r.dWd[i].any()
    if run.name == "one_expert":
        offs = host(r.offsets)
        assert (np.diff(offs) > 0).sum() == 1 and offs[-1] == run.w.T


def test_edge_route_backward(run):
    """Router backward on the degenerate routings (k = E, one expert, ties)."""
    from test_gpu_parity import route_bwd_check
    e_alone, e_acc = route_bwd_check(run.w, run.r, run.ref, 993)
    log(f"{run.name}: route bwd {e_alone:.2e} / {e_acc:.2e}")
    assert e_alone <= TOL_FFN and e_acc <= TOL_FFN


# Token counts that reach each tile size of the persistent router on a
# 256-CU MI355X: 32-token tiles below 64 tokens per CU, 64-token tiles from
# there, 128-token tiles from 128 per CU (ragged last tiles), each with a
# router of one or two 32-expert groups and k from 1 to 16.
PERSISTENT_ROUTER = {
    "tile32_E20_k16": (1000, 256, 20, 16),
    "tile64_E64_k1": (20000, 384, 64, 1),
    "tile128_E20_k5": (33000, 256, 20, 5),
    "tile128_E64_k16": (32845, 128, 64, 16),
}


@pytest.mark.parametrize("name", list(PERSISTENT_ROUTER))
def test_router_tile_sizes(name):
    """Routing (idx, gate, logits), the int8 histogram with its top-k sets, and
    the profiling route (histogram, idx and gate) against the oracle at every
    tile size of the persistent router."""
    T, d, E, k = PERSISTENT_ROUTER[name]
    w = W.LayerWorkload(name=name, cid=211, T=T, d=d, E=E, k=k, I=64, dtype="bf16", bias_kind="normal",
                        bias_var=1.0)
    inp = LayerInputs(w, with_experts=False)
    ref = OracleLayer(w, inp, with_ffn_weights=False)
    log(f"persistent router {name}: T={T} d={d} E={E} k={k}")
    X, Wr = W.to_torch(inp.X, "cuda"), W.to_torch(inp.Wr, "cuda")
    bias = torch.from_numpy(inp.bias).cuda()
    i32 = lambda *s: torch.full(s, -1, dtype=torch.int32, device="cuda")
    f32 = lambda *s: torch.full(s, float("nan"), dtype=torch.float32, device="cuda")
    idx, gate, logits = i32(T, k), f32(T, k), f32(T, E)
    api.moe_route_topk(X, Wr, bias, k, idx, gate, logits)
    Wq = torch.empty(E, d, dtype=torch.int8, device="cuda")
    sc = torch.empty(E, dtype=torch.float32, device="cuda")
    api.moe_quantize_int8(Wr, Wq, sc)
    counts, idx8 = torch.zeros(E, dtype=torch.int32, device="cuda"), i32(T, k)
    api.moe_profile_hist(X, Wq, sc, bias, k, counts, idx8)
    counts2, idx8b, gate8 = torch.zeros(E, dtype=torch.int32, device="cuda"), i32(T, k), f32(T, k)
    api.moe_profile_route(X, Wq, sc, bias, k, counts2, idx8b, gate8)
    torch.cuda.synchronize()
    excl, bad = compare_topk(host(idx), host(logits), ref.idx, ref.logits, k)
    log(f"  route: {excl} of {T} tokens in the tie window, {bad} mismatched")
    assert bad == 0 and excl <= max(2, T // 1000)
    np.testing.assert_allclose(host(logits), ref.logits, rtol=0, atol=2e-5 * max(1.0, np.abs(ref.logits).max()))
    keep = O.topk_gap(ref.logits, k) >= GAP
    np.testing.assert_allclose(host(gate)[keep], ref.gate[keep], rtol=1e-5, atol=1e-7)
    excl8 = compare_hist(host(counts), host(idx8), ref, k, E)
    log(f"  histogram: {excl8} tokens in the tie window, the rest bit-exact")
    # the profiling route: same histogram and sets, gates of the int8 logits
    np.testing.assert_array_equal(host(counts2), host(counts))
    np.testing.assert_array_equal(host(idx8b), host(idx8))
    keep8 = O.topk_gap(ref.logits8, k) >= GAP
    g8 = O.softmax_rows(np.take_along_axis(ref.logits8, np.asarray(ref.idx8), axis=1))
    np.testing.assert_allclose(host(gate8)[keep8], g8[keep8], rtol=1e-5, atol=1e-7)


def test_router_limits():
    """E = 256 experts, k = 16: the largest router the ABI accepts."""
    w = W.LayerWorkload(name="router_max", cid=207, T=777, d=256, E=256, k=16, I=64, dtype="bf16",
                        bias_kind="normal", bias_var=1.0)
    inp = LayerInputs(w, with_experts=False)
    ref = OracleLayer(w, inp, with_ffn_weights=False)
    X, Wr = W.to_torch(inp.X, "cuda"), W.to_torch(inp.Wr, "cuda")
    bias = torch.from_numpy(inp.bias).cuda()
    idx = torch.empty(w.T, w.k, dtype=torch.int32, device="cuda")
    gate = torch.empty(w.T, w.k, dtype=torch.float32, device="cuda")
    logits = torch.empty(w.T, w.E, dtype=torch.float32, device="cuda")
    api.moe_route_topk(X, Wr, bias, w.k, idx, gate, logits)
    Wq = torch.empty(w.E, w.d, dtype=torch.int8, device="cuda")
    sc = torch.empty(w.E, dtype=torch.float32, device="cuda")
    counts = torch.zeros(w.E, dtype=torch.int32, device="cuda")
    api.moe_quantize_int8(Wr, Wq, sc)
    idx8 = torch.full((w.T, w.k), -1, dtype=torch.int32, device="cuda")
    api.moe_profile_hist(X, Wq, sc, bias, w.k, counts, idx8)
    excl, bad = compare_topk(host(idx), host(logits), ref.idx, ref.logits, w.k)
    assert bad == 0 and excl <= 2
    c = host(counts)
    assert c.sum() == w.T * w.k
    excl8 = compare_hist(c, host(idx8), ref, w.k, w.E)
    log(f"router limits: {excl} / {excl8} tokens in the tie windows")


def test_empty_calls_launch_nothing():
    """T = 0 is a no-op for every per-token entry point (outputs untouched)."""
    d, E, k = 64, 8, 2
    X = torch.empty(0, d, dtype=torch.bfloat16, device="cuda")      # T = 0 (may have no storage)
    Wr = torch.zeros(E, d, dtype=torch.bfloat16, device="cuda")
    idx = torch.full((1, k), -7, dtype=torch.int32, device="cuda")
    gate = torch.full((1, k), -7.0, dtype=torch.float32, device="cuda")
    assert api.moe_route_topk(X, Wr, None, k, idx, gate, None) == 0
    Wq = torch.zeros(E, d, dtype=torch.int8, device="cuda")
    sc = torch.ones(E, dtype=torch.float32, device="cuda")
    counts = torch.full((E,), 5, dtype=torch.int32, device="cuda")
    assert api.moe_profile_hist(X, Wq, sc, None, k, counts) == 0
    torch.cuda.synchronize()
    assert (host(idx) == -7).all() and (host(counts) == 5).all()


def test_backward_without_tokens_zeroes_weight_gradients():
    """T = 0 with every per-token buffer NULL: a non-accumulating backward
    writes zero weight gradients (only offsets and the workspace are read);
    an accumulating one leaves them as they are."""
    d, I, S_r, n_sh, k = 128, 64, 3, 1, 2
    dt = torch.bfloat16
    S = S_r + n_sh
    Wg = torch.randn(S, I, d, device="cuda").to(dt)
    Wu = torch.randn(S, I, d, device="cuda").to(dt)
    Wd = torch.randn(S, d, I, device="cuda").to(dt)
    dWg = torch.full((S, I, d), 3.0, device="cuda")
    dWu = torch.full((S, I, d), 3.0, device="cuda")
    dWd = torch.full((S, d, I), 3.0, device="cuda")
    tun = [0, 2, 3]                                    # slot 1 frozen
    dw = lambda t: [t[s] if s in tun else None for s in range(S)]
    lay = api.LayerTables(d, I, dt, S_r, n_sh, list(Wg), list(Wu), list(Wd), dw(dWg), dw(dWu), dw(dWd))
    offsets = torch.zeros(S_r + 1, dtype=torch.int32, device="cuda")
    ws = torch.empty(api.moe_grouped_swiglu_bwd_workspace_size(lay, 0, k), dtype=torch.uint8, device="cuda")
    assert api.moe_grouped_swiglu_bwd(lay, None, None, offsets, 0, k, None, None, None, None, None, True, ws) == 0
    torch.cuda.synchronize()
    assert bool((dWg == 3).all() and (dWu == 3).all() and (dWd == 3).all())
    assert api.moe_grouped_swiglu_bwd(lay, None, None, offsets, 0, k, None, None, None, None, None, False, ws) == 0
    torch.cuda.synchronize()
    for t in (dWg, dWu, dWd):
        for s in range(S):
            assert bool((t[s] == 0).all()) == (s in tun), s
        assert bool((t[1] == 3).all())


def test_utility_of_a_layer_without_routed_slots():
    """A layer of shared experts only (S_routed = 0): forward, backward and the
    expert utility with the permutation maps NULL (the routed part of the row
    space is never read), against the fp64 oracle."""
    T, d, I, k, n_sh = 300, 128, 192, 2, 2
    dt = torch.bfloat16
    g = torch.Generator(device="cpu").manual_seed(611)
    X = (torch.randn(T, d, generator=g)).to(dt).cuda()
    dY = (torch.randn(T, d, generator=g) * 0.1).to(dt).cuda()
    Wg = (torch.randn(n_sh, I, d, generator=g) / d ** 0.5).to(dt).cuda()
    Wu = (torch.randn(n_sh, I, d, generator=g) / d ** 0.5).to(dt).cuda()
    Wd = (torch.randn(n_sh, d, I, generator=g) / I ** 0.5).to(dt).cuda()
    dWg, dWu, dWd = (torch.zeros(n_sh, *t.shape[1:], device="cuda") for t in (Wg, Wu, Wd))
    lay = api.LayerTables(d, I, dt, 0, n_sh, list(Wg), list(Wu), list(Wd), list(dWg), list(dWu), list(dWd))
    Rt = T * (k + n_sh)
    A_g, A_u, H = (torch.zeros(Rt, I, dtype=dt, device="cuda") for _ in range(3))
    Ob = torch.zeros(Rt, d, dtype=dt, device="cuda")
    dO = torch.zeros(Rt, d, dtype=dt, device="cuda")
    for i in range(n_sh):
        dO[T * k + i * T:T * k + (i + 1) * T] = dY
    dXp = torch.zeros(Rt, d, dtype=dt, device="cuda")
    offsets = torch.zeros(1, dtype=torch.int32, device="cuda")
    wsf = torch.empty(api.moe_grouped_swiglu_fwd_workspace_size(lay, T, k), dtype=torch.uint8, device="cuda")
    wsb = torch.empty(api.moe_grouped_swiglu_bwd_workspace_size(lay, T, k), dtype=torch.uint8, device="cuda")
    assert api.moe_grouped_swiglu_fwd(lay, X, None, offsets, T, k, A_g, A_u, H, Ob, wsf) == 0
    assert api.moe_grouped_swiglu_bwd(lay, X, None, offsets, T, k, A_g, A_u, H, dO, dXp, False, wsb) == 0
    x_sq = X.float().pow(2).sum(1).contiguous()
    dy_sq = dY.float().pow(2).sum(1).contiguous()
    u = torch.full((n_sh,), -1.0, dtype=torch.float32, device="cuda")
    assert api.moe_expert_utility(lay, x_sq, dy_sq, None, None, offsets, T, k, wsb, u) == 0
    torch.cuda.synchronize()
    f64 = lambda t: host(t.float()).astype(np.float64)
    slots = O.SlotWeights([f64(w) for w in Wg], [f64(w) for w in Wu], [f64(w) for w in Wd], [True] * n_sh,
                          n_shared=n_sh)
    exp = O.expert_utility(f64(X), f64(dY), np.zeros((T, k), dtype=np.int64), np.ones((T, k)),
                           np.zeros(1, dtype=np.int64), slots)
    got = host(u)
    log(f"shared-only utility: got {got}, oracle {exp}")
    assert rel_fro(got, exp) <= TOL_FFN and bool(np.all(got > 0))


def test_permute_with_debug_range_checks(monkeypatch):
    """FLUXMOE_DEBUG_CHECKS: moe_permute copies idx and expert_map to the host
    and range-checks them before launching; valid maps give the same result as
    without the checks (the rejection of invalid maps is a host-only test)."""
    w = W.scaled(W.WORKLOADS["deepseek_moe"], name="dbg", cid=209, T=300, d=64, I=64)
    inp = LayerInputs(w)
    r = MoELayerRunner(w, inp)
    r.profile()
    r.merge()
    r.route()
    r.forward()
    torch.cuda.synchronize()
    plain = [host(t).copy() for t in (r.offsets, r.perm_token, r.inv, r.X_perm)]
    monkeypatch.setenv("FLUXMOE_DEBUG_CHECKS", "1")
    r.forward()
    torch.cuda.synchronize()
    for a, t in zip(plain, (r.offsets, r.perm_token, r.inv, r.X_perm)):
        np.testing.assert_array_equal(a, host(t))


def test_step_with_debug_range_checks(monkeypatch):
    """FLUXMOE_DEBUG_CHECKS over the whole step and the utility: with valid maps
    every output equals the run without the checks; maps with an entry out of
    range are refused with MOE_ERR_ARG before anything is launched.  Each bad
    entry still lies inside its buffer's allocation (a row just past the routed
    rows, offsets[0] = 1, the token index T), so nothing could read outside
    device memory even if a check were missing."""
    w = W.scaled(W.WORKLOADS["deepseek_moe"], name="dbg2", cid=210, T=700, d=128, I=128)
    inp = LayerInputs(w)
    r = MoELayerRunner(w, inp)
    util = torch.empty(r.S_r + w.n_shared, dtype=torch.float32, device="cuda")

    def run():
        r.step()
        r.backward(dgate=True)
        assert api.moe_expert_utility(r.layer_tables, r.x_sq, r.dy_sq, r.perm_token, r.perm_gate, r.offsets, w.T,
                                      w.k, r.ws_bwd, util) == 0
        torch.cuda.synchronize()
        return [host(t).copy() for t in (r.counts, r.idx, r.offsets, r.inv, r.Y, r.dX, r.dgate, r.dWg, util,
                                         r.x_sq, r.dy_sq)]

    plain = run()
    monkeypatch.setenv("FLUXMOE_DEBUG_CHECKS", "1")
    for a, b in zip(plain, run()):
        np.testing.assert_array_equal(a, b)
    R = w.T * w.k
    bad_inv = r.inv.clone()
    bad_inv[3, 1] = R + 3                  # a shared row of the same buffers, past the routed ones
    L = api.lib()
    for name, call in (
            ("moe_unpermute", lambda: api.moe_unpermute(r.layer_tables, r.O, bad_inv, r.perm_gate, w.T, w.k, r.Y)),
            ("moe_unpermute_bwd", lambda: api.moe_unpermute_bwd(r.layer_tables, r.dY, r.O, bad_inv, r.offsets,
                                                                r.perm_gate, w.T, w.k, r.dO, None)),
            ("moe_permute_bwd", lambda: api.moe_permute_bwd(r.layer_tables, r.dX_perm, bad_inv, w.T, w.k, r.dX))):
        with pytest.raises(RuntimeError, match="inv"):
            call()
        log(f"debug check refused a bad inv in {name}")
    bad_off = r.offsets.clone()
    bad_off[0] = 1
    with pytest.raises(RuntimeError, match="offsets"):
        api.moe_grouped_swiglu_fwd(r.layer_tables, r.X, r.X_perm, bad_off, w.T, w.k, r.A_g, r.A_u, r.H, r.O,
                                   r.ws_fwd)
    with pytest.raises(RuntimeError, match="offsets"):
        api.moe_grouped_swiglu_bwd(r.layer_tables, r.X, r.X_perm, bad_off, w.T, w.k, r.A_g, r.A_u, r.H, r.dO,
                                   r.dX_perm, False, r.ws_bwd)
    bad_tok = r.perm_token.clone()
    bad_tok[0] = w.T
    with pytest.raises(RuntimeError, match="perm_token"):
        api.moe_expert_utility(r.layer_tables, r.x_sq, r.dy_sq, bad_tok, r.perm_gate, r.offsets, w.T, w.k,
                               r.ws_bwd, util)
    torch.cuda.synchronize()
    assert L.moe_last_error()


def test_step_is_deterministic():
    """Two runs of the whole step on the same inputs agree bit for bit."""
    w = W.scaled(W.WORKLOADS["deepseek_moe"], name="det", cid=208, T=1500, d=256, I=320)
    inp = LayerInputs(w)
    outs = []
    for _ in range(2):
        r = MoELayerRunner(w, inp)
        r.step()
        r.backward(dgate=True)
        torch.cuda.synchronize()
        outs.append([host(t) for t in (r.counts, r.idx, r.gate, r.Y, r.dX, r.dgate, r.dWg, r.dWu, r.dWd)])
    for a, b in zip(*outs):
        np.testing.assert_array_equal(a, b)


RB_SHAPES = {
    # name: (T, d, E, k, dtype): k up to 16, E up to 256, partial column groups
    "k16_partial_group": (500, 1032, 64, 16, torch.bfloat16),
    "fp32_odd_tokens": (97, 520, 40, 3, torch.float32),
    "E256_k16": (777, 256, 256, 16, torch.bfloat16),
    "E65_short_rows": (33, 64, 65, 2, torch.bfloat16),
}


@pytest.mark.parametrize("name", list(RB_SHAPES))
def test_route_backward_shapes(name):
    """moe_route_bwd on shapes the layer workloads do not reach: k = 16, E up
    to 256, rows that end inside a group of column chunks (d = 1032 bf16,
    d = 520 fp32, d = 64), an odd token count.  Inputs: selection and gates as
    the forward would hand them over (distinct experts per token, softmax
    gates), dgate ~ N(0, 1)."""
    T, d, E, k, dt = RB_SHAPES[name]
    rng = np.random.default_rng([995, T, d, E, k])
    Wr = torch.from_numpy((rng.standard_normal((E, d)) / np.sqrt(d)).astype(np.float32)).to(dt)
    idx = np.argsort(rng.random((T, E)), axis=1)[:, :k].astype(np.int32)
    z = rng.standard_normal((T, k))
    gate = (np.exp(z) / np.exp(z).sum(1, keepdims=True)).astype(np.float32)
    dgate = rng.standard_normal((T, k)).astype(np.float32)
    base = torch.from_numpy(rng.standard_normal((T, d)).astype(np.float32)).to(dt).cuda()
    log(f"route bwd {name}: T={T} d={d} E={E} k={k} {dt}")
    g_t, i_t, dg_t, W_t = (torch.from_numpy(gate).cuda(), torch.from_numpy(idx).cuda(),
                           torch.from_numpy(dgate).cuda(), Wr.cuda())
    out = torch.full((T, d), float("nan"), dtype=dt, device="cuda")
    acc = base.clone()
    assert api.moe_route_bwd(g_t, i_t, dg_t, W_t, out, accumulate=False) == 0
    assert api.moe_route_bwd(g_t, i_t, dg_t, W_t, acc, accumulate=True) == 0
    torch.cuda.synchronize()
    _, ref = O.route_topk_backward(host(W_t), idx, gate, dgate)
    e1, e2 = rel_fro(host(out), ref), rel_fro(host(acc), host(base) + ref)
    log(f"  dX {e1:.2e}, accumulated {e2:.2e}")
    tol = 1e-5 if dt == torch.float32 else TOL_FFN
    assert e1 <= tol and e2 <= tol
