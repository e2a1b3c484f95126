"""Full-size parity: the LLaMA-MoE, DeepSeek-MoE and stress layers at their real
shapes, and layers of the 28-layer DeepSeek stack, through the same entry
points, kernels and launch configuration the benchmark times.

Every output is compared whole against the fp64 oracle on the same inputs:
router top-k (bit-exact outside the near-tie window) and gates, int8 quantiser,
per-token int8 top-k sets and histogram (bit-exact outside the window), merge
plan, merged weights, permutation maps and every gathered row, the combine
output Y, dX, dgate and the full weight gradients of every tuning slot, the
router backward, and the expert utility of every slot.  Downstream stages run
on the oracle's routing and histogram, so they compare like with like.  The
stress layer's fp64 oracle takes about a minute of the host's cores."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2508_19078_amd import api
from paper_2508_19078_amd import workloads as W
from paper_2508_19078_amd.layer import LayerInputs, MoELayerRunner

from gpu_harness import (GAP, TOL_FFN, TOL_MERGE, OracleLayer, compare_hist, compare_topk, host, log, rel_fro,
                         rne_bf16)

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(600)]

FULL = ["llama_moe", "deepseek_moe", "stress"]


def bits(t: torch.Tensor) -> np.ndarray:
    """Raw storage bits of a device tensor, on the host."""
    t = t.detach().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


class FullRun:
    """One full-size layer: the GPU's outputs copied to the host, and the
    oracle's routing, plan and merge.  The oracle's forward and backward are
    computed once, on first use."""

    def __init__(self, w, layer=0):
        log(f"full {w.name} layer {layer}: T={w.T} d={w.d} E={w.E}+{w.n_shared} k={w.k} I={w.I} drawing")
        self.w, self.layer = w, layer
        self.inp = inp = LayerInputs(w, layer)
        self.ref = ref = OracleLayer(w, inp, layer)
        log("oracle routing / plan / merge done; GPU")
        r = MoELayerRunner(w, inp, layer=layer)
        self.r = r
        idx8 = torch.full((w.T, w.k), -1, dtype=torch.int32, device="cuda")
        r.profile(idx8=idx8)
        api.moe_route_topk(r.X, r.Wr, r.bias, w.k, r.idx, r.gate, r.logits)
        self.idx_g, self.gate_g, self.logits_g = host(r.idx), host(r.gate), host(r.logits)
        self.q_g, self.s_g, self.counts_g, self.idx8_g = host(r.Wq), host(r.wscale), host(r.counts), host(idx8)
        r.merge(counts=torch.from_numpy(ref.counts.astype(np.int32)).cuda())
        idx = torch.from_numpy(ref.idx.astype(np.int32)).cuda()
        gate = torch.from_numpy(ref.gate.astype(np.float32)).cuda()
        r.forward(idx=idx, gate=gate)
        r.backward(dgate=True)
        torch.cuda.synchronize()
        self.Y = host(r.Y)
        self.dX = host(r.dX)
        self.dgate = host(r.dgate)
        log(f"full {w.name} layer {layer}: GPU done")
        self._fwd = self._bwd = None

    def oracle_forward(self):
        if self._fwd is None:
            log(f"oracle forward over all {self.w.T} tokens")
            self._fwd = self.ref.forward()
        return self._fwd

    def oracle_backward(self):
        if self._bwd is None:
            log(f"oracle backward over all {self.w.T} tokens")
            self._bwd = self.ref.backward()
            log("oracle backward done")
        return self._bwd


@pytest.fixture(scope="module", params=FULL)
def run(request):
    """Module scope: the tests of one workload run together, one full-size
    layer resident at a time."""
    torch.cuda.empty_cache()
    fr = FullRun(W.WORKLOADS[request.param])
    yield fr
    del fr
    torch.cuda.empty_cache()


def test_full_router(run):
    ref, w = run.ref, run.w
    excl, bad = compare_topk(run.idx_g, run.logits_g, ref.idx, ref.logits, w.k)
    log(f"router {w.name}: excluded {excl} of {w.T}, mismatches {bad}")
    assert bad == 0 and excl <= max(2, w.T // 1000)
    keep = O.topk_gap(ref.logits, w.k) >= GAP
    np.testing.assert_allclose(run.gate_g[keep], ref.gate[keep], rtol=1e-5, atol=1e-7)


def test_full_route_backward(run):
    """Router backward over every token of the full-size layer."""
    from test_gpu_parity import route_bwd_check
    e_alone, e_acc = route_bwd_check(run.w, run.r, run.ref, 992)
    log(f"route bwd {run.w.name}: {e_alone:.2e} / accumulated {e_acc:.2e}")
    assert e_alone <= TOL_FFN and e_acc <= TOL_FFN


def test_full_quantizer_and_histogram(run):
    ref, w = run.ref, run.w
    np.testing.assert_array_equal(run.q_g, ref.q)
    np.testing.assert_array_equal(run.s_g.astype(np.float32), ref.s)
    excl = compare_hist(run.counts_g, run.idx8_g, ref, w.k, w.E)
    log(f"histogram {w.name}: {excl} tokens in the tie window, the rest bit-exact")


def test_full_plan_and_merge(run):
    ref, r = run.ref, run.r
    plan = ref.plan
    np.testing.assert_array_equal(host(r.expert_map), plan.expert_map)
    np.testing.assert_array_equal(host(r.slot_src)[:len(plan.kept)], plan.kept)
    np.testing.assert_allclose(host(r.alpha), ref.alpha, rtol=1e-6)
    for g in range(len(plan.groups)):
        for got, exact in zip((r.Mg[g], r.Mu[g], r.Md[g]), ref.merged[g]):
            assert rel_fro(host(got), rne_bf16(exact)) <= TOL_MERGE


def test_full_permute_maps_and_rows(run):
    """Maps bit-exact, and every gathered row of X_perm equal, bit for bit, to
    the input row the oracle's map names."""
    ref, r, w = run.ref, run.r, run.w
    offsets, ptok, pgate, inv = O.permute_maps(ref.idx, ref.gate, ref.plan.expert_map, ref.plan.S)
    np.testing.assert_array_equal(host(r.offsets), offsets)
    N = int(offsets[-1])
    np.testing.assert_array_equal(host(r.perm_token)[:N], ptok)
    np.testing.assert_array_equal(host(r.inv), inv)
    np.testing.assert_allclose(host(r.perm_gate)[:N], pgate, rtol=2e-6)
    Xs = run.inp.X.store.reshape(w.T, w.d)
    step = 16384
    for p0 in range(0, N, step):
        p1 = min(N, p0 + step)
        np.testing.assert_array_equal(bits(r.X_perm[p0:p1]), Xs[ptok[p0:p1]], err_msg=f"rows {p0}..{p1}")


def test_full_forward(run):
    Y = run.oracle_forward()
    err = rel_fro(run.Y, Y)
    log(f"{run.w.name}: Y rel err {err:.2e} over all {run.w.T} tokens")
    assert np.isfinite(run.Y).all() and err <= TOL_FFN


def test_full_backward(run):
    """dX, dgate and the weight gradients of every tuning slot, whole."""
    ref, r, w = run.ref, run.r, run.w
    dX, dW, dgate = run.oracle_backward()
    e_dx, e_dg = rel_fro(run.dX, dX), rel_fro(run.dgate, dgate)
    slots = r.tuning_slots
    assert sorted(dW) == slots
    num = den = 0.0
    worst = (0.0, None)
    for i, s in enumerate(slots):
        got = (host(r.dWg[i]), host(r.dWu[i]), host(r.dWd[i]))
        if all(np.all(a == 0) for a in dW[s]):             # empty tuning slot: exactly zero
            assert not any(g.any() for g in got), s
            continue
        n2 = sum(float(np.sum((g - e) ** 2)) for g, e in zip(got, dW[s]))
        d2 = sum(float(np.sum(e ** 2)) for e in dW[s])
        num, den = num + n2, den + d2
        e_s = np.sqrt(n2 / d2)
        worst = max(worst, (e_s, s))
        assert e_s <= TOL_FFN, (s, e_s)
    e_dw = np.sqrt(num / den)
    log(f"{w.name}: dX {e_dx:.2e} dgate {e_dg:.2e} dW {e_dw:.2e} over {len(slots)} tuning slots "
        f"(worst slot {worst[1]}: {worst[0]:.2e})")
    assert np.isfinite(run.dX).all()
    assert e_dx <= TOL_FFN and e_dg <= TOL_FFN and e_dw <= TOL_FFN


def test_full_expert_utility(run):
    """Utility of every slot (the oracle's batched rank-one route, pinned on
    the CPU against explicit per-token gradients); zero exactly when empty;
    linear in dY (a second backward with 2 dY doubles every utility)."""
    w, r, ref = run.w, run.r, run.ref
    u = torch.full((r.S_r + w.n_shared,), -1.0, dtype=torch.float32, device="cuda")
    api.moe_expert_utility(r.layer_tables, r.x_sq, r.dy_sq, r.perm_token, r.perm_gate, r.offsets, w.T, w.k, r.ws_bwd, u)
    torch.cuda.synchronize()
    got = host(u)
    exp = O.expert_utility_rank_one(ref.X, ref.dY, ref.idx, ref.gate, ref.plan.expert_map, ref.slots)
    rel = np.abs(got - exp) / np.maximum(exp, 1e-300)
    log(f"utility {w.name}: {len(exp)} slots, rel err {rel_fro(got, exp):.2e}, worst slot {rel[exp > 0].max():.2e}")
    assert np.array_equal(got == 0, exp == 0)
    assert rel_fro(got, exp) <= TOL_FFN and np.all(rel[exp > 0] <= TOL_FFN)
    r.dY.mul_(2)
    r.backward()
    api.moe_expert_utility(r.layer_tables, r.x_sq, r.dy_sq, r.perm_token, r.perm_gate, r.offsets, w.T, w.k, r.ws_bwd, u)
    torch.cuda.synchronize()
    got2 = host(u)
    r.dY.div_(2)
    r.backward()
    torch.cuda.synchronize()
    np.testing.assert_allclose(got2, 2 * got, rtol=1e-5)


# ------------------------------------------------------ 28-layer stack ----

def stack_layer_merge(w, layer):
    """Histogram, plan and merged weights of one stack layer through the C ABI.
    Only the experts that end up in a merged group are drawn and uploaded."""
    inp = LayerInputs(w, layer, with_experts=False)
    ref = OracleLayer(w, inp, layer, with_ffn_weights=False)
    dev = "cuda"
    X, Wr = W.to_torch(inp.X, dev), W.to_torch(inp.Wr, dev)
    bias = torch.from_numpy(inp.bias).to(dev)
    E, d, I, k, T = w.E, w.d, w.I, w.k, w.T
    Wq = torch.empty(E, d, dtype=torch.int8, device=dev)
    sc = torch.empty(E, dtype=torch.float32, device=dev)
    counts = torch.zeros(E, dtype=torch.int32, device=dev)
    idx8 = torch.full((T, k), -1, dtype=torch.int32, device=dev)
    api.moe_quantize_int8(Wr, Wq, sc)
    api.moe_profile_hist(X, Wq, sc, bias, k, counts, idx8)
    compare_hist(host(counts), host(idx8), ref, k, E)

    _, m, g = W.layer_merge_spec(w, layer)
    G = m // g
    zi = lambda n: torch.zeros(max(1, n), dtype=torch.int32, device=dev)
    emap, ssrc, gptr, gmem = zi(E), zi(E - m + G), zi(G + 1), zi(m)
    alpha = torch.empty(E, dtype=torch.float32, device=dev)
    api.moe_merge_plan(torch.from_numpy(ref.counts.astype(np.int32)).to(dev), m, g, T, emap, ssrc, gptr, gmem,
                       alpha)
    plan = ref.plan
    np.testing.assert_array_equal(host(emap), plan.expert_map)
    np.testing.assert_array_equal(host(ssrc)[:len(plan.kept)], plan.kept)
    np.testing.assert_allclose(host(alpha), ref.alpha, rtol=1e-6)
    if G == 0:
        return 0
    gp, gm = host(gptr), host(gmem)
    for j, members in enumerate(plan.groups):
        np.testing.assert_array_equal(gm[gp[j]:gp[j + 1]], members)
    members = sorted({e for grp in plan.groups for e in grp})
    wg, wu, wd = W.draw_experts(w, layer, experts=members)
    tg, tu, td = (W.to_torch(t, dev) for t in (wg, wu, wd))
    pos = {e: i for i, e in enumerate(members)}
    src = []
    for e in range(E):                      # experts outside every group are never read
        i = pos.get(e, 0)
        src += [tg[i].data_ptr(), tu[i].data_ptr(), td[i].data_ptr()]
    Mg, Mu, Md = (torch.empty(G, I, d, dtype=torch.bfloat16, device=dev),
                  torch.empty(G, I, d, dtype=torch.bfloat16, device=dev),
                  torch.empty(G, d, I, dtype=torch.bfloat16, device=dev))
    dst = []
    for j in range(G):
        dst += [Mg[j].data_ptr(), Mu[j].data_ptr(), Md[j].data_ptr()]
    api.moe_merge_experts(torch.tensor(src, dtype=torch.int64, device=dev), torch.bfloat16, d, I, G, gptr, gmem,
                          alpha, torch.tensor(dst, dtype=torch.int64, device=dev), torch.bfloat16)
    torch.cuda.synchronize()
    f64 = [t.f64() for t in (wg, wu, wd)]
    alpha_local = ref.alpha[members]         # alpha indexed by position in `members`
    for j, grp in enumerate(plan.groups):
        loc = [pos[e] for e in grp]
        for got, M in zip((Mg[j], Mu[j], Md[j]), f64):
            exact = O.merge_experts(M, loc, alpha_local)
            assert rel_fro(host(got), rne_bf16(exact)) <= TOL_MERGE, (layer, j)
    return G


def test_stack_all_layers_histogram_and_merge():
    w = W.WORKLOADS["deepseek_stack"]
    torch.cuda.empty_cache()
    groups = 0
    for layer in range(w.n_layers):
        groups += stack_layer_merge(w, layer)
        torch.cuda.empty_cache()
    log(f"stack: 28 layers, {groups} merged groups checked")
    assert groups == sum(W.layer_merge_spec(w, l)[1] // 4 for l in range(w.n_layers))


@pytest.mark.parametrize("layer", [0, 9, 18, 27])
def test_stack_layer_ffn(layer):
    """Whole-tensor Y, dX, dgate and dW of stack layers across the merge
    schedule (0 % merged at layer 0 to 75 % at layer 27, 16 tuning slots)."""
    w = W.WORKLOADS["deepseek_stack"]
    torch.cuda.empty_cache()
    run = FullRun(w, layer)
    test_full_forward(run)
    test_full_backward(run)
    del run
