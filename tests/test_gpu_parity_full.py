"""Full-size parity: the LLaMA-MoE, DeepSeek-MoE and stress layers at their real
shapes, and the 28-layer DeepSeek stack, through the same entry points, kernels
and launch configuration the benchmark times.

Whatever the oracle computes cheaply at full size is compared whole: router
top-k (bit-exact outside the near-tie window), int8 quantiser, histogram, merge
plan, merged weights, permutation maps.  The FFN outputs are sampled: Y, dX and
dgate on a seeded sample of tokens (each depends only on its own token), and
dW on a few intermediate columns of a few tuning slots, which the oracle
computes over all of the slot's rows (``expert_grad_columns``).  Properties that
hold at any size are checked on the whole output (sum of counts, exact zeros of
empty tuning slots, finite values)."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2508_19078_amd import api
from paper_2508_19078_amd import workloads as W
from paper_2508_19078_amd.layer import LayerInputs, MoELayerRunner

from gpu_harness import (GAP, TOL_FFN, TOL_MERGE, OracleLayer, compare_topk, host, log, rel_fro,
                         rne_bf16)

pytestmark = pytest.mark.gpu

N_SAMPLE = 96          # sampled tokens for Y / dX / dgate
FULL = ["llama_moe", "deepseek_moe", "stress"]


def sample_cols(I, rng):
    """Intermediate columns at tile edges and inside: 0, 127, 128, 255, 256, I-1, two random."""
    c = {0, min(127, I - 1), min(128, I - 1), min(255, I - 1), min(256, I - 1), I - 1}
    c |= set(int(x) for x in rng.integers(0, I, 2))
    return sorted(c)


class FullRun:
    def __init__(self, w, layer=0, with_ffn=True):
        log(f"full {w.name} layer {layer}: T={w.T} d={w.d} E={w.E} k={w.k} I={w.I} drawing")
        self.w, self.layer = w, layer
        inp = LayerInputs(w, layer)
        self.ref = ref = OracleLayer(w, inp, layer)
        log("oracle routing / plan done; GPU")
        r = MoELayerRunner(w, inp, layer=layer)
        self.r = r
        r.profile()
        api.moe_route_topk(r.X, r.Wr, r.bias, w.k, r.idx, r.gate, r.logits)
        self.idx_g, self.gate_g, self.logits_g = host(r.idx), host(r.gate), host(r.logits)
        self.q_g, self.s_g, self.counts_g = host(r.Wq), host(r.wscale), host(r.counts)
        r.merge(counts=torch.from_numpy(ref.counts.astype(np.int32)).cuda())
        rng = np.random.default_rng([w.cid, layer, 777])
        self.sample = np.sort(rng.choice(w.T, size=min(N_SAMPLE, w.T), replace=False))
        self.cols = sample_cols(w.I, rng)
        if with_ffn:
            idx = torch.from_numpy(ref.idx.astype(np.int32)).cuda()
            gate = torch.from_numpy(ref.gate.astype(np.float32)).cuda()
            r.forward(idx=idx, gate=gate)
            r.backward(dgate=True)
            torch.cuda.synchronize()
            s = torch.from_numpy(self.sample).cuda()
            self.Y_s = host(r.Y[s])
            self.dX_s = host(r.dX[s])
            self.dgate_s = host(r.dgate[s])
            self.Y_finite = bool(torch.isfinite(r.Y.float()).all())
            self.dX_finite = bool(torch.isfinite(r.dX.float()).all())
        torch.cuda.synchronize()
        log(f"full {w.name} layer {layer}: GPU done")


_runs = {}


def get_run(name):
    if name not in _runs:
        _runs.clear()                       # one full-size layer resident at a time
        torch.cuda.empty_cache()
        _runs[name] = FullRun(W.WORKLOADS[name])
    return _runs[name]


@pytest.fixture(params=FULL)
def run(request):
    return get_run(request.param)


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


def test_full_expert_utility(run):
    """Utility at full size: the oracle on the two smallest non-empty slots,
    every slot non-negative and zero exactly when empty, and linear in dY
    (a second backward with 2 dY doubles every utility)."""
    from test_gpu_parity import utility_check
    w, r, ref = run.w, run.r, run.ref
    rows = np.array([len(np.unique(np.nonzero(ref.plan.expert_map[ref.idx] == s)[0])) for s in range(r.S_r)]
                    + [w.T] * w.n_shared)
    small = [int(s) for s in np.argsort(np.where(rows > 0, rows, 1 << 30), kind="stable")[:2]]
    got, exp = utility_check(w, r, ref, only=small)
    log(f"utility {w.name}: slots {small} ({rows[small]} rows) got {got[small]} oracle {exp[small]}")
    np.testing.assert_allclose(got[small], exp[small], rtol=2e-2)
    assert np.all(got >= 0) and np.array_equal(got == 0, rows == 0)
    r.dY.mul_(2)
    r.backward()
    torch.cuda.synchronize()
    got2, _ = utility_check(w, r, ref, only=[])
    r.dY.div_(2)
    r.backward()
    torch.cuda.synchronize()
    np.testing.assert_allclose(got2, 2 * got, rtol=1e-5)


def test_full_quantizer_and_histogram(run):
    ref, w = run.ref, run.w
    np.testing.assert_array_equal(run.q_g, ref.q)
    np.testing.assert_array_equal(run.s_g.astype(np.float32), ref.s)
    assert run.counts_g.sum() == w.T * w.k
    excl = O.topk_gap(ref.logits8, w.k) < GAP
    log(f"histogram {w.name}: {int(excl.sum())} tokens in the tie window")
    adj = np.bincount(ref.idx8[excl].ravel(), minlength=w.E)
    assert np.abs(run.counts_g - ref.counts).sum() <= 2 * adj.sum()
    if excl.sum() == 0:
        np.testing.assert_array_equal(run.counts_g, ref.counts)


def test_full_plan_and_merge(run):
    ref, r = run.ref, run.r
    plan = ref.plan
    np.testing.assert_array_equal(host(r.expert_map), plan.expert_map)
    np.testing.assert_array_equal(host(r.slot_src)[:len(plan.kept)], plan.kept)
    np.testing.assert_allclose(host(r.alpha), ref.alpha, rtol=1e-6)
    for g in range(len(plan.groups)):
        for got, exact in zip((r.Mg[g], r.Mu[g], r.Md[g]), ref.merged[g]):
            assert rel_fro(host(got), rne_bf16(exact)) <= TOL_MERGE


def test_full_permute_maps(run):
    ref, r = run.ref, run.r
    offsets, ptok, pgate, inv = O.permute_maps(ref.idx, ref.gate, ref.plan.expert_map, ref.plan.S)
    np.testing.assert_array_equal(host(r.offsets), offsets)
    N = int(offsets[-1])
    np.testing.assert_array_equal(host(r.perm_token)[:N], ptok)
    np.testing.assert_array_equal(host(r.inv), inv)
    np.testing.assert_allclose(host(r.perm_gate)[:N], pgate, rtol=2e-6)
    # gathered rows: a seeded sample of positions, bit-exact
    pos = np.random.default_rng(5).choice(N, size=min(512, N), replace=False)
    got = host(r.X_perm[torch.from_numpy(pos).cuda()])
    np.testing.assert_array_equal(got, ref.X[ptok[pos]])


def test_full_forward_sampled(run):
    Y = run.ref.forward(tokens=run.sample)
    err = rel_fro(run.Y_s, Y)
    log(f"{run.w.name}: Y (sampled) rel err {err:.2e}")
    assert run.Y_finite and err <= TOL_FFN


def test_full_backward_sampled(run):
    ref, r, w = run.ref, run.r, run.w
    dX, _, dgate = ref.backward(tokens=run.sample)
    e_dx, e_dg = rel_fro(run.dX_s, dX), rel_fro(run.dgate_s, dgate)
    # dW on sampled columns of the most, median and least loaded tuning slots
    slots = r.tuning_slots
    rows = [len(ref.slot_rows(s)[0]) for s in slots]
    order = np.argsort(rows)
    pick = sorted({slots[order[-1]], slots[order[len(order) // 2]], slots[order[0]]})
    got, exp = [], []
    cols = torch.tensor(run.cols).cuda()
    for s in pick:
        i = slots.index(s)
        g_dwg, g_dwu, g_dwd = ref.grad_columns(s, run.cols)
        got += [host(r.dWg[i][cols]).ravel(), host(r.dWu[i][cols]).ravel(), host(r.dWd[i][:, cols]).ravel()]
        exp += [g_dwg.ravel(), g_dwu.ravel(), g_dwd.ravel()]
        if rows[slots.index(s)] == 0:
            assert not r.dWg[i].any() and not r.dWu[i].any() and not r.dWd[i].any()
    e_dw = rel_fro(np.concatenate(got), np.concatenate(exp))
    log(f"{w.name}: dX {e_dx:.2e} dgate {e_dg:.2e} dW cols {e_dw:.2e} (slots {pick}, rows "
        f"{[rows[slots.index(s)] for s in pick]})")
    assert run.dX_finite
    assert e_dx <= TOL_FFN and e_dg <= TOL_FFN and e_dw <= TOL_FFN


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
    api.moe_quantize_int8(Wr, Wq, sc)
    api.moe_profile_hist(X, Wq, sc, bias, k, counts)
    counts_g = host(counts)
    excl = O.topk_gap(ref.logits8, k) < GAP
    adj = np.bincount(ref.idx8[excl].ravel(), minlength=E)
    assert counts_g.sum() == T * k
    assert np.abs(counts_g - ref.counts).sum() <= 2 * adj.sum(), layer
    if excl.sum() == 0:
        np.testing.assert_array_equal(counts_g, ref.counts)

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
    _runs.clear()
    torch.cuda.empty_cache()
    groups = 0
    for layer in range(w.n_layers):
        groups += stack_layer_merge(w, layer)
        torch.cuda.empty_cache()
    log(f"stack: 28 layers, {groups} merged groups checked")
    assert groups == sum(W.layer_merge_spec(w, l)[1] // 4 for l in range(w.n_layers))


@pytest.mark.parametrize("layer", [0, 9, 18, 27])
def test_stack_layer_ffn_sampled(layer):
    w = W.WORKLOADS["deepseek_stack"]
    _runs.clear()
    torch.cuda.empty_cache()
    run = FullRun(w, layer)
    test_full_forward_sampled(run)
    test_full_backward_sampled(run)
    del run
