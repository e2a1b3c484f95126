"""HIP path vs the fp64 oracle, element by element, on shapes the oracle
finishes in seconds: several row tiles per slot, ragged row counts, N and K
tails (I = 200, 384 and 688), merged and frozen slots, a shared expert, and the
fp32 workload; then eight seeded irregular layers (d and I multiples of 8 but
not of 16 or of a tile, tens of tokens to a thousand, one to 79 experts, up to
two shared experts, everything but a few experts merged, both storage types).
Everything goes through the C ABI."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2508_19078_amd import workloads as W
from paper_2508_19078_amd.layer import LayerInputs, MoELayerRunner

from gpu_harness import (GAP, TOL_FFN, TOL_MERGE, OracleLayer, compare_hist, compare_topk, host, log, rel_fro,
                         rne_bf16)

pytestmark = pytest.mark.gpu

CASES = {
    "tiny": W.WORKLOADS["tiny"],
    "small_mix": W.LayerWorkload(name="small_mix", cid=101, T=700, d=192, E=12, k=3, I=200, dtype="bf16",
                                 n_shared=1, bias_kind="normal", bias_var=1.0, merge=("frequency", 4, 2),
                                 n_tune=5),
    "small_llama": W.scaled(W.WORKLOADS["llama_moe"], name="small_llama", cid=102, T=520, d=512),
    "small_deepseek": W.scaled(W.WORKLOADS["deepseek_moe"], name="small_deepseek", cid=103, T=1030, d=256,
                               I=384),
}


def _irregular(n, seed=25081907):
    """Seeded layers off every tile grid: d, I multiples of 8 in [24, 1032] and
    [24, 792], T in [1, 1100], E in [1, 79], k up to min(E, 8), 0-2 shared
    experts, the frequency merge of n_merge = g * j experts in groups of g, a
    zero, normal or Zipf router bias; cases 2 and 6 in fp32."""
    import numpy as np
    rng = np.random.default_rng(seed)
    out = {}
    for i in range(n):
        f32 = i in (2, 6)
        d = 8 * int(rng.integers(3, 130))
        I = 8 * int(rng.integers(3, 100))
        E = int(rng.integers(1, 80))
        k = int(rng.integers(1, min(E, 8) + 1))
        T = int(rng.integers(1, 1100))
        ns = int(rng.integers(0, 3))
        merge, n_tune = None, None
        if E >= 4 and rng.random() < 0.7:
            g = int(rng.integers(2, 5))
            m = g * int(rng.integers(1, E // g + 1))
            merge, n_tune = ("frequency", m, g), int(rng.integers(0, E - m + 1))
        bias = ["zero", "normal", "zipf"][int(rng.integers(0, 3))]
        name = f"irregular{i}"
        out[name] = W.LayerWorkload(name=name, cid=300 + i, T=T, d=d, E=E, k=k, I=I,
                                    dtype="f32" if f32 else "bf16", n_shared=ns, bias_kind=bias,
                                    bias_var=1.0 if bias == "normal" else 0.0,
                                    zipf_s=1.2 if bias == "zipf" else 0.0, merge=merge, n_tune=n_tune)
    return out


CASES.update(_irregular(8))


class Run:
    def __init__(self, name):
        w = CASES[name]
        log(f"case {name}: T={w.T} d={w.d} E={w.E} k={w.k} I={w.I} {w.dtype}")
        self.w = w
        inp = LayerInputs(w)
        self.ref = OracleLayer(w, inp)
        r = MoELayerRunner(w, inp)
        self.r = r
        idx8 = torch.full((w.T, w.k), -1, dtype=torch.int32, device="cuda")
        r.profile(idx8=idx8)
        self.idx8_g = host(idx8)
        api_logits = r.logits
        from paper_2508_19078_amd import api
        api.moe_route_topk(r.X, r.Wr, r.bias, w.k, r.idx, r.gate, api_logits)
        self.idx_g, self.gate_g, self.logits_g = host(r.idx), host(r.gate), host(r.logits)
        self.q_g, self.s_g, self.counts_g = host(r.Wq), host(r.wscale), host(r.counts)
        # downstream stages run on the oracle's routing and histogram
        r.merge(counts=torch.from_numpy(self.ref.counts.astype(np.int32)).cuda())
        idx = torch.from_numpy(self.ref.idx.astype(np.int32)).cuda()
        gate = torch.from_numpy(self.ref.gate.astype(np.float32)).cuda()
        r.forward(idx=idx, gate=gate)
        r.backward(dgate=True)
        torch.cuda.synchronize()
        log(f"case {name}: gpu done")


_runs = {}


@pytest.fixture(params=list(CASES))
def run(request):
    if request.param not in _runs:
        _runs[request.param] = Run(request.param)
    return _runs[request.param]


def test_router(run):
    ref, w = run.ref, run.w
    excl, bad = compare_topk(run.idx_g, run.logits_g, ref.idx, ref.logits, w.k)
    log(f"router: excluded {excl} of {w.T}, mismatches {bad}")
    assert bad == 0 and excl <= max(2, w.T // 1000)
    np.testing.assert_allclose(run.logits_g, ref.logits, rtol=0, atol=2e-5 * max(1.0, np.abs(ref.logits).max()))
    keep = O.topk_gap(ref.logits, w.k) >= GAP
    np.testing.assert_allclose(run.gate_g[keep], ref.gate[keep], rtol=1e-5, atol=1e-7)


def test_quantizer_bit_exact(run):
    np.testing.assert_array_equal(run.q_g, run.ref.q)
    np.testing.assert_array_equal(run.s_g.astype(np.float32), run.ref.s)


def test_histogram_bit_exact(run):
    """Per-token int8 top-k sets and the histogram, bit-exact outside the
    near-tie window (the excluded tokens' choices removed on both sides)."""
    ref, w = run.ref, run.w
    excl = compare_hist(run.counts_g, run.idx8_g, ref, w.k, w.E)
    log(f"histogram: {excl} of {w.T} tokens in the tie window")
    assert excl <= max(2, w.T // 1000)
    assert run.counts_g.sum() == w.T * w.k


def test_merge_plan_bit_exact(run):
    ref, r = run.ref, run.r
    plan = ref.plan
    np.testing.assert_array_equal(host(r.expert_map), plan.expert_map)
    K = len(plan.kept)
    src = host(r.slot_src)
    np.testing.assert_array_equal(src[:K], plan.kept)
    np.testing.assert_array_equal(src[K:], w_e := np.arange(len(plan.groups)) + run.w.E)
    if plan.groups:
        gp = host(r.grp_ptr)
        gm = host(r.grp_member)
        for g, members in enumerate(plan.groups):
            np.testing.assert_array_equal(gm[gp[g]:gp[g + 1]], members)
    np.testing.assert_allclose(host(r.alpha), ref.alpha, rtol=1e-6)


def test_merged_weights(run):
    ref, r = run.ref, run.r
    if not ref.plan.groups:
        pytest.skip("no merging in this workload")
    for g in range(len(ref.plan.groups)):
        for got, exact in zip((r.Mg[g], r.Mu[g], r.Md[g]), ref.merged[g]):
            got = host(got)
            if run.w.dtype == "bf16":
                err = rel_fro(got, rne_bf16(exact))
            else:
                err = rel_fro(got, exact)
                assert err <= 1e-6
            assert err <= TOL_MERGE, (g, err)


def test_permute_maps_bit_exact(run):
    ref, r, w = run.ref, run.r, run.w
    offsets, ptok, pgate, inv = O.permute_maps(ref.idx, ref.gate, ref.plan.expert_map, ref.plan.S)
    np.testing.assert_array_equal(host(r.offsets), offsets)
    N = int(offsets[-1])
    np.testing.assert_array_equal(host(r.perm_token)[:N], ptok)
    np.testing.assert_array_equal(host(r.inv), inv)
    np.testing.assert_allclose(host(r.perm_gate)[:N], pgate, rtol=2e-6)
    np.testing.assert_array_equal(host(r.X_perm[:N]), ref.X[ptok])


def test_forward_output(run):
    ref, r = run.ref, run.r
    Y = ref.forward()
    err = rel_fro(host(r.Y), Y)
    log(f"Y rel err {err:.2e}")
    assert err <= (1e-5 if run.w.dtype == "f32" else TOL_FFN)


def test_backward_outputs(run):
    ref, r, w = run.ref, run.r, run.w
    dX, dW, dgate = ref.backward()
    e_dx = rel_fro(host(r.dX), dX)
    e_dg = rel_fro(host(r.dgate), dgate)
    slots = r.tuning_slots
    assert sorted(dW) == slots
    got = np.concatenate([np.concatenate([host(r.dWg[i]).ravel(), host(r.dWu[i]).ravel(), host(r.dWd[i]).ravel()])
                          for i in range(len(slots))])
    exp = np.concatenate([np.concatenate([dW[s][0].ravel(), dW[s][1].ravel(), dW[s][2].ravel()]) for s in slots])
    e_dw = rel_fro(got, exp)
    log(f"dX {e_dx:.2e} dW {e_dw:.2e} dgate {e_dg:.2e}")
    tol = 1e-5 if w.dtype == "f32" else TOL_FFN
    assert e_dx <= tol and e_dw <= tol and e_dg <= tol
    for i, s in enumerate(slots):                 # empty tuning slots: exactly zero
        if all(np.all(a == 0) for a in dW[s]):
            assert not host(r.dWg[i]).any() and not host(r.dWu[i]).any() and not host(r.dWd[i]).any()


def test_backward_accumulates_weight_gradients(run):
    """accumulate_dw = 1 adds the step's weight gradients to what dW holds: a
    second identical backward doubles every element exactly (fp32 x + x)."""
    r = run.r
    once = [host(t).copy() for t in (*r.dWg, *r.dWu, *r.dWd)]
    r.backward(dgate=False, accumulate_dw=True)
    torch.cuda.synchronize()
    twice = [host(t) for t in (*r.dWg, *r.dWu, *r.dWd)]
    r.backward(dgate=False, accumulate_dw=False)    # leave the single-pass values for other tests
    torch.cuda.synchronize()
    for a, b in zip(once, twice):
        np.testing.assert_array_equal(b, 2 * a)


def route_bwd_check(w, r, ref, seed):
    """moe_route_bwd (selection fixed) against the oracle on seeded dgate, alone
    and added to the expert path's dX (accumulate = 1).  Returns the errors."""
    rng = np.random.default_rng([w.cid, seed])
    dgate = rng.normal(size=(w.T, w.k)).astype(np.float32)
    gate32 = ref.gate.astype(np.float32)
    _, dX_ref = O.route_topk_backward(host(r.Wr), ref.idx, gate32, dgate)
    dev = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(dt).cuda()
    idx_t, gate_t, dg_t = dev(ref.idx.astype(np.int32), torch.int32), dev(gate32, torch.float32), \
        dev(dgate, torch.float32)
    out = torch.empty_like(r.dX)
    from paper_2508_19078_amd import api
    assert api.moe_route_bwd(gate_t, idx_t, dg_t, r.Wr, out, accumulate=False) == 0
    base = r.dX.clone()
    acc = base.clone()
    assert api.moe_route_bwd(gate_t, idx_t, dg_t, r.Wr, acc, accumulate=True) == 0
    torch.cuda.synchronize()
    return rel_fro(host(out), dX_ref), rel_fro(host(acc), host(base) + dX_ref)


def test_route_backward(run):
    e_alone, e_acc = route_bwd_check(run.w, run.r, run.ref, 991)
    log(f"route bwd: dX_router {e_alone:.2e}, accumulated {e_acc:.2e}")
    tol = 1e-5 if run.w.dtype == "f32" else TOL_FFN
    assert e_alone <= tol and e_acc <= tol


def utility_check(w, r, ref, only=None):
    """moe_expert_utility after the run's backward against the oracle (all
    slots, or `only`).  Returns (GPU utilities, oracle utilities)."""
    from paper_2508_19078_amd import api
    u = torch.full((r.S_r + w.n_shared,), -1.0, dtype=torch.float32, device="cuda")
    assert api.moe_expert_utility(r.layer_tables, r.x_sq, r.dy_sq, r.perm_token, r.perm_gate, r.offsets, w.T, w.k,
                                  r.ws_bwd, u) == 0
    torch.cuda.synchronize()
    exp = O.expert_utility(ref.X, ref.dY, ref.idx, ref.gate, ref.plan.expert_map, ref.slots, only=only)
    return host(u), exp


def test_expert_utility(run):
    got, exp = utility_check(run.w, run.r, run.ref)
    err = rel_fro(got, exp)
    log(f"utility: rel err {err:.2e} over {len(exp)} slots")
    assert err <= (1e-5 if run.w.dtype == "f32" else TOL_FFN)
    np.testing.assert_array_equal(got == 0, exp == 0)      # exactly the empty slots are 0
    rel = np.abs(got - exp) / np.maximum(exp, 1e-30)
    assert np.all(rel[exp > 0] <= 5e-2)
    # a second call on the same workspace (its block counter was set back to
    # zero by the first) gives the same utilities bit for bit
    from paper_2508_19078_amd import api
    w, r = run.w, run.r
    u2 = torch.full((r.S_r + w.n_shared,), -1.0, dtype=torch.float32, device="cuda")
    assert api.moe_expert_utility(r.layer_tables, r.x_sq, r.dy_sq, r.perm_token, r.perm_gate, r.offsets, w.T, w.k,
                                  r.ws_bwd, u2) == 0
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(u2), got)
