"""Benchmark of one MoE-layer fine-tuning step on one MI355X.

One step = one pass of the whole hot path over one batch:
  int8 quantise + activation histogram -> merge plan + merge + slot tables ->
  route -> permute -> grouped SwiGLU forward -> combine ->
  combine backward -> grouped SwiGLU backward -> permute backward.
Inputs are resident in HBM before timing.  Prints ONE JSON line.

Default workload: the DeepSeek-MoE-16B-shaped layer (T=8192 tokens, d=2048,
64 routed experts top-6 + 2 shared, I=1408, 32 least-activated experts merged
into 8 groups), bf16 with fp32 accumulation, synthetic seeded data.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3        # MI355X fp32 matrix/vector
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="deepseek_moe")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-sample-tokens", type=int, default=8192)
    p.add_argument("--no-cold", action="store_true", help="skip the cold-cache timing of the HBM-bound calls")
    p.add_argument("--no-merging", action="store_true", help="skip the layer-aware merging (Section 5) timing")
    p.add_argument("--no-profiling", action="store_true",
                   help="skip the quantised profiling pass over the layer stack (Section 4.1)")
    p.add_argument("--part", choices=("all", "merging", "profiling"), default="all",
                   help="merging / profiling: time only that once-per-round pass and print its JSON")
    p.add_argument("--calib-copy", action="store_true",
                   help="end with a device-to-device copy of 256 MiB (counter calibration)")
    return p.parse_args()


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "grouped_swiglu_deepseek_moe_traffic.md")


def measured_traffic(workload):
    """HBM bytes per step of the grouped SwiGLU fwd+bwd from the committed
    FETCH_SIZE / WRITE_SIZE summary, or None when it was taken on other kernel
    sources or another workload."""
    from paper_2508_19078_amd.rocprof_summary import ffn_source_hash
    if workload != "deepseek_moe" or not os.path.exists(TRAFFIC_FILE):
        return None
    kv = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line and line.split(":")[0] in ("source_sha256", "traffic_bytes"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_sha256") != ffn_source_hash():
        return None
    return float(kv["traffic_bytes"]) if "traffic_bytes" in kv else None


def ffn_flops(r, offsets):
    """Algorithmic flops of the grouped SwiGLU forward and backward: 6 d I per
    row forward; 6 d I per row backward for dX, plus 6 d I for the weight
    gradients of tuning slots."""
    w = r.w
    per = 2 * w.d * w.I
    rows = [int(offsets[s + 1] - offsets[s]) for s in range(r.S_r)] + [w.T] * w.n_shared
    fwd = sum(3 * per * n for n in rows)
    bwd = sum((3 + 3 * int(r.tuning[s])) * per * n for s, n in enumerate(rows))
    return fwd, bwd


def ffn_rows(r, offsets):
    """Row and slot counts of the step's grouped SwiGLU (the operand sizes of its
    kernels): rows of all slots and of tuning slots, slots with rows."""
    w = r.w
    rows = [int(offsets[s + 1] - offsets[s]) for s in range(r.S_r)] + [w.T] * w.n_shared
    return {"total": sum(rows), "tuning": sum(n for s, n in enumerate(rows) if r.tuning[s]),
            "slots": sum(1 for n in rows if n), "tuning_slots": sum(1 for s in range(len(rows)) if r.tuning[s]),
            "d": w.d, "I": w.I, "bytes": w.x_bytes}


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cold_hbm(r, w, st, N, reps=5):
    """The HBM-bound entry points timed one launch at a time with a cold MALL:
    a 512 MiB scrub buffer is read before every launch (outside the timed
    interval, which HIP events on the launch stream bracket).  Median of
    `reps`; algorithmic bytes per launch as in the kernel table."""
    import numpy as np
    import torch
    from paper_2508_19078_amd import api

    b = w.x_bytes
    Ntot = N + w.T * w.n_shared
    calls = {
        "route": (lambda: api.moe_route_topk(r.X, r.Wr, r.bias, w.k, r.idx, r.gate, None),
                  w.T * w.d * b + w.E * w.d * b + w.T * w.k * 8),
        "profile_hist": (lambda: api.moe_profile_hist(r.X, r.Wq, r.wscale, r.bias, w.k, r.counts),
                         w.T * w.d * b + w.E * w.d + 12 * w.E),
        "permute": (lambda: api.moe_permute(r.X, r.idx, r.gate, r.expert_map, r.S_r, r.offsets, r.perm_token,
                                            r.perm_gate, r.inv, r.X_perm, r.ws_perm, E=w.E, x_sq=r.x_sq),
                    w.T * w.d * b + N * w.d * b + w.T * w.k * 8 + N * 12 + 4 * (r.S_r + 1) + 4 * w.T),
        "combine": (lambda: api.moe_unpermute(r.layer_tables, r.O, r.inv, r.perm_gate, w.T, w.k, r.Y),
                    Ntot * w.d * b + w.T * w.d * b + w.T * w.k * 8),
        "combine_bwd": (lambda: api.moe_unpermute_bwd(r.layer_tables, r.dY, r.O, r.inv, r.offsets, r.perm_gate,
                                                      w.T, w.k, r.dO, None, dy_sq=r.dy_sq),
                        Ntot * w.d * b + w.T * w.d * b + 4 * w.T),
        "permute_bwd": (lambda: api.moe_permute_bwd(r.layer_tables, r.dX_perm, r.inv, w.T, w.k, r.dX),
                        Ntot * w.d * b + w.T * w.d * b + w.T * w.k * 4),
        # router backward (selection fixed), added to the layer's dX
        "route_bwd": (lambda: api.moe_route_bwd(r.gate, r.idx, r.dgate, r.Wr, r.dX, accumulate=True),
                      w.T * w.k * 12 + 2 * w.T * w.d * b + w.E * w.d * b),
        # expert utility (Eq. 3): the tokens' squared norms (from the permutation and
        # the combine backward), the rows' maps and the per-row norm partials the
        # backward left (8 bytes per row and dH column tile)
        "expert_utility": (lambda: api.moe_expert_utility(r.layer_tables, r.x_sq, r.dy_sq, r.perm_token,
                                                          r.perm_gate, r.offsets, w.T, w.k, r.ws_bwd, util),
                           2 * w.T * 4 + N * 8 + Ntot * 8 * -(-w.I // 256)),
    }
    util = torch.empty(r.S_r + w.n_shared, dtype=torch.float32, device="cuda")
    if r.G:
        calls["merge"] = (lambda: api.moe_merge_experts(r.w_src, r.dt, w.d, w.I, r.G, r.grp_ptr, r.grp_member,
                                                        r.alpha, r.w_dst, r.dt),
                          (w.E - r.K + r.G) * 3 * w.d * w.I * b)
    # read, not written: dirty scrub lines would be written back to HBM while
    # the timed kernel evicts them
    scrub = torch.ones(256 << 20, dtype=torch.int16, device="cuda")
    sink = torch.empty((), dtype=torch.int64, device="cuda")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    out = {}
    for name, (fn, nbytes) in calls.items():
        ts = []
        for i in range(reps):
            torch.sum(scrub, dim=0, dtype=torch.int64, out=sink)
            e0.record(st)
            fn()
            e1.record(st)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        us = float(np.median(ts)) * 1e3
        gbs = nbytes / (us * 1e-6) / 1e9
        out[name] = {"us": round(us, 1), "GBps": round(gbs, 1), "frac_hbm": round(gbs / PEAK_HBM_GBS, 3)}
    del scrub, sink
    return out


def cpu_baseline(w, n_tok):
    """The fp64 oracle on a bounded sample of the same workload (its first n_tok
    tokens; by default all of them): routing, int8 histogram, merge plan + merge (all experts), permute
    maps, forward and backward.  Reported in tokens/s of the sample."""
    import numpy as np
    import oracle as O
    from paper_2508_19078_amd import workloads as W
    from paper_2508_19078_amd.layer import LayerInputs

    ws = W.scaled(w, T=n_tok)
    inp = LayerInputs(ws)
    stages = {}
    t0 = time.perf_counter()
    tl = [t0]

    def lap(name):
        now = time.perf_counter()
        stages[name] = round(now - tl[0], 3)
        tl[0] = now

    X = inp.X.f64()
    b = inp.bias.astype(np.float64)
    idx, gate, _ = O.route_topk(X, inp.Wr.f64(), b, w.k)
    lap("route")
    q, s = O.quantize_int8_rows(inp.Wr.f32())
    counts, _, _ = O.profile_hist(X, q, s, b, w.k)
    lap("profile_hist")
    spec = W.layer_merge_spec(w, 0)
    if spec is None:
        plan = O.MergePlan(w.E, list(range(w.E)), [], n_tune=w.n_tune)
    elif spec[0] == "groups":
        plan = O.explicit_merge_plan(w.E, spec[1])
    else:
        plan = O.frequency_merge_plan(counts, spec[1], spec[2], n_tune=w.n_tune)
    wg, wu, wd = (t.f64() for t in inp.experts)
    alpha = counts / float(n_tok)
    merged = [[O.merge_experts(M, g, alpha) for M in (wg, wu, wd)] for g in plan.groups]
    lap("merge")
    sl = [[], [], []]
    for e in plan.kept:
        for i, M in enumerate((wg, wu, wd)):
            sl[i].append(M[e])
    for m in merged:
        for i in range(3):
            sl[i].append(m[i])
    tuning = list(plan.tuning)
    if w.n_shared:
        sh = [t.f64() for t in inp.shared]
        for j in range(w.n_shared):
            for i in range(3):
                sl[i].append(sh[i][j])
            tuning.append(True)
    slots = O.SlotWeights(sl[0], sl[1], sl[2], tuning, n_shared=w.n_shared)
    O.permute_maps(idx, gate, plan.expert_map, plan.S)
    lap("permute")
    O.moe_forward(X, idx, gate, plan.expert_map, slots)
    lap("forward")
    O.moe_backward(X, inp.dY.f64(), idx, gate, plan.expert_map, slots)
    lap("backward")
    dt = time.perf_counter() - t0
    # the thread pools NumPy's BLAS and OpenMP actually run with, and the
    # router, histogram and permute stages again on one thread
    pools, one_thread = None, {}
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
    except ImportError:
        threadpool_info = threadpool_limits = None
    if threadpool_info is not None:
        pools = [{"api": i.get("internal_api"), "user_api": i.get("user_api"), "threads": i.get("num_threads")}
                 for i in threadpool_info()]
        with threadpool_limits(limits=1):
            t1 = time.perf_counter()
            O.route_topk(X, inp.Wr.f64(), b, w.k)
            t2 = time.perf_counter()
            O.profile_hist(X, q, s, b, w.k)
            t3 = time.perf_counter()
            O.permute_maps(idx, gate, plan.expert_map, plan.S)
            t4 = time.perf_counter()
        one_thread = {"route": round(t2 - t1, 3), "profile_hist": round(t3 - t2, 3), "permute": round(t4 - t3, 3)}
    blas_threads = [p["threads"] for p in (pools or []) if p["user_api"] == "blas"]
    cores = max(blas_threads) if blas_threads else int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"value": round(n_tok / dt, 2), "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "cpu": cpu_model(), "cpu_count": os.cpu_count(), "thread_pools": pools,
            "omp_num_threads": os.environ.get("OMP_NUM_THREADS"), "stages_s": stages,
            "stages_1_thread_s": one_thread,
            "sample": (f"all {w.T} tokens" if n_tok >= w.T else f"first {n_tok} of {w.T} tokens")
                      + " of the same workload, full fp64 layer step "
                      f"(route, int8 histogram, plan+merge of all experts, permute, fwd+bwd); "
                      f"{dt:.1f} s on the host"}


def layer_merging(reps=3, B_non=840, r=16, n_classes=32, mix=0.6, max_iter=100):
    """Layer-aware merging of Section 5 over the 28-layer DeepSeek-MoE stack
    (64 experts per layer, d = 2048, I = 1408, top-16 tuning): the Eq. 1 budget
    and the fused PCA + K-Means clustering of the 48 non-tuning experts of every
    layer.  Expert weights are drawn on the GPU (torch's seeded generator) with
    n_classes planted classes per layer, W = sqrt(mix) P_class + sqrt(1 - mix) N;
    the counts come from the seeded counts generator.  The clustering call's
    algorithmic bytes are the non-tuning experts' parameters, read once."""
    import numpy as np
    import torch
    from paper_2508_19078_amd import api, workloads as W

    w = W.WORKLOADS["deepseek_stack"]
    dev = torch.device("cuda")
    L, E, d, I = w.n_layers, w.E, w.d, w.I
    g = torch.Generator(device=dev)
    g.manual_seed(2508190780)
    mats, ptrs = [], []
    for l in range(L):
        cls = torch.randint(0, n_classes, (E,), generator=g, device=dev)
        layer = []
        for shape, std in (((I, d), d ** -0.5), ((I, d), d ** -0.5), ((d, I), I ** -0.5)):
            proto = torch.randn((n_classes,) + shape, generator=g, device=dev)
            m = torch.randn((E,) + shape, generator=g, device=dev)
            m.mul_((1 - mix) ** 0.5).add_(proto[cls], alpha=mix ** 0.5).mul_(std)
            layer.append(m.to(torch.bfloat16))
            del proto, m
        mats.append(layer)
        for e in range(E):
            for t in layer:
                ptrs.append(t[e].data_ptr())
    w_src = torch.tensor(ptrs, dtype=torch.int64, device=dev)
    counts = np.stack([W.draw_counts(w, l) for l in range(L)])
    tun = np.zeros((L, E), dtype=np.uint8)
    for l in range(L):
        tun[l, sorted(range(E), key=lambda e: (-int(counts[l, e]), e))[:w.n_tune]] = 1
    counts_d = torch.from_numpy(counts).to(dev)
    tun_d = torch.from_numpy(tun).to(dev)
    budget = torch.empty(L, dtype=torch.int32, device=dev)
    labels = torch.empty((L, E), dtype=torch.int32, device=dev)
    iters = torch.empty(L, dtype=torch.int32, device=dev)
    ws = torch.empty(api.moe_cluster_workspace_size(L, E, d, I), dtype=torch.uint8, device=dev)
    st = torch.cuda.current_stream()
    e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    tb, tc = [], []
    for i in range(reps + 1):
        e0.record(st)
        api.moe_merge_budget(counts_d, tun_d, w.T, B_non, budget)
        e1.record(st)
        api.moe_cluster_experts(w_src, torch.bfloat16, L, E, d, I, tun_d, budget, r, max_iter, ws, labels,
                                None, iters)
        e2.record(st)
        torch.cuda.synchronize()
        if i:
            tb.append(e0.elapsed_time(e1))
            tc.append(e1.elapsed_time(e2))
    n_non = int((tun == 0).sum())
    nbytes = n_non * 3 * d * I * 2
    ms = float(np.median(tc))
    gbs = nbytes / (ms * 1e-3) / 1e9
    out = {"workload": f"deepseek_stack: {L} layers x {E} experts, d={d} I={I}, {w.n_tune} tuning per layer, "
                       f"B_non={B_non}, r={r}, {n_classes} planted classes, mix={mix}",
           "budget_us": round(float(np.median(tb)) * 1e3, 1),
           "cluster_ms": round(ms, 4), "bytes": nbytes, "GBps": round(gbs, 1),
           "frac_hbm": round(gbs / PEAK_HBM_GBS, 3), "groups": int(budget.sum().item()),
           "kmeans_passes": iters.cpu().tolist()}
    del mats, w_src, ws
    torch.cuda.empty_cache()
    return out


def profiling_stack(reps=3, workload="deepseek_stack"):
    """The quantised profiling pass of Section 4.1 over a stack of layers: the
    28-layer DeepSeek-MoE stack (64 experts, d = 2048, I = 1408, top-6, T = 4096
    tokens), or the one LLaMA-MoE layer whose profiling pass uses int8 router and
    expert weights (16 experts, d = 4096, I = 688, top-4, T = 4096): per layer
    int8 routing with the histogram on the RMS-normalised stream, permute, the
    grouped SwiGLU forward straight from the int8 expert codes, combine, and the
    residual add fused with the next layer's normalisation.  The weights are
    drawn on the GPU (torch's seeded generator, the workload's distributions)
    and quantised once; the pass is timed with HIP events per stage, median over
    `reps` passes after one warm-up."""
    import numpy as np
    import torch
    from paper_2508_19078_amd import workloads as W
    from paper_2508_19078_amd.profiling import QuantizedStack

    w = W.WORKLOADS[workload]
    dev = torch.device("cuda")
    L, E, d, I, T, k = w.n_layers, w.E, w.d, w.I, w.T, w.k
    g = torch.Generator(device=dev)
    g.manual_seed(2508190781)
    layers = []
    for l in range(L):
        rn = lambda *shape, std: (torch.randn(*shape, generator=g, device=dev) * std).to(torch.bfloat16)
        layers.append(dict(Wr=rn(E, d, std=d ** -0.5), bias=torch.from_numpy(W.router_bias(w, l)).to(dev),
                           wg=rn(E, I, d, std=d ** -0.5), wu=rn(E, I, d, std=d ** -0.5),
                           wd=rn(E, d, I, std=I ** -0.5)))
    X0 = torch.randn(T, d, generator=g, device=dev).to(torch.bfloat16)
    st = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(st)
    qs = QuantizedStack(layers, T, k)
    e1.record(st)
    torch.cuda.synchronize()
    quant_ms = e0.elapsed_time(e1)
    del layers
    torch.cuda.empty_cache()
    passes = []
    for rep in range(reps + 1):
        evs = [torch.cuda.Event(enable_timing=True)]
        names = []
        evs[0].record(st)

        def mark(name):
            ev = torch.cuda.Event(enable_timing=True)
            ev.record(st)
            evs.append(ev)
            names.append(name)
        Xout = qs.run(X0, mark)
        torch.cuda.synchronize()
        stages = {}
        for i, nm in enumerate(names):
            stages[nm] = stages.get(nm, 0.0) + evs[i].elapsed_time(evs[i + 1])
        passes.append((evs[0].elapsed_time(evs[-1]), stages))
    total = float(np.median([p[0] for p in passes[1:]]))
    stages = {nm: round(float(np.median([p[1][nm] for p in passes[1:]])), 3) for nm in passes[1][1]}
    # the whole pass captured once into a HIP graph and replayed (same kernels)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        qs.run(X0)
    graph.replay()
    torch.cuda.synchronize()
    gts = []
    for _ in range(reps):
        e0.record(st)
        graph.replay()
        e1.record(st)
        torch.cuda.synchronize()
        gts.append(e0.elapsed_time(e1))
    graph_ms = float(np.median(gts))
    del graph
    Xout = qs.run(X0)
    torch.cuda.synchronize()
    counts = qs.counts.cpu().numpy()
    # the grouped forward's algorithmic flops: 6 d I per routed row (T k rows per layer; no shared experts)
    ffn_flops = 6.0 * d * I * T * k * L
    out = {"workload": f"{w.name}: {L} layer{'s' if L > 1 else ''} x {E} experts, d={d} I={I}, T={T}, top-{k}, "
                       "int8 router and experts (per-row scales), RMS-normalised layer inputs, residual stream",
           "pass_ms": round(total, 3), "tokens_per_s": round(T / (total * 1e-3), 1),
           "graph_pass_ms": round(graph_ms, 3),
           "stages_ms": stages, "quantise_ms": round(quant_ms, 3),
           "ffn_fwd_TFLOPs": round(ffn_flops / (stages["ffn_fwd"] * 1e-3) / 1e12, 1),
           "ffn_fwd_frac_bf16_peak": round(ffn_flops / (stages["ffn_fwd"] * 1e-3) / 2.5e15, 4),
           "int8_weight_bytes": int(sum(q[n][0].numel() for q in qs.q for n in ("wg", "wu", "wd", "Wr"))),
           "hist_ok": bool((counts.sum(axis=1) == T * k).all()),
           "stream_out_rms": round(float(Xout.float().pow(2).mean().sqrt()), 3),
           "stream_finite": bool(torch.isfinite(Xout.float()).all())}
    del qs
    torch.cuda.empty_cache()
    return out


def main():
    a = parse()
    if a.gpus != 1:
        print(f"bench.py measures one GPU only (the multi-GPU path is not implemented); got --gpus {a.gpus}",
              file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch
    from paper_2508_19078_amd import api, workloads as W
    from paper_2508_19078_amd.layer import LayerInputs, MoELayerRunner

    if not os.path.exists(api.LIB_PATH):
        from paper_2508_19078_amd import build
        build.build()
    if a.part != "all":
        print(json.dumps(layer_merging() if a.part == "merging" else profiling_stack()))
        return
    w = W.WORKLOADS[a.workload]
    print(f"# workload {w.name}: drawing inputs", file=sys.stderr, flush=True)
    inp = LayerInputs(w)
    r = MoELayerRunner(w, inp)
    torch.cuda.synchronize()
    print("# inputs resident; warming up", file=sys.stderr, flush=True)
    st = torch.cuda.current_stream()

    # per-entry-point events, recorded on the stream the kernels run on
    names = ["profile", "merge", "route", "permute", "ffn_fwd", "combine", "combine_bwd", "ffn_bwd",
             "permute_bwd"]

    def timed_step(evs):
        def mark(i):
            evs[i].record(st)
        mark(0); r.profile()
        mark(1); r.merge()
        mark(2); r.route()
        mark(3)
        api.moe_permute(r.X, r.idx, r.gate, r.expert_map, r.S_r, r.offsets, r.perm_token, r.perm_gate, r.inv,
                        r.X_perm, r.ws_perm, E=w.E, x_sq=r.x_sq)
        mark(4)
        api.moe_grouped_swiglu_fwd(r.layer_tables, r.X, r.X_perm, r.offsets, w.T, w.k, r.A_g, r.A_u, r.H, r.O,
                                   r.ws_fwd)
        mark(5)
        api.moe_unpermute(r.layer_tables, r.O, r.inv, r.perm_gate, w.T, w.k, r.Y)
        mark(6)
        api.moe_unpermute_bwd(r.layer_tables, r.dY, r.O, r.inv, r.offsets, r.perm_gate, w.T, w.k, r.dO, None,
                              dy_sq=r.dy_sq)
        mark(7)
        api.moe_grouped_swiglu_bwd(r.layer_tables, r.X, r.X_perm, r.offsets, w.T, w.k, r.A_g, r.A_u, r.H, r.dO,
                                   r.dX_perm, 0, r.ws_bwd)
        mark(8)
        api.moe_permute_bwd(r.layer_tables, r.dX_perm, r.inv, w.T, w.k, r.dX)
        mark(9)

    for _ in range(a.warmup):
        r.step()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(10)] for _ in range(a.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(a.steps):
        timed_step(events[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = {n: float(np.mean([events[i][j].elapsed_time(events[i][j + 1]) for i in range(a.steps)]))
           for j, n in enumerate(names)}
    ms_step = wall * 1e3 / a.steps
    tok_s = w.T / (ms_step / 1e3)

    # the same step captured once into a HIP graph and replayed (no per-call
    # host work; the replays run the same kernels on the same buffers)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        r.step()
    graph.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(a.steps):
        graph.replay()
    torch.cuda.synchronize()
    ms_graph = (time.perf_counter() - t0) * 1e3 / a.steps
    del graph

    offsets = r.offsets.cpu().numpy()
    fl_fwd, fl_bwd = ffn_flops(r, offsets)
    ffn_ms = per["ffn_fwd"] + per["ffn_bwd"]
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    achieved = (fl_fwd + fl_bwd) / (ffn_ms * 1e-3) / 1e12
    N = int(offsets[-1])
    b = w.x_bytes
    route_bytes = w.T * w.d * b + w.E * w.d * b + w.T * w.k * 8
    permute_bytes = w.T * w.d * b + N * w.d * b + w.T * w.k * 8 + N * 12 + 4 * (r.S_r + 1) + 4 * w.T
    merge_bytes = (w.E - r.K + r.G) * 3 * w.d * w.I * b if r.G else 0
    hist_bytes = w.T * w.d * b + w.E * w.d + 12 * w.E
    gbs = lambda by, ms: round(by / (ms * 1e-3) / 1e9, 1) if ms > 0 else None
    out = {
        "metric": "MoE-layer fwd+bwd tokens/sec on 1 MI355X",
        "value": round(tok_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded normal draws shaped like the paper's workload; no dataset or checkpoint)",
        "config": {"workload": f"{w.name}: T={w.T} d={w.d} E={w.E}+{w.n_shared} shared k={w.k} I={w.I}"
                               + (f" merge={W.layer_merge_spec(w)}" if w.merge else ""),
                   "global_batch": w.T, "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "kernel": "grouped SwiGLU fwd+bwd (moe_grouped_swiglu_fwd + _bwd)",
                     "achieved": round(achieved, 1), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4), "traffic": measured_traffic(a.workload),
                     "flops_per_step": fl_fwd + fl_bwd, "ms": round(ffn_ms, 4),
                     "rows": ffn_rows(r, offsets)},
        "stages_ms": {k: round(v, 4) for k, v in per.items()},
        "graph_ms_per_step": round(ms_graph, 4),
        "hbm_kernels_GBps": {"route": gbs(route_bytes, per["route"]), "profile": gbs(hist_bytes, per["profile"]),
                             "merge": gbs(merge_bytes, per["merge"]), "permute": gbs(permute_bytes, per["permute"])},
    }
    if not a.no_cold:
        print("# cold-cache timing of the HBM-bound entry points", file=sys.stderr, flush=True)
        out["hbm_cold"] = cold_hbm(r, w, st, N)
    if not a.no_merging:
        print("# layer-aware merging over the 28-layer stack", file=sys.stderr, flush=True)
        out["layer_merging"] = layer_merging()
    if not a.no_profiling:
        # the LLaMA-MoE layer's own int8 profiling pass; the 28-layer DeepSeek-MoE stack otherwise
        pw = "llama_moe" if a.workload == "llama_moe" else "deepseek_stack"
        print(f"# quantised profiling pass ({pw})", file=sys.stderr, flush=True)
        out["profiling_stack"] = profiling_stack(workload=pw)
    if a.calib_copy:
        src = torch.ones(128 << 20, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
    if not a.no_cpu_baseline:
        print("# timing the oracle on the host", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w, a.cpu_sample_tokens)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
