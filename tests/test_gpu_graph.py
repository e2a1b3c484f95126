"""The layer step captured into a HIP graph and replayed.

No entry point of the step synchronises with the host, allocates, or clears
memory with a memset (every zeroing is a kernel), so a caller can capture a
whole step -- quantise, int8 histogram, merge plan, merge, slot tables, route,
permute, grouped SwiGLU forward, combine, combine backward, grouped SwiGLU
backward, permute backward -- into one graph and replay it.  The kernels are
deterministic, so every replay must reproduce the eager step bit for bit.
Before each replay the step's outputs are overwritten with garbage (so a replay
that skipped a kernel would be caught), and eager steps with synchronisations
run between the replays."""
import pytest
import torch

from paper_2508_19078_amd import workloads as W
from paper_2508_19078_amd.layer import LayerInputs, MoELayerRunner

from gpu_harness import host, log

pytestmark = pytest.mark.gpu

CASES = {
    # a scaled DeepSeek-MoE layer: merged groups, shared experts, ragged slots
    "scaled_deepseek": lambda: W.scaled(W.WORKLOADS["deepseek_moe"], name="graph", cid=209, T=1500, d=256, I=320),
    # the fp32 path
    "tiny": lambda: W.WORKLOADS["tiny"],
    # the benchmark's layer in its launch configuration
    "deepseek_moe": lambda: W.WORKLOADS["deepseek_moe"],
}


# Outputs the step writes in full before anything in the step reads them (so
# they may be overwritten between replays): the histogram is zeroed by the step,
# idx and gate are written by the route, inv and offsets by the permutation.
# Slot maps, slot pointer tables and workspaces are never touched here: for an
# explicit grouping the maps are inputs of the step.
FULL = ("counts", "idx", "gate", "inv", "offsets", "Y", "dX", "dWg", "dWu", "dWd", "Mg", "Md")
# Per-row buffers: only the rows of the step's row space are written (routed rows
# [0, N), then T rows per shared expert); rows past them are never read.
ROWS = ("perm_token", "perm_gate", "X_perm", "A_g", "H", "O", "dO", "dX_perm")


def tensors(r):
    ts = {name: getattr(r, name) for name in FULL + ROWS}
    return {k: v for k, v in ts.items() if v is not None}


def scribble(r):
    """Overwrite the step's outputs with garbage (fill kernels on the current stream)."""
    for t in tensors(r).values():
        if t.dtype.is_floating_point:
            t.fill_(float("nan"))
        else:
            t.fill_(-7)


def snapshot(r, N):
    """Device copies of the written parts of the outputs (compared on the GPU)."""
    w = r.w
    out = {}
    for k, v in tensors(r).items():
        if k in ROWS:
            out[k + "[routed]"] = v[:N].clone()
            if k not in ("perm_token", "perm_gate", "X_perm") and w.n_shared:
                out[k + "[shared]"] = v[w.T * w.k:w.T * (w.k + w.n_shared)].clone()
        else:
            out[k] = v.clone()
    return out


def assert_same(a, b, what):
    for k in a:
        assert torch.equal(a[k].view(torch.uint8), b[k].view(torch.uint8)), f"{what}: {k} differs"


@pytest.mark.parametrize("case", list(CASES))
def test_step_graph_replays_bit_exact(case):
    w = CASES[case]()
    log(f"graph case {case}: T={w.T} d={w.d} E={w.E}+{w.n_shared} k={w.k} I={w.I} {w.dtype}")
    r = MoELayerRunner(w, LayerInputs(w))
    r.step()
    torch.cuda.synchronize()
    N = int(host(r.offsets)[-1])
    ref = snapshot(r, N)
    assert bool(torch.isfinite(ref["Y"]).all()) and bool(torch.isfinite(ref["dX"]).all())

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        r.step()
    torch.cuda.synchronize()
    for rep in range(3):
        scribble(r)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert_same(ref, snapshot(r, N), f"{case} replay {rep}")
        # eager work between replays: an eager step on the same buffers
        scribble(r)
        r.step()
        torch.cuda.synchronize()
        assert_same(ref, snapshot(r, N), f"{case} eager step after replay {rep}")
    log(f"graph case {case}: 3 replays and 3 eager steps equal the first eager step bit for bit")
    del g
