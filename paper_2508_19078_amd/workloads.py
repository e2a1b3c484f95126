"""Seeded synthetic inputs for the MoE-layer hot path.

This module only draws random numbers and rounds them to the storage type. It
holds none of the method's arithmetic, and it is the one piece of code that both
the fp64 oracle (through the tests) and the HIP path (through the tests and the
benchmark) consume.

The shapes are those of the paper's two fine-tuned models at one MoE layer
(Section 8.1 names LLaMA-MoE and DeepSeek-MoE; Table 1 gives their layer and
expert counts). The activation skew that Section 2.2 (Observation 2) reports on
real data is imposed here by a per-expert logit bias, since no dataset or
trained checkpoint is available.

Every tensor comes from its own ``numpy.random.PCG64`` stream keyed by
``SeedSequence([config_id, layer, tensor_id, expert])``: a single expert's
weights can be regenerated on their own, and generation runs in parallel
threads.  Values are drawn as float32 normals, scaled, and rounded to
nearest-even into bf16 (or kept as fp32 for the fp32 workload).
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Optional, Sequence, Tuple

import numpy as np

# tensor ids of the seed key
TID_X, TID_WR, TID_BIAS, TID_WG, TID_WU, TID_WD, TID_DY, TID_SHARED = range(8)
TID_PROTO, TID_CLASS, TID_COUNTS = 8, 9, 10


@dataclass(frozen=True)
class LayerWorkload:
    """One MoE layer's shapes, storage type and routing skew."""

    name: str
    cid: int                 # first element of every seed key
    T: int                   # tokens (batch x sequence, flattened)
    d: int                   # hidden size
    E: int                   # routed experts before merging
    k: int                   # top-k
    I: int                   # expert intermediate size
    dtype: str               # "f32" or "bf16"
    n_shared: int = 0        # always-on shared experts (gate 1.0)
    bias_kind: str = "zero"  # "zero" | "normal" | "zipf"
    bias_var: float = 0.0    # variance of the normal bias
    zipf_s: float = 0.0      # exponent of the Zipf bias
    # merging: None, ("groups", ((e, e), ...)) or ("frequency", n_merge, group)
    merge: Optional[tuple] = None
    n_tune: Optional[int] = None   # kept routed experts that tune; None = all
    n_layers: int = 1

    @property
    def x_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2


def merge_count_linear(layer: int, n_layers: int = 28, max_groups: int = 12,
                       group: int = 4) -> int:
    """Experts merged at ``layer`` under a linear 0 -> 75 % schedule.

    Layer l merges group * round(max_groups * l / (n_layers - 1)) experts, i.e.
    0 at the first layer and 48 of 64 (75 %) at the last.  The ratio of
    max_groups*l/(n_layers-1) is never an exact half for 28 layers and 12 groups,
    so Python's rounding rule does not matter here.
    """
    return group * int(round(max_groups * layer / (n_layers - 1)))


WORKLOADS = {
    "tiny": LayerWorkload(
        name="tiny", cid=1, T=256, d=128, E=8, k=2, I=256, dtype="f32",
        merge=("groups", ((0, 1), (2, 3)))),
    "llama_moe": LayerWorkload(
        name="llama_moe", cid=2, T=4096, d=4096, E=16, k=4, I=688, dtype="bf16",
        bias_kind="normal", bias_var=1.5),
    "deepseek_moe": LayerWorkload(
        name="deepseek_moe", cid=3, T=8192, d=2048, E=64, k=6, I=1408,
        dtype="bf16", n_shared=2, bias_kind="normal", bias_var=1.0,
        merge=("frequency", 32, 4), n_tune=32),
    "deepseek_stack": LayerWorkload(
        name="deepseek_stack", cid=4, T=4096, d=2048, E=64, k=6, I=1408,
        dtype="bf16", bias_kind="normal", bias_var=1.0,
        merge=("linear", 4), n_tune=16, n_layers=28),
    "stress": LayerWorkload(
        name="stress", cid=5, T=32768, d=4096, E=64, k=8, I=1024, dtype="bf16",
        bias_kind="zipf", zipf_s=1.2),
}


def layer_merge_spec(w: LayerWorkload, layer: int = 0) -> Optional[tuple]:
    """The merge rule of one layer: ("groups", ...) or ("frequency", m, g)."""
    if w.merge is None:
        return None
    if w.merge[0] == "linear":
        g = w.merge[1]
        m = merge_count_linear(layer, w.n_layers, max_groups=(3 * w.E // 4) // g,
                               group=g)
        return ("frequency", m, g)   # m == 0 still ranks the slots by popularity
    return w.merge


def scaled(w: LayerWorkload, **kw) -> LayerWorkload:
    """A copy of ``w`` with some fields replaced (smaller test shapes)."""
    from dataclasses import replace
    return replace(w, **kw)


# ---------------------------------------------------------------- drawing ----

def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def round_to_bf16_bits(x32: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass
class Tensor:
    """A drawn tensor in storage form plus its exact float64 value view."""

    store: np.ndarray   # uint16 bf16 bits, or float32
    dtype: str          # "bf16" | "f32"
    shape: Tuple[int, ...] = field(default=())

    def f32(self) -> np.ndarray:
        if self.dtype == "bf16":
            return bf16_bits_to_f32(self.store).reshape(self.shape)
        return self.store.reshape(self.shape)

    def f64(self) -> np.ndarray:
        return self.f32().astype(np.float64)


def _draw(key: Sequence[int], n: int, std: float, dtype: str) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key))))
    x = rng.standard_normal(n, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return round_to_bf16_bits(x) if dtype == "bf16" else x


def draw(key: Sequence[int], shape: Tuple[int, ...], std: float, dtype: str) -> Tensor:
    n = int(np.prod(shape))
    return Tensor(_draw(key, n, std, dtype), dtype, tuple(shape))


def draw_stacked(keys: Sequence[Sequence[int]], shape: Tuple[int, ...], std: float,
                 dtype: str) -> Tensor:
    """Several equally shaped tensors, one seed key each, stacked on axis 0."""
    n = int(np.prod(shape))
    out = np.empty((len(keys), n), dtype=np.uint16 if dtype == "bf16" else np.float32)

    def one(i):
        out[i] = _draw(keys[i], n, std, dtype)

    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(one, range(len(keys))))
    return Tensor(out.reshape(-1), dtype, (len(keys),) + tuple(shape))


def router_bias(w: LayerWorkload, layer: int = 0) -> np.ndarray:
    """Per-expert logit bias (float32) that skews expert popularity."""
    if w.bias_kind == "zero":
        return np.zeros(w.E, dtype=np.float32)
    rng = np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([w.cid, layer, TID_BIAS])))
    if w.bias_kind == "normal":
        # N(0, v) with v read as the variance
        return (rng.standard_normal(w.E) * np.sqrt(w.bias_var)).astype(np.float32)
    if w.bias_kind == "zipf":
        # popularity ~ rank^-s: logit bias -s*ln(rank), ranks a seeded permutation
        ranks = rng.permutation(w.E) + 1
        return (-w.zipf_s * np.log(ranks)).astype(np.float32)
    raise ValueError(w.bias_kind)


def draw_x(w: LayerWorkload, layer: int = 0) -> Tensor:
    return draw([w.cid, layer, TID_X], (w.T, w.d), 1.0, w.dtype)


def draw_dy(w: LayerWorkload, layer: int = 0) -> Tensor:
    return draw([w.cid, layer, TID_DY], (w.T, w.d), 1.0, w.dtype)


def draw_router(w: LayerWorkload, layer: int = 0) -> Tensor:
    return draw([w.cid, layer, TID_WR], (w.E, w.d), 1.0 / np.sqrt(w.d), w.dtype)


def draw_experts(w: LayerWorkload, layer: int = 0,
                 experts: Optional[Sequence[int]] = None, shared: bool = False):
    """(W_gate [n,I,d], W_up [n,I,d], W_down [n,d,I]) for the listed experts.

    Shared experts use the same distributions with their own seed keys.
    """
    if experts is None:
        experts = range(w.n_shared if shared else w.E)
    experts = list(experts)
    base = TID_SHARED * 16 if shared else 0
    wg = draw_stacked([[w.cid, layer, base + TID_WG, e] for e in experts],
                      (w.I, w.d), 1.0 / np.sqrt(w.d), w.dtype)
    wu = draw_stacked([[w.cid, layer, base + TID_WU, e] for e in experts],
                      (w.I, w.d), 1.0 / np.sqrt(w.d), w.dtype)
    wd = draw_stacked([[w.cid, layer, base + TID_WD, e] for e in experts],
                      (w.d, w.I), 1.0 / np.sqrt(w.I), w.dtype)
    return wg, wu, wd


def draw_counts(w: LayerWorkload, layer: int = 0) -> np.ndarray:
    """Activation counts of one layer (int32 [E]): its T*k routing choices
    spread over the experts by a multinomial draw with probabilities
    proportional to exp(bias), the layer's router bias.  A stand-in for the
    profiled histogram where only the counts matter (the per-layer budget)."""
    rng = np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([w.cid, layer, TID_COUNTS])))
    b = router_bias(w, layer).astype(np.float64)
    p = np.exp(b - b.max())
    return rng.multinomial(w.T * w.k, p / p.sum()).astype(np.int32)


def expert_classes(w: LayerWorkload, layer: int, n_classes: int) -> np.ndarray:
    """A seeded class in [0, n_classes) for each of the layer's E experts."""
    rng = np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([w.cid, layer, TID_CLASS])))
    return rng.integers(0, n_classes, size=w.E)


def draw_planted_experts(w: LayerWorkload, layer: int, n_classes: int, mix: float,
                         experts: Optional[Sequence[int]] = None):
    """Experts with shared structure, for the similarity clustering of merging.

    Expert e of class c = expert_classes(...)[e] is
        W_e = sqrt(mix) * P_c + sqrt(1 - mix) * N_e
    for each of its three matrices, P_c a prototype of the class drawn like an
    expert (its own seed keys) and N_e the expert's own draw of draw_experts;
    the sum is formed in float32 and rounded once to the storage type, so the
    entries keep the variance of a plain expert.  mix = 0 gives draw_experts.
    Returns (W_gate [n,I,d], W_up [n,I,d], W_down [n,d,I]).
    """
    if experts is None:
        experts = range(w.E)
    experts = list(experts)
    cls = expert_classes(w, layer, n_classes)
    a, b = np.float32(np.sqrt(mix)), np.float32(np.sqrt(1.0 - mix))
    out = []
    for tid, shape, std in ((TID_WG, (w.I, w.d), 1.0 / np.sqrt(w.d)),
                            (TID_WU, (w.I, w.d), 1.0 / np.sqrt(w.d)),
                            (TID_WD, (w.d, w.I), 1.0 / np.sqrt(w.I))):
        n = int(np.prod(shape))
        protos = {}
        store = np.empty((len(experts), n), dtype=np.uint16 if w.dtype == "bf16" else np.float32)

        def one(i):
            e = experts[i]
            c = int(cls[e])
            x = _draw([w.cid, layer, tid, e], n, std, "f32")
            x *= b
            x += a * protos[c]
            store[i] = round_to_bf16_bits(x) if w.dtype == "bf16" else x

        for c in sorted({int(cls[e]) for e in experts}):
            protos[c] = _draw([w.cid, layer, TID_PROTO * 16 + tid, c], n, std, "f32")
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(one, range(len(experts))))
        out.append(Tensor(store.reshape(-1), w.dtype, (len(experts),) + shape))
    return tuple(out)


def to_torch(t: Tensor, device="cpu"):
    """A torch tensor of the storage dtype (bf16 or float32) with ``t``'s values."""
    import torch
    if t.dtype == "bf16":
        x = torch.from_numpy(t.store.view(np.int16).reshape(t.shape)).view(torch.bfloat16)
    else:
        x = torch.from_numpy(t.store.reshape(t.shape))
    return x.to(device)
