"""Device buffers and call sequence of one MoE layer's fine-tuning step.

``MoELayerRunner`` owns the HBM-resident tensors of one layer (inputs, the
per-slot tables, every intermediate) and enqueues the C entry points on one
stream.  It is plumbing: every value is computed by libfluxmoe.

  profile()  int8 router quantisation + activation histogram (once per round)
  merge()    merge plan, Eq. 2 merge and the slot tables (once per round)
  route()    softmax top-k gate
  forward()  permute -> grouped SwiGLU forward -> combine
  backward() combine backward -> grouped SwiGLU backward -> permute backward
  step()     all of the above in that order: one pass of the whole hot path

HBM layout.  Expert weights are stacked per matrix ([E, I, d], [E, I, d],
[E, d, I]); merged groups get their own stacks and shared experts theirs.
Per-row activations use the row space of the ABI: T*k routed rows (bucketed by
slot) followed by T rows per shared expert.
"""
from __future__ import annotations

from typing import Optional

import numpy as np
import torch

from . import api
from .workloads import LayerWorkload, layer_merge_spec, draw_x, draw_dy, draw_router, draw_experts, \
    router_bias, to_torch

TORCH_DT = {"bf16": torch.bfloat16, "f32": torch.float32}


class LayerInputs:
    """Host-side draws of one layer (storage form, see workloads)."""

    def __init__(self, w: LayerWorkload, layer: int = 0, with_experts: bool = True):
        self.w, self.layer = w, layer
        self.X = draw_x(w, layer)
        self.Wr = draw_router(w, layer)
        self.bias = router_bias(w, layer)
        self.dY = draw_dy(w, layer)
        self.experts = draw_experts(w, layer) if with_experts else None
        self.shared = draw_experts(w, layer, shared=True) if (with_experts and w.n_shared) else None


def tuning_flags(w: LayerWorkload, K: int, G: int):
    """Which slots tune: the first n_tune kept slots (all kept when n_tune is
    None), merged groups only for caller-given groupings, shared experts always."""
    n_tune = K if w.n_tune is None else w.n_tune
    spec = layer_merge_spec(w, 0) if w.merge is not None else None
    groups_tune = spec is not None and spec[0] == "groups"
    return [j < n_tune for j in range(K)] + [groups_tune] * G + [True] * w.n_shared


class MoELayerRunner:
    def __init__(self, w: LayerWorkload, inputs: Optional[LayerInputs] = None, layer: int = 0,
                 device: str = "cuda"):
        self.w, self.layer, self.dev = w, layer, device
        inp = inputs if inputs is not None else LayerInputs(w, layer)
        dt = TORCH_DT[w.dtype]
        self.dt = dt
        T, d, E, k, I = w.T, w.d, w.E, w.k, w.I
        z = lambda *shape, dtype=dt: torch.empty(*shape, dtype=dtype, device=device)
        zi = lambda *shape: torch.zeros(*shape, dtype=torch.int32, device=device)

        # inputs, resident in HBM
        self.X = to_torch(inp.X, device)
        self.Wr = to_torch(inp.Wr, device)
        self.bias = torch.from_numpy(inp.bias).to(device)
        self.dY = to_torch(inp.dY, device)
        self.Wg, self.Wu, self.Wd = (to_torch(t, device) for t in inp.experts)
        if w.n_shared:
            self.Sg, self.Su, self.Sd = (to_torch(t, device) for t in inp.shared)

        # profiling
        self.Wq = z(E, d, dtype=torch.int8)
        self.wscale = z(E, dtype=torch.float32)
        self.counts = zi(E)

        # merge plan -> slots
        spec = layer_merge_spec(w, layer)
        self.spec = spec
        if spec is None:
            self.K, self.G = E, 0
        elif spec[0] == "groups":
            self.K, self.G = E - sum(len(g) for g in spec[1]), len(spec[1])
        else:
            self.K, self.G = E - spec[1], spec[1] // spec[2]
        self.S_r = self.K + self.G
        S = self.S_r + w.n_shared
        self.expert_map = zi(E)
        self.slot_src = zi(self.S_r)
        self.grp_ptr = zi(self.G + 1)
        self.grp_member = zi(max(1, E - self.K))
        self.alpha = z(E, dtype=torch.float32)
        if spec is not None and spec[0] == "groups":
            pa = api.plan_from_groups(E, spec[1])
            self.expert_map.copy_(torch.from_numpy(pa["expert_map"]))
            self.slot_src.copy_(torch.from_numpy(pa["slot_src"]))
            self.grp_ptr.copy_(torch.from_numpy(pa["grp_ptr"]))
            self.grp_member[:len(pa["grp_member"])].copy_(torch.from_numpy(pa["grp_member"]))
        elif spec is None:
            self.expert_map.copy_(torch.arange(E, dtype=torch.int32))
            self.slot_src.copy_(torch.arange(E, dtype=torch.int32))
        if self.G:
            self.Mg, self.Mu, self.Md = z(self.G, I, d), z(self.G, I, d), z(self.G, d, I)
            esz = self.Wg.element_size()
            src = []
            for e in range(E):
                src += [self.Wg[e].data_ptr(), self.Wu[e].data_ptr(), self.Wd[e].data_ptr()]
            dst = []
            for g in range(self.G):
                dst += [self.Mg[g].data_ptr(), self.Mu[g].data_ptr(), self.Md[g].data_ptr()]
            self.w_src = torch.tensor(src, dtype=torch.int64, device=device)
            self.w_dst = torch.tensor(dst, dtype=torch.int64, device=device)
        else:
            self.Mg = self.Mu = self.Md = None

        # slot tables: routed part written by moe_slot_pointers, shared part fixed here
        def table(shared_stack):
            t = torch.zeros(S, dtype=torch.int64, device=device)
            if w.n_shared:
                t[self.S_r:] = torch.tensor([shared_stack[i].data_ptr() for i in range(w.n_shared)],
                                            dtype=torch.int64)
            return t
        self.t_wg = table(self.Sg if w.n_shared else None)
        self.t_wu = table(self.Su if w.n_shared else None)
        self.t_wd = table(self.Sd if w.n_shared else None)
        self.tuning = tuning_flags(w, self.K, self.G)
        nt = sum(self.tuning)
        self.dWg = torch.zeros(nt, I, d, dtype=torch.float32, device=device)
        self.dWu = torch.zeros(nt, I, d, dtype=torch.float32, device=device)
        self.dWd = torch.zeros(nt, d, I, dtype=torch.float32, device=device)
        slots_t = [s for s in range(S) if self.tuning[s]]
        self.tuning_slots = slots_t
        dwt = lambda stack: [stack[slots_t.index(s)] if self.tuning[s] else None for s in range(S)]
        self.layer_tables = api.LayerTables(d, I, dt, self.S_r, w.n_shared, self.t_wg, self.t_wu, self.t_wd,
                                            dwt(self.dWg), dwt(self.dWu), dwt(self.dWd), device=device)

        # routing and permutation
        self.idx = zi(T, k)
        self.gate = z(T, k, dtype=torch.float32)
        self.logits = z(T, E, dtype=torch.float32)
        R, Rt = T * k, T * (k + w.n_shared)
        self.offsets = zi(self.S_r + 1)
        self.perm_token = zi(R)
        self.perm_gate = z(R, dtype=torch.float32)
        self.inv = zi(T, k)
        self.X_perm = z(R, d)
        # per-token ||X||^2 and ||dY||^2 (written by the permutation and the
        # combine backward; the expert utility reads them)
        self.x_sq = z(T, dtype=torch.float32)
        self.dy_sq = z(T, dtype=torch.float32)
        self.ws_perm = torch.empty(api.moe_permute_workspace_size(T, k, self.S_r), dtype=torch.uint8,
                                   device=device)
        # forward / backward activations
        self.A_g, self.A_u, self.H = z(Rt, I), z(Rt, I), z(Rt, I)
        self.O = z(Rt, d)
        self.Y = z(T, d)
        self.dO = z(Rt, d)
        self.dgate = z(T, k, dtype=torch.float32)
        self.dX_perm = z(Rt, d)
        self.dX = z(T, d)
        self.ws_fwd = torch.empty(api.moe_grouped_swiglu_fwd_workspace_size(self.layer_tables, T, k),
                                  dtype=torch.uint8, device=device)
        self.ws_bwd = torch.empty(api.moe_grouped_swiglu_bwd_workspace_size(self.layer_tables, T, k),
                                  dtype=torch.uint8, device=device)

    # ------------------------------------------------------------ stages --
    def profile(self, idx8: Optional[torch.Tensor] = None):
        """idx8 [T,k] int32, if given, receives the int8 router's top-k sets."""
        w = self.w
        api.moe_quantize_int8(self.Wr, self.Wq, self.wscale)
        self.counts.zero_()
        api.moe_profile_hist(self.X, self.Wq, self.wscale, self.bias, w.k, self.counts, idx8)

    def merge(self, counts: Optional[torch.Tensor] = None):
        """Plan from `counts` (default: this layer's histogram), merge, slot tables."""
        w = self.w
        counts = self.counts if counts is None else counts
        if self.spec is not None and self.spec[0] == "frequency":
            api.moe_merge_plan(counts, self.spec[1], self.spec[2], w.T, self.expert_map, self.slot_src,
                               self.grp_ptr, self.grp_member, self.alpha)
        else:
            api.moe_activation_frequency(counts, w.T, self.alpha)
        if self.G:
            api.moe_merge_experts(self.w_src, self.dt, w.d, w.I, self.G, self.grp_ptr, self.grp_member,
                                  self.alpha, self.w_dst, self.dt)
        merged = (self.Mg, self.Mu, self.Md)
        api.moe_slot_pointers(self.slot_src, self.S_r, w.E, w.d, w.I, self.dt, (self.Wg, self.Wu, self.Wd),
                              merged, self.t_wg, self.t_wu, self.t_wd)

    def route(self):
        api.moe_route_topk(self.X, self.Wr, self.bias, self.w.k, self.idx, self.gate, None)

    def forward(self, idx=None, gate=None):
        w = self.w
        idx = self.idx if idx is None else idx
        gate = self.gate if gate is None else gate
        api.moe_permute(self.X, idx, gate, self.expert_map, self.S_r, self.offsets, self.perm_token,
                        self.perm_gate, self.inv, self.X_perm, self.ws_perm, E=w.E, x_sq=self.x_sq)
        api.moe_grouped_swiglu_fwd(self.layer_tables, self.X, self.X_perm, self.offsets, w.T, w.k, self.A_g,
                                   self.A_u, self.H, self.O, self.ws_fwd)
        api.moe_unpermute(self.layer_tables, self.O, self.inv, self.perm_gate, w.T, w.k, self.Y)

    def backward(self, dgate: bool = False, accumulate_dw: bool = False):
        w = self.w
        api.moe_unpermute_bwd(self.layer_tables, self.dY, self.O, self.inv, self.offsets, self.perm_gate,
                              w.T, w.k, self.dO, self.dgate if dgate else None, dy_sq=self.dy_sq)
        api.moe_grouped_swiglu_bwd(self.layer_tables, self.X, self.X_perm, self.offsets, w.T, w.k, self.A_g,
                                   self.A_u, self.H, self.dO, self.dX_perm, accumulate_dw, self.ws_bwd)
        api.moe_permute_bwd(self.layer_tables, self.dX_perm, self.inv, w.T, w.k, self.dX)

    def step(self):
        self.profile()
        self.merge()
        self.route()
        self.forward()
        self.backward()
