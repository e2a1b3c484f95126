"""Device buffers and call sequence of the quantised profiling pass over a
stack of MoE layers (Section 4.1: a low-bit copy of the model is run over the
participant's data to learn which experts each layer activates).

``QuantizedStack`` quantises every layer's router and expert matrices to int8
with one scale per row (``moe_quantize_int8``) and keeps only the codes and
scales resident.  ``run`` then passes a batch through the stack, layer by
layer, on one stream:

  moe_rms_norm        the layer's input: the RMS-normalised stream (fused with
                      the previous layer's residual add)
  moe_profile_route   int8 routing: histogram, top-k indices and gates
  moe_permute         the layer's rows into per-expert buckets
  moe_grouped_swiglu_fwd_q8   the experts straight from their int8 codes
                      (bf16 activations, d and I multiples of 16); otherwise
                      moe_dequant_int8 into one reused buffer and
                      moe_grouped_swiglu_fwd
  moe_unpermute       Y_l, then X_{l+1} = X_l + Y_l (moe_rms_norm, which also
                      normalises X_{l+1} for the next layer; moe_residual_add
                      after the last layer)

Every value is computed by libfluxmoe; this module only owns buffers and
orders the calls.
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import torch

from . import api


class QuantizedStack:
    """layers[l] = dict(Wr [E,d], bias [E] fp32 or None, wg [E,I,d], wu [E,I,d],
    wd [E,d,I], and optionally sg/su/sd for shared experts), device tensors in
    one float dtype.  Only the int8 codes and fp32 scales are kept."""

    def __init__(self, layers: Sequence[dict], T: int, k: int, device: str = "cuda",
                 record: bool = False, fused: Optional[bool] = None, eps: float = 1e-6):
        L0 = layers[0]
        self.dt = L0["wg"].dtype
        self.E, self.I, self.d = L0["wg"].shape
        self.n_sh = 0 if L0.get("sg") is None else L0["sg"].shape[0]
        self.T, self.k, self.L = T, k, len(layers)
        self.record = record
        self.eps = eps
        E, I, d, n_sh = self.E, self.I, self.d, self.n_sh
        dev = device

        def quant(W):
            cols = W.shape[-1]
            q = torch.empty(W.shape, dtype=torch.int8, device=dev)
            s = torch.empty(W.numel() // cols, dtype=torch.float32, device=dev)
            api.moe_quantize_int8(W.reshape(-1, cols), q.view(-1, cols), s)
            return q, s

        self.q = []
        for lay in layers:
            ql = {"Wr": quant(lay["Wr"]), "bias": lay.get("bias")}
            for name in ("wg", "wu", "wd", "sg", "su", "sd"):
                if lay.get(name) is not None:
                    ql[name] = quant(lay[name])
            self.q.append(ql)

        can_fuse = self.dt == torch.bfloat16 and d % 16 == 0 and I % 16 == 0
        self.fused = can_fuse if fused is None else bool(fused)
        if self.fused and not can_fuse:
            raise ValueError("the int8 forward needs bf16 activations and d, I multiples of 16")
        z = lambda *shape, dtype=self.dt: torch.empty(*shape, dtype=dtype, device=dev)

        def per_slot(ql, name, sname, rows):
            """Per-slot codes and scales of one matrix: routed slots, then shared."""
            out_q, out_s = [], []
            for nm, n in ((name, E), (sname, n_sh)):
                if n == 0:
                    continue
                q, sc = ql[nm]
                out_q += [q[e] for e in range(n)]
                out_s += [sc[e * rows:(e + 1) * rows] for e in range(n)]
            return out_q, out_s
        if self.fused:
            # per-layer tables of the int8 codes and their row scales
            self.qtables = []
            for ql in self.q:
                gq, gs = per_slot(ql, "wg", "sg", I)
                uq, us = per_slot(ql, "wu", "su", I)
                dq, ds = per_slot(ql, "wd", "sd", d)
                self.qtables.append(api.LayerTablesQ8(d, I, E, n_sh, gq, uq, dq, gs, us, ds, device=dev))
            # the combine reads only the layer's shape
            self.layer = api.moe_layer(d, I, api.dtype_code(self.dt), E, n_sh, None, None, None, None, None, None)
            ws_fwd = api.moe_grouped_swiglu_fwd_q8_workspace_size(self.qtables[0], T, k)
        else:
            # one layer's dequantised experts, reused by every layer
            self.Dg, self.Du, self.Dd = z(E, I, d), z(E, I, d), z(E, d, I)
            if n_sh:
                self.Sg, self.Su, self.Sd = z(n_sh, I, d), z(n_sh, I, d), z(n_sh, d, I)
            wg = [self.Dg[e] for e in range(E)] + ([self.Sg[i] for i in range(n_sh)] if n_sh else [])
            wu = [self.Du[e] for e in range(E)] + ([self.Su[i] for i in range(n_sh)] if n_sh else [])
            wd = [self.Dd[e] for e in range(E)] + ([self.Sd[i] for i in range(n_sh)] if n_sh else [])
            self.layer = api.LayerTables(d, I, self.dt, E, n_sh, wg, wu, wd, device=dev)
            ws_fwd = api.moe_grouped_swiglu_fwd_workspace_size(self.layer, T, k)

        R, Rt = T * k, T * (k + n_sh)
        zi = lambda *shape: torch.zeros(*shape, dtype=torch.int32, device=dev)
        self.counts = zi(self.L, E)
        self.idx = zi(T, k)
        self.gate = z(T, k, dtype=torch.float32)
        self.offsets = zi(E + 1)
        self.perm_token, self.inv = zi(R), zi(T, k)
        self.perm_gate = z(R, dtype=torch.float32)
        self.X_perm = z(R, d)
        self.ws_perm = torch.empty(api.moe_permute_workspace_size(T, k, E), dtype=torch.uint8, device=dev)
        if not self.fused:
            self.A_g, self.A_u = z(Rt, I), z(Rt, I)
        self.H, self.O = z(Rt, I), z(Rt, d)
        self.Y = z(T, d)
        self.Xa, self.Xb, self.Xn = z(T, d), z(T, d), z(T, d)
        self.ws_fwd = torch.empty(ws_fwd, dtype=torch.uint8, device=dev)
        self.trace: List[dict] = []

    def run(self, X0: torch.Tensor, mark=None) -> torch.Tensor:
        """The stack on the batch X0 [T,d]; per-layer histograms land in
        self.counts [L,E]; returns the last layer's output stream.  mark(name),
        if given, is called after each stage (e.g. to record a HIP event)."""
        mark = mark if mark is not None else (lambda name: None)
        T, k = self.T, self.k
        self.counts.zero_()
        self.trace = []
        self.Xa.copy_(X0)
        X, Xnext, Xn = self.Xa, self.Xb, self.Xn
        api.moe_rms_norm(X, None, Xn, eps=self.eps)
        mark("norm")
        for l, ql in enumerate(self.q):
            if not self.fused:
                api.moe_dequant_int8(ql["wg"][0], ql["wg"][1], self.Dg)
                api.moe_dequant_int8(ql["wu"][0], ql["wu"][1], self.Du)
                api.moe_dequant_int8(ql["wd"][0], ql["wd"][1], self.Dd)
                if self.n_sh:
                    api.moe_dequant_int8(ql["sg"][0], ql["sg"][1], self.Sg)
                    api.moe_dequant_int8(ql["su"][0], ql["su"][1], self.Su)
                    api.moe_dequant_int8(ql["sd"][0], ql["sd"][1], self.Sd)
                mark("dequant")
            Wq, ws = ql["Wr"]
            api.moe_profile_route(Xn, Wq, ws, ql["bias"], k, self.counts[l], self.idx, self.gate)
            mark("route")
            api.moe_permute(Xn, self.idx, self.gate, None, self.E, self.offsets, self.perm_token, self.perm_gate,
                            self.inv, self.X_perm, self.ws_perm, E=self.E)
            mark("permute")
            if self.fused:
                api.moe_grouped_swiglu_fwd_q8(self.qtables[l], Xn, self.X_perm, self.offsets, T, k, self.H, self.O,
                                              self.ws_fwd)
            else:
                api.moe_grouped_swiglu_fwd(self.layer, Xn, self.X_perm, self.offsets, T, k, self.A_g, self.A_u,
                                           self.H, self.O, self.ws_fwd)
            mark("ffn_fwd")
            api.moe_unpermute(self.layer, self.O, self.inv, self.perm_gate, T, k, self.Y)
            if self.record:
                self.trace.append({"idx": self.idx.clone(), "gate": self.gate.clone(), "X": X.clone(),
                                   "Xn": Xn.clone(), "Y": self.Y.clone()})
            if l + 1 < self.L:
                api.moe_rms_norm(X, self.Y, Xn, out_sum=Xnext, eps=self.eps)
            else:
                api.moe_residual_add(X, self.Y, Xnext)
            mark("combine")
            X, Xnext = Xnext, X
        return X
