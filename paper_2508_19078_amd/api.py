"""Thin ctypes binding of libfluxmoe (include/fluxmoe.h).

Each function has the name of the C entry point it calls and only marshals
arguments: torch tensors become device pointers, dtypes become MOE_* codes,
the stream defaults to torch's current stream.  No arithmetic of the method
happens here.  If the library is not built, the first call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

import torch

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libfluxmoe.so")

MOE_OK, MOE_ERR_ARG, MOE_ERR_UNSUPPORTED, MOE_ERR_ALIGN, MOE_ERR_WORKSPACE, MOE_ERR_HIP = range(6)
MOE_F32, MOE_BF16, MOE_I8 = 0, 1, 2

_c_int, _c_size, _vp, _f = ctypes.c_int, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_float


class MoeError(RuntimeError):
    def __init__(self, code: int, fn: str, msg: str):
        super().__init__(f"{fn} failed with code {code}: {msg}")
        self.code = code


class moe_layer(ctypes.Structure):
    _fields_ = [("d", _c_int), ("I", _c_int), ("dtype", _c_int), ("S_routed", _c_int),
                ("S_shared", _c_int), ("w_gate", _vp), ("w_up", _vp), ("w_down", _vp),
                ("dw_gate", _vp), ("dw_up", _vp), ("dw_down", _vp)]


class moe_layer_q8(ctypes.Structure):
    _fields_ = [("d", _c_int), ("I", _c_int), ("S_routed", _c_int), ("S_shared", _c_int),
                ("q_gate", _vp), ("q_up", _vp), ("q_down", _vp), ("s_gate", _vp), ("s_up", _vp),
                ("s_down", _vp)]


# name -> (restype, argtypes)
_SIGS = {
    "moe_last_error": (ctypes.c_char_p, []),
    "moe_abi_version": (_c_int, []),
    "moe_route_topk": (_c_int, [_vp, _vp, _c_int, _vp, _c_int, _c_int, _c_int, _c_int, _vp, _vp, _vp, _vp]),
    "moe_route_bwd": (_c_int, [_vp, _vp, _vp, _vp, _c_int, _c_int, _c_int, _c_int, _c_int, _vp, _c_int, _vp]),
    "moe_quantize_int8": (_c_int, [_vp, _c_int, _c_int, _c_int, _vp, _vp, _vp]),
    "moe_profile_hist": (_c_int, [_vp, _c_int, _vp, _vp, _vp, _c_int, _c_int, _c_int, _c_int, _vp, _vp, _vp]),
    "moe_merge_plan": (_c_int, [_vp, _c_int, _c_int, _c_int, _f, _c_int, _c_int, _c_int, _vp, _vp, _vp,
                                _vp, _vp, _vp]),
    "moe_activation_frequency": (_c_int, [_vp, _c_int, _f, _vp, _vp]),
    "moe_merge_experts": (_c_int, [_vp, _c_int, _c_int, _c_int, _c_int, _vp, _vp, _vp, _vp, _c_int, _vp]),
    "moe_slot_pointers": (_c_int, [_vp, _c_int, _c_int, _c_int, _c_int, _c_int, _vp, _vp, _vp, _vp, _vp,
                                   _vp, _vp, _vp, _vp, _vp]),
    "moe_permute": (_c_int, [_vp, _c_int, _vp, _vp, _vp, _c_int, _c_int, _c_int, _c_int, _c_int, _vp, _vp,
                             _vp, _vp, _vp, _vp, _c_size, _vp, _vp]),
    "moe_permute_workspace_size": (_c_size, [_c_int, _c_int, _c_int]),
    "moe_validate_routing": (_c_int, [_vp, _vp, _c_int, _c_int, _c_int, _c_int]),
    "moe_permute_noalloc": (_c_int, [_vp, _c_int, _vp, _vp, _vp, _c_int, _c_int, _c_int, _c_int, _c_int, _vp,
                                     _vp, _vp, _vp, _vp, _vp, _vp]),
    "moe_permute_noalloc_max_bytes": (_c_size, []),
    "moe_grouped_swiglu_fwd": (_c_int, [_vp, _vp, _vp, _vp, _c_int, _c_int, _vp, _vp, _vp, _vp, _vp,
                                        _c_size, _vp]),
    "moe_grouped_swiglu_fwd_workspace_size": (_c_size, [_vp, _c_int, _c_int]),
    "moe_grouped_swiglu_fwd_q8": (_c_int, [_vp, _vp, _vp, _vp, _c_int, _c_int, _vp, _vp, _vp, _c_size, _vp]),
    "moe_grouped_swiglu_fwd_q8_workspace_size": (_c_size, [_vp, _c_int, _c_int]),
    "moe_unpermute": (_c_int, [_vp, _vp, _vp, _vp, _c_int, _c_int, _vp, _vp]),
    "moe_unpermute_bwd": (_c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _c_int, _c_int, _vp, _vp, _vp, _vp]),
    "moe_grouped_swiglu_bwd": (_c_int, [_vp, _vp, _vp, _vp, _c_int, _c_int, _vp, _vp, _vp, _vp, _vp,
                                        _c_int, _vp, _c_size, _vp]),
    "moe_grouped_swiglu_bwd_workspace_size": (_c_size, [_vp, _c_int, _c_int]),
    "moe_permute_bwd": (_c_int, [_vp, _vp, _vp, _c_int, _c_int, _vp, _vp]),
    "moe_expert_utility": (_c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _c_int, _c_int, _vp, _c_size, _vp, _vp]),
    "moe_profile_route": (_c_int, [_vp, _c_int, _vp, _vp, _vp, _c_int, _c_int, _c_int, _c_int, _vp, _vp, _vp,
                                   _vp]),
    "moe_dequant_int8": (_c_int, [_vp, _vp, ctypes.c_long, _c_int, _c_int, _vp, _vp]),
    "moe_residual_add": (_c_int, [_vp, _vp, _c_int, _c_int, _c_int, _vp, _vp]),
    "moe_rms_norm": (_c_int, [_vp, _vp, _c_int, _c_int, _c_int, _f, _vp, _vp, _vp]),
    "moe_merge_budget": (_c_int, [_vp, _vp, _c_int, _c_int, _f, _c_int, ctypes.c_double, _vp, _vp]),
    "moe_cluster_workspace_size": (_c_size, [_c_int, _c_int, _c_int, _c_int]),
    "moe_cluster_experts": (_c_int, [_vp, _c_int, _c_int, _c_int, _c_int, _c_int, _vp, _vp, _c_int, _c_int,
                                     _vp, _c_size, _vp, _vp, _vp, _vp]),
}

_lib = None
ABI_VERSION = 3   # FLUXMOE_ABI_VERSION of the header these signatures follow


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2508_19078_amd.build` (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype, fn.argtypes = res, args
        v = L.moe_abi_version()
        if v != ABI_VERSION:
            raise RuntimeError(f"{LIB_PATH} has ABI version {v}, this binding marshals version {ABI_VERSION}: "
                               "rebuild it with `python -m paper_2508_19078_amd.build`")
        _lib = L
    return _lib


def exported_names() -> List[str]:
    return list(_SIGS)


# ------------------------------------------------------------- marshalling --

def dtype_code(t: torch.dtype) -> int:
    if t == torch.bfloat16:
        return MOE_BF16
    if t == torch.float32:
        return MOE_F32
    if t == torch.int8:
        return MOE_I8
    raise TypeError(f"unsupported dtype {t}")


I32, F32, I64, U8, I8 = torch.int32, torch.float32, torch.int64, torch.uint8, torch.int8
FLOAT = (torch.float32, torch.bfloat16)


def ptr(x, dt=None) -> Optional[int]:
    """Device address of a tensor argument (ints, structs and None pass through).

    A tensor must be dense (contiguous), on a GPU, and of dtype `dt` when one is
    given (a dtype or a tuple of them): the library reads raw memory with the
    layout and element type its header states, so an int64 index tensor or a
    strided view would otherwise be misread silently."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if isinstance(x, torch.Tensor):
        if not x.is_contiguous():
            raise ValueError(f"tensor argument of shape {tuple(x.shape)} is not contiguous")
        if x.device.type != "cuda":
            raise ValueError(f"tensor argument is on {x.device}, the library reads device memory")
        if dt is not None and x.dtype not in (dt if isinstance(dt, tuple) else (dt,)):
            raise TypeError(f"tensor argument has dtype {x.dtype}, expected {dt}")
        return x.data_ptr()
    if isinstance(x, ctypes.Structure):
        return ctypes.addressof(x)
    if hasattr(x, "struct"):
        return ctypes.addressof(x.struct)
    raise TypeError(type(x))


def stream_ptr(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else None
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _call(name: str, *args) -> int:
    rc = getattr(lib(), name)(*args)
    if rc != MOE_OK:
        raise MoeError(rc, name, lib().moe_last_error().decode())
    return rc


# --------------------------------------------------------------- routing ----

def moe_route_topk(X, Wr, bias, k, idx, gate, logits=None, stream=None):
    T, d = X.shape
    E = Wr.shape[0]
    return _call("moe_route_topk", ptr(X, FLOAT), ptr(Wr, X.dtype), dtype_code(X.dtype), ptr(bias, F32), T, d,
                 E, k, ptr(idx, I32), ptr(gate, F32), ptr(logits, F32), stream_ptr(stream))


def moe_route_bwd(gate, idx, dgate, Wr, dX, accumulate=False, stream=None):
    T, k = gate.shape
    E, d = Wr.shape
    return _call("moe_route_bwd", ptr(gate, F32), ptr(idx, I32), ptr(dgate, F32), ptr(Wr, FLOAT),
                 dtype_code(Wr.dtype), T, d, E, k, ptr(dX, Wr.dtype), int(bool(accumulate)), stream_ptr(stream))


def moe_quantize_int8(W, Wq, scale, stream=None):
    E, d = W.shape
    return _call("moe_quantize_int8", ptr(W, FLOAT), dtype_code(W.dtype), E, d, ptr(Wq, I8), ptr(scale, F32),
                 stream_ptr(stream))


def moe_profile_hist(X, Wq, scale, bias, k, counts, idx=None, stream=None):
    T, d = X.shape
    E = Wq.shape[0]
    return _call("moe_profile_hist", ptr(X, FLOAT), dtype_code(X.dtype), ptr(Wq, I8), ptr(scale, F32),
                 ptr(bias, F32), T, d, E, k, ptr(counts, I32), ptr(idx, I32), stream_ptr(stream))


# --------------------------------------------------------------- merging ----

def moe_profile_route(X, Wq, scale, bias, k, counts, idx, gate, stream=None):
    T, d = X.shape
    E = Wq.shape[0]
    return _call("moe_profile_route", ptr(X, FLOAT), dtype_code(X.dtype), ptr(Wq, I8), ptr(scale, F32),
                 ptr(bias, F32), T, d, E, k, ptr(counts, I32), ptr(idx, I32), ptr(gate, F32), stream_ptr(stream))


def moe_dequant_int8(q, scale, out, stream=None):
    """q [..., cols] int8 with one scale per row of the flattened [rows, cols]."""
    cols = q.shape[-1]
    rows = q.numel() // cols
    return _call("moe_dequant_int8", ptr(q, I8), ptr(scale, F32), rows, cols, dtype_code(out.dtype),
                 ptr(out, FLOAT), stream_ptr(stream))


def moe_residual_add(X, Y, out, stream=None):
    T, d = X.shape
    return _call("moe_residual_add", ptr(X, FLOAT), ptr(Y, X.dtype), T, d, dtype_code(X.dtype), ptr(out, X.dtype),
                 stream_ptr(stream))


def moe_rms_norm(X, Y, out_norm, out_sum=None, eps=1e-6, stream=None):
    """out_norm = RMS-normalised (X + Y) (or X when Y is None); out_sum = X + Y."""
    T, d = X.shape
    return _call("moe_rms_norm", ptr(X, FLOAT), ptr(Y, X.dtype), T, d, dtype_code(X.dtype), float(eps),
                 ptr(out_sum, X.dtype), ptr(out_norm, X.dtype), stream_ptr(stream))


def moe_merge_plan(counts, n_merge, group, total_tokens, expert_map, slot_src, grp_ptr, grp_member,
                   alpha, expert_base=0, grp_base=0, member_base=0, stream=None):
    E = counts.shape[0]
    return _call("moe_merge_plan", ptr(counts, I32), E, n_merge, group, float(total_tokens), expert_base,
                 grp_base, member_base, ptr(expert_map, I32), ptr(slot_src, I32), ptr(grp_ptr, I32),
                 ptr(grp_member, I32), ptr(alpha, F32), stream_ptr(stream))


def moe_activation_frequency(counts, total_tokens, freq, stream=None):
    return _call("moe_activation_frequency", ptr(counts, I32), counts.shape[0], float(total_tokens),
                 ptr(freq, F32), stream_ptr(stream))


def plan_from_groups(E: int, groups):
    """ABI arrays of a caller-given grouping: kept experts in index order take
    slots 0..K-1, group g takes slot K+g.  Host-side bookkeeping only."""
    import numpy as np
    grouped = {int(e) for g in groups for e in g}
    kept = [e for e in range(E) if e not in grouped]
    K = len(kept)
    expert_map = np.zeros(E, dtype=np.int32)
    slot_src = np.zeros(K + len(groups), dtype=np.int32)
    for j, e in enumerate(kept):
        expert_map[e] = j
        slot_src[j] = e
    grp_ptr = [0]
    members = []
    for g, grp in enumerate(groups):
        for e in grp:
            expert_map[e] = K + g
            members.append(int(e))
        grp_ptr.append(len(members))
        slot_src[K + g] = E + g
    return dict(expert_map=expert_map, slot_src=slot_src, grp_ptr=np.array(grp_ptr, dtype=np.int32),
                grp_member=np.array(members, dtype=np.int32), K=K, G=len(groups))


def moe_merge_experts(w_src_ptrs, dtype, d, I, G, grp_ptr, grp_member, alpha, w_dst_ptrs, out_dtype,
                      stream=None):
    """w_src_ptrs / w_dst_ptrs: int64 device tensors of 3 pointers per expert / group."""
    return _call("moe_merge_experts", ptr(w_src_ptrs, I64), dtype_code(dtype), d, I, G, ptr(grp_ptr, I32),
                 ptr(grp_member, I32), ptr(alpha, F32), ptr(w_dst_ptrs, I64), dtype_code(out_dtype),
                 stream_ptr(stream))


def moe_slot_pointers(slot_src, S, E, d, I, dtype, orig, merged, w_gate, w_up, w_down, stream=None):
    """orig / merged: (gate, up, down) stacked tensors; merged may be (None,)*3."""
    return _call("moe_slot_pointers", ptr(slot_src, I32), S, E, d, I, dtype_code(dtype), ptr(orig[0], dtype),
                 ptr(orig[1], dtype), ptr(orig[2], dtype), ptr(merged[0], dtype), ptr(merged[1], dtype),
                 ptr(merged[2], dtype), ptr(w_gate, I64), ptr(w_up, I64), ptr(w_down, I64), stream_ptr(stream))


# --------------------------------------------------- layer-aware merging ----

def moe_merge_budget(counts, tuning, total_tokens, B_non, budget, eps=1e-12, stream=None):
    """counts [L, E] int32, tuning [L, E] uint8 (1 = tuning), budget [L] int32."""
    L, E = counts.shape
    return _call("moe_merge_budget", ptr(counts, I32), ptr(tuning, U8), L, E, float(total_tokens), int(B_non),
                 float(eps), ptr(budget, I32), stream_ptr(stream))


def moe_cluster_workspace_size(L, E, d, I) -> int:
    return lib().moe_cluster_workspace_size(L, E, d, I)


def moe_cluster_experts(w_src_ptrs, dtype, L, E, d, I, tuning, budget, r, max_iter, ws, labels,
                        features=None, iters=None, stream=None):
    """w_src_ptrs: int64 device tensor of 3 pointers per expert (layer-major)."""
    return _call("moe_cluster_experts", ptr(w_src_ptrs, I64), dtype_code(dtype), L, E, d, I, ptr(tuning, U8),
                 ptr(budget, I32), int(r), int(max_iter), ptr(ws), ws.numel() * ws.element_size(),
                 ptr(labels, I32), ptr(features, F32), ptr(iters, I32), stream_ptr(stream))


# ------------------------------------------------------------- the layer ----

def moe_permute_workspace_size(T, k, S_routed) -> int:
    return lib().moe_permute_workspace_size(T, k, S_routed)


def moe_permute(X, idx, gate, expert_map, S_routed, offsets, perm_token, perm_gate, inv, X_perm, ws,
                E=None, x_sq=None, stream=None):
    """x_sq [T] fp32, if given, receives ||X[t]||^2 (for moe_expert_utility)."""
    T, d = X.shape
    k = idx.shape[1]
    E = E if E is not None else (expert_map.shape[0] if expert_map is not None else S_routed)
    return _call("moe_permute", ptr(X, FLOAT), dtype_code(X.dtype), ptr(idx, I32), ptr(gate, F32),
                 ptr(expert_map, I32), T, d, E, k, S_routed, ptr(offsets, I32), ptr(perm_token, I32),
                 ptr(perm_gate, F32), ptr(inv, I32), ptr(X_perm, X.dtype), ptr(ws),
                 ws.numel() * ws.element_size() if ws is not None else 0, ptr(x_sq, F32), stream_ptr(stream))


def moe_permute_noalloc(X, idx, gate, expert_map, S_routed, offsets, perm_token, perm_gate, inv, X_perm, E=None,
                        x_sq=None, stream=None):
    """moe_permute without a workspace (the library's own device scratch)."""
    T, d = X.shape
    k = idx.shape[1]
    E = E if E is not None else (expert_map.shape[0] if expert_map is not None else S_routed)
    return _call("moe_permute_noalloc", ptr(X, FLOAT), dtype_code(X.dtype), ptr(idx, I32), ptr(gate, F32),
                 ptr(expert_map, I32), T, d, E, k, S_routed, ptr(offsets, I32), ptr(perm_token, I32),
                 ptr(perm_gate, F32), ptr(inv, I32), ptr(X_perm, X.dtype), ptr(x_sq, F32), stream_ptr(stream))


def moe_permute_noalloc_max_bytes() -> int:
    return lib().moe_permute_noalloc_max_bytes()


def moe_validate_routing(idx, expert_map, S_routed, E=None):
    """Host-side range check of a routing (idx [T,k], expert_map [E] or None),
    given as CPU tensors or NumPy arrays (copied to int32 host arrays here)."""
    import numpy as np
    hi = np.ascontiguousarray(np.asarray(idx.cpu() if isinstance(idx, torch.Tensor) else idx), dtype=np.int32)
    T, k = hi.shape
    hm = None
    if expert_map is not None:
        hm = np.ascontiguousarray(np.asarray(expert_map.cpu() if isinstance(expert_map, torch.Tensor)
                                             else expert_map), dtype=np.int32)
    E = E if E is not None else (len(hm) if hm is not None else S_routed)
    return _call("moe_validate_routing", hi.ctypes.data if hi.size else None,
                 hm.ctypes.data if hm is not None else None, T, E, k, S_routed)


def moe_grouped_swiglu_fwd_workspace_size(layer, T, k) -> int:
    return lib().moe_grouped_swiglu_fwd_workspace_size(ptr(layer), T, k)


def moe_grouped_swiglu_bwd_workspace_size(layer, T, k) -> int:
    return lib().moe_grouped_swiglu_bwd_workspace_size(ptr(layer), T, k)


def moe_grouped_swiglu_fwd(layer, X, X_perm, offsets, T, k, A_g, A_u, H, O, ws, stream=None):
    return _call("moe_grouped_swiglu_fwd", ptr(layer), ptr(X, FLOAT), ptr(X_perm, FLOAT), ptr(offsets, I32), T,
                 k, ptr(A_g, FLOAT), ptr(A_u, FLOAT), ptr(H, FLOAT), ptr(O, FLOAT), ptr(ws),
                 ws.numel() * ws.element_size(), stream_ptr(stream))


def moe_grouped_swiglu_fwd_q8_workspace_size(layer, T, k) -> int:
    return lib().moe_grouped_swiglu_fwd_q8_workspace_size(ptr(layer), T, k)


def moe_grouped_swiglu_fwd_q8(layer, X, X_perm, offsets, T, k, H, O, ws, stream=None):
    return _call("moe_grouped_swiglu_fwd_q8", ptr(layer), ptr(X, FLOAT), ptr(X_perm, FLOAT), ptr(offsets, I32),
                 T, k, ptr(H, FLOAT), ptr(O, FLOAT), ptr(ws), ws.numel() * ws.element_size(), stream_ptr(stream))


def moe_unpermute(layer, O, inv, perm_gate, T, k, Y, stream=None):
    return _call("moe_unpermute", ptr(layer), ptr(O, FLOAT), ptr(inv, I32), ptr(perm_gate, F32), T, k,
                 ptr(Y, FLOAT), stream_ptr(stream))


def moe_unpermute_bwd(layer, dY, O, inv, offsets, perm_gate, T, k, dO, dgate=None, dy_sq=None, stream=None):
    """dy_sq [T] fp32, if given, receives ||dY[t]||^2 (for moe_expert_utility)."""
    return _call("moe_unpermute_bwd", ptr(layer), ptr(dY, FLOAT), ptr(O, FLOAT), ptr(inv, I32), ptr(offsets, I32),
                 ptr(perm_gate, F32), T, k, ptr(dO, FLOAT), ptr(dgate, F32), ptr(dy_sq, F32), stream_ptr(stream))


def moe_grouped_swiglu_bwd(layer, X, X_perm, offsets, T, k, A_g, A_u, H, dO, dX_perm, accumulate_dw, ws,
                           stream=None):
    return _call("moe_grouped_swiglu_bwd", ptr(layer), ptr(X, FLOAT), ptr(X_perm, FLOAT), ptr(offsets, I32), T,
                 k, ptr(A_g, FLOAT), ptr(A_u, FLOAT), ptr(H, FLOAT), ptr(dO, FLOAT), ptr(dX_perm, FLOAT),
                 int(accumulate_dw), ptr(ws), ws.numel() * ws.element_size(), stream_ptr(stream))


def moe_permute_bwd(layer, dX_perm, inv, T, k, dX, stream=None):
    return _call("moe_permute_bwd", ptr(layer), ptr(dX_perm, FLOAT), ptr(inv, I32), T, k, ptr(dX, FLOAT),
                 stream_ptr(stream))


def moe_expert_utility(layer, x_sq, dy_sq, perm_token, perm_gate, offsets, T, k, ws, utility, stream=None):
    """After moe_grouped_swiglu_bwd with the same workspace `ws`; x_sq and dy_sq
    as written by moe_permute and moe_unpermute_bwd."""
    return _call("moe_expert_utility", ptr(layer), ptr(x_sq, F32), ptr(dy_sq, F32), ptr(perm_token, I32),
                 ptr(perm_gate, F32), ptr(offsets, I32), T, k, ptr(ws), ws.numel() * ws.element_size(),
                 ptr(utility, F32), stream_ptr(stream))


# ----------------------------------------------------- layer descriptor ----

class LayerTables:
    """Device pointer tables of a layer's slots and the moe_layer struct.

    w_gate/w_up/w_down: per-slot weight tensors (routed slots, then shared),
    or pre-filled int64 device pointer tensors (e.g. written by
    moe_slot_pointers).  dw: per-slot fp32 gradient tensors or None (frozen).
    """

    def __init__(self, d: int, I: int, dtype: torch.dtype, S_routed: int, S_shared: int,
                 w_gate, w_up, w_down, dw_gate: Sequence = None, dw_up: Sequence = None,
                 dw_down: Sequence = None, device="cuda"):
        S = S_routed + S_shared

        def table(x):
            if isinstance(x, torch.Tensor) and x.dtype == torch.int64 and x.dim() == 1:
                assert x.numel() == S
                return x
            vals = [0 if t is None else ptr(t) for t in x]
            assert len(vals) == S
            return torch.tensor(vals, dtype=torch.int64, device=device)

        self.keep = [w_gate, w_up, w_down, dw_gate, dw_up, dw_down]
        self.w_gate, self.w_up, self.w_down = table(w_gate), table(w_up), table(w_down)
        none = [None] * S
        self.dw_gate = table(dw_gate if dw_gate is not None else none)
        self.dw_up = table(dw_up if dw_up is not None else none)
        self.dw_down = table(dw_down if dw_down is not None else none)
        self.struct = moe_layer(d, I, dtype_code(dtype), S_routed, S_shared, ptr(self.w_gate),
                                ptr(self.w_up), ptr(self.w_down), ptr(self.dw_gate), ptr(self.dw_up),
                                ptr(self.dw_down))


class LayerTablesQ8:
    """Device pointer tables of a layer's int8 experts and the moe_layer_q8
    struct.  q_*: per-slot int8 code tensors (routed slots, then shared);
    s_*: the matching per-row fp32 scales."""

    def __init__(self, d: int, I: int, S_routed: int, S_shared: int, q_gate, q_up, q_down, s_gate, s_up,
                 s_down, device="cuda"):
        S = S_routed + S_shared

        def table(x):
            vals = [ptr(t) for t in x]
            assert len(vals) == S and all(v for v in vals)
            return torch.tensor(vals, dtype=torch.int64, device=device)

        self.keep = [q_gate, q_up, q_down, s_gate, s_up, s_down]
        self.tabs = [table(x) for x in self.keep]
        self.struct = moe_layer_q8(d, I, S_routed, S_shared, *[ptr(t) for t in self.tabs])
