"""Host-side checks of the C ABI: the library loads, exports every function the
header declares, and rejects invalid arguments before any HIP call (so these
run on a machine without a GPU)."""
import ctypes
import os
import re

import pytest

from paper_2508_19078_amd import api

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fluxmoe.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(api.LIB_PATH):
        from paper_2508_19078_amd import build
        build.build(verbose=False)
    return api.lib()


def declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z0-9_]+)\s*\(", src)))


def test_every_declared_function_is_exported_and_bound(L):
    names = declared()
    assert len(names) >= 18
    for n in names:
        assert hasattr(L, n), n
        assert n in api.exported_names(), n
    assert L.moe_abi_version() == api.ABI_VERSION == 3


FAKE = 0x100000          # aligned, never dereferenced: validation fails first
MIS = FAKE + 4


def rc_and_msg(L, name, *args):
    rc = getattr(L, name)(*args)
    return rc, L.moe_last_error().decode()


def test_route_rejections(L):
    # k > E
    rc, msg = rc_and_msg(L, "moe_route_topk", FAKE, FAKE, api.MOE_BF16, None, 16, 64, 4, 5, FAKE, FAKE, None, None)
    assert rc == api.MOE_ERR_UNSUPPORTED and "k=5" in msg
    # E > 256
    rc, _ = rc_and_msg(L, "moe_route_topk", FAKE, FAKE, api.MOE_BF16, None, 16, 64, 300, 4, FAKE, FAKE, None, None)
    assert rc == api.MOE_ERR_UNSUPPORTED
    # d not a multiple of 8
    rc, _ = rc_and_msg(L, "moe_route_topk", FAKE, FAKE, api.MOE_BF16, None, 16, 60, 8, 2, FAKE, FAKE, None, None)
    assert rc == api.MOE_ERR_UNSUPPORTED
    # NULL X, NULL idx
    rc, msg = rc_and_msg(L, "moe_route_topk", None, FAKE, api.MOE_BF16, None, 16, 64, 8, 2, FAKE, FAKE, None, None)
    assert rc == api.MOE_ERR_ARG and "X" in msg
    rc, _ = rc_and_msg(L, "moe_route_topk", FAKE, FAKE, api.MOE_BF16, None, 16, 64, 8, 2, None, FAKE, None, None)
    assert rc == api.MOE_ERR_ARG
    # misaligned
    rc, _ = rc_and_msg(L, "moe_route_topk", MIS, FAKE, api.MOE_BF16, None, 16, 64, 8, 2, FAKE, FAKE, None, None)
    assert rc == api.MOE_ERR_ALIGN
    # unsupported dtype (int8 activations)
    rc, _ = rc_and_msg(L, "moe_route_topk", FAKE, FAKE, api.MOE_I8, None, 16, 64, 8, 2, FAKE, FAKE, None, None)
    assert rc == api.MOE_ERR_UNSUPPORTED
    # T == 0 is a no-op that touches nothing; per-token buffers may be NULL
    rc, _ = rc_and_msg(L, "moe_route_topk", FAKE, FAKE, api.MOE_BF16, None, 0, 64, 8, 2, FAKE, FAKE, None, None)
    assert rc == api.MOE_OK
    rc, _ = rc_and_msg(L, "moe_route_topk", None, None, api.MOE_BF16, None, 0, 64, 8, 2, None, None, None, None)
    assert rc == api.MOE_OK
    rc, _ = rc_and_msg(L, "moe_profile_hist", None, api.MOE_BF16, None, None, None, 0, 64, 8, 2, None, None, None)
    assert rc == api.MOE_OK
    # ... but the shape is still validated
    rc, _ = rc_and_msg(L, "moe_route_topk", None, None, api.MOE_BF16, None, 0, 64, 8, 9, None, None, None, None)
    assert rc != api.MOE_OK


def test_route_bwd_rejections(L):
    args = lambda **o: [o.get(n, v) for n, v in (("gate", FAKE), ("idx", FAKE), ("dgate", FAKE), ("Wr", FAKE),
                                                 ("dtype", api.MOE_BF16), ("T", 16), ("d", 64), ("E", 8), ("k", 2),
                                                 ("dX", FAKE), ("acc", 0), ("st", None))]
    rc, msg = rc_and_msg(L, "moe_route_bwd", *args(k=9))
    assert rc == api.MOE_ERR_UNSUPPORTED and "k=9" in msg
    rc, msg = rc_and_msg(L, "moe_route_bwd", *args(dgate=None))
    assert rc == api.MOE_ERR_ARG and "dgate" in msg
    rc, _ = rc_and_msg(L, "moe_route_bwd", *args(dX=MIS))
    assert rc == api.MOE_ERR_ALIGN
    rc, _ = rc_and_msg(L, "moe_route_bwd", *args(dtype=api.MOE_I8))
    assert rc == api.MOE_ERR_UNSUPPORTED
    rc, _ = rc_and_msg(L, "moe_route_bwd", *args(d=60))
    assert rc == api.MOE_ERR_UNSUPPORTED
    rc, _ = rc_and_msg(L, "moe_route_bwd", *args(T=0, gate=None, idx=None, dgate=None, Wr=None, dX=None))
    assert rc == api.MOE_OK


def test_profile_and_merge_rejections(L):
    rc, _ = rc_and_msg(L, "moe_profile_hist", FAKE, api.MOE_BF16, FAKE, FAKE, None, 8, 64, 8, 9, FAKE, None, None)
    assert rc == api.MOE_ERR_UNSUPPORTED
    rc, _ = rc_and_msg(L, "moe_profile_hist", FAKE, api.MOE_BF16, FAKE, None, None, 8, 64, 8, 2, FAKE, None, None)
    assert rc == api.MOE_ERR_ARG                                    # scale is required
    rc, _ = rc_and_msg(L, "moe_merge_plan", FAKE, 64, 30, 4, ctypes.c_float(1.0), 0, 0, 0,
                       FAKE, FAKE, FAKE, FAKE, FAKE, None)
    assert rc == api.MOE_ERR_ARG                                    # 30 % 4 != 0
    rc, _ = rc_and_msg(L, "moe_merge_plan", FAKE, 64, 32, 4, ctypes.c_float(0.0), 0, 0, 0,
                       FAKE, FAKE, FAKE, FAKE, FAKE, None)
    assert rc == api.MOE_ERR_ARG                                    # no tokens
    rc, _ = rc_and_msg(L, "moe_merge_experts", FAKE, api.MOE_BF16, 2048, 1404, 8, FAKE, FAKE, FAKE, FAKE,
                       api.MOE_BF16, None)
    assert rc == api.MOE_ERR_UNSUPPORTED                            # I % 8 != 0
    rc, _ = rc_and_msg(L, "moe_merge_experts", FAKE, api.MOE_BF16, 2048, 1408, 0, FAKE, FAKE, FAKE, FAKE,
                       api.MOE_BF16, None)
    assert rc == api.MOE_OK                                         # no groups: nothing to do
    rc, _ = rc_and_msg(L, "moe_quantize_int8", FAKE, api.MOE_BF16, 0, 64, FAKE, FAKE, None)
    assert rc == api.MOE_ERR_ARG


def test_permute_workspace_and_layer_rejections(L):
    need = L.moe_permute_workspace_size(4096, 4, 16)
    assert need >= (4096 // 256) * 16 * 4
    rc, msg = rc_and_msg(L, "moe_permute", FAKE, api.MOE_BF16, FAKE, FAKE, None, 4096, 4096, 16, 4, 16,
                         FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, ctypes.c_size_t(need - 1), None, None)
    assert rc == api.MOE_ERR_WORKSPACE and "workspace" in msg
    rc, _ = rc_and_msg(L, "moe_permute", FAKE, api.MOE_BF16, FAKE, FAKE, None, 4096, 4096, 16, 4, 8,
                       FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, ctypes.c_size_t(need), None, None)
    assert rc == api.MOE_ERR_ARG                                    # identity map needs S >= E
    # a layer with an unsupported intermediate size
    lay = api.moe_layer(2048, 1404, api.MOE_BF16, 40, 2, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)
    rc, _ = rc_and_msg(L, "moe_grouped_swiglu_fwd", ctypes.byref(lay), FAKE, FAKE, FAKE, 8192, 6, FAKE, FAKE,
                       FAKE, FAKE, FAKE, ctypes.c_size_t(1 << 30), None)
    assert rc == api.MOE_ERR_UNSUPPORTED
    lay = api.moe_layer(2048, 1408, api.MOE_BF16, 40, 2, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)
    need = L.moe_grouped_swiglu_fwd_workspace_size(ctypes.byref(lay), 8192, 6)
    assert need > 0
    rc, _ = rc_and_msg(L, "moe_grouped_swiglu_fwd", ctypes.byref(lay), FAKE, FAKE, FAKE, 8192, 6, FAKE, FAKE,
                       FAKE, FAKE, FAKE, ctypes.c_size_t(need - 1), None)
    assert rc == api.MOE_ERR_WORKSPACE
    bneed = L.moe_grouped_swiglu_bwd_workspace_size(ctypes.byref(lay), 8192, 6)
    assert bneed >= need + 2 * 8192 * 8 * 1408 * 2
    rc, _ = rc_and_msg(L, "moe_grouped_swiglu_bwd", ctypes.byref(lay), FAKE, FAKE, FAKE, 8192, 6, FAKE, FAKE,
                       FAKE, MIS, FAKE, 0, FAKE, ctypes.c_size_t(bneed), None)
    assert rc == api.MOE_ERR_ALIGN
    # the utility pass reads the backward's workspace: same size required
    rc, msg = rc_and_msg(L, "moe_expert_utility", ctypes.byref(lay), FAKE, FAKE, FAKE, FAKE, FAKE, 8192, 6, FAKE,
                         ctypes.c_size_t(bneed - 1), FAKE, None)
    assert rc == api.MOE_ERR_WORKSPACE and "workspace" in msg
    rc, msg = rc_and_msg(L, "moe_expert_utility", ctypes.byref(lay), FAKE, FAKE, FAKE, FAKE, FAKE, 8192, 6, FAKE,
                         ctypes.c_size_t(bneed), None, None)
    assert rc == api.MOE_ERR_ARG and "utility" in msg
    rc, msg = rc_and_msg(L, "moe_expert_utility", ctypes.byref(lay), FAKE, FAKE, None, FAKE, FAKE, 8192, 6, FAKE,
                         ctypes.c_size_t(bneed), FAKE, None)
    assert rc == api.MOE_ERR_ARG and "perm_token" in msg        # routed slots need the maps
    rc, _ = rc_and_msg(L, "moe_unpermute", None, FAKE, FAKE, FAKE, 8, 2, FAKE, None)
    assert rc == api.MOE_ERR_ARG
    rc, _ = rc_and_msg(L, "moe_permute_bwd", ctypes.byref(lay), FAKE, FAKE, 8, 17, FAKE, None)
    assert rc == api.MOE_ERR_UNSUPPORTED                            # k > 16


def test_error_message_is_cleared_on_success(L):
    rc_and_msg(L, "moe_route_topk", None, FAKE, api.MOE_BF16, None, 16, 64, 8, 2, FAKE, FAKE, None, None)
    assert L.moe_last_error().decode() != ""
    rc, msg = rc_and_msg(L, "moe_route_topk", FAKE, FAKE, api.MOE_BF16, None, 0, 64, 8, 2, FAKE, FAKE, None, None)
    assert rc == 0 and msg == ""


def test_plan_from_groups_arrays():
    pa = api.plan_from_groups(8, ((0, 1), (2, 3)))
    assert list(pa["expert_map"]) == [4, 4, 5, 5, 0, 1, 2, 3]
    assert list(pa["slot_src"]) == [4, 5, 6, 7, 8, 9]
    assert list(pa["grp_ptr"]) == [0, 2, 4] and list(pa["grp_member"]) == [0, 1, 2, 3]


def test_merge_budget_and_cluster_rejections(L):
    dbl = ctypes.c_double
    rc, msg = rc_and_msg(L, "moe_merge_budget", FAKE, FAKE, 0, 8, ctypes.c_float(10.0), 4, dbl(1e-12), FAKE, None)
    assert rc == api.MOE_ERR_UNSUPPORTED and "L=0" in msg
    rc, _ = rc_and_msg(L, "moe_merge_budget", FAKE, FAKE, 2000, 8, ctypes.c_float(10.0), 4, dbl(1e-12), FAKE, None)
    assert rc == api.MOE_ERR_UNSUPPORTED
    rc, msg = rc_and_msg(L, "moe_merge_budget", FAKE, None, 4, 8, ctypes.c_float(10.0), 4, dbl(1e-12), FAKE, None)
    assert rc == api.MOE_ERR_ARG and "tuning" in msg
    rc, _ = rc_and_msg(L, "moe_merge_budget", FAKE, FAKE, 4, 8, ctypes.c_float(0.0), 4, dbl(1e-12), FAKE, None)
    assert rc == api.MOE_ERR_ARG
    rc, _ = rc_and_msg(L, "moe_merge_budget", FAKE, FAKE, 4, 8, ctypes.c_float(10.0), -1, dbl(1e-12), FAKE, None)
    assert rc == api.MOE_ERR_ARG
    rc, _ = rc_and_msg(L, "moe_merge_budget", FAKE, FAKE, 4, 8, ctypes.c_float(10.0), 4, dbl(0.0), FAKE, None)
    assert rc == api.MOE_ERR_ARG

    need = L.moe_cluster_workspace_size(28, 64, 2048, 1408)
    # Gram partials of 264 chunks per layer (3 tiles) and the fp64 sums
    assert need >= 28 * 264 * 3 * 1024 * 4 + 28 * 3 * 1024 * 8
    assert L.moe_cluster_workspace_size(28, 65, 2048, 1408) == 0

    def call(E=64, d=2048, I=1408, r=16, it=50, ws=FAKE, nbytes=need, dtype=api.MOE_BF16, labels=FAKE):
        return rc_and_msg(L, "moe_cluster_experts", FAKE, dtype, 28, E, d, I, FAKE, FAKE, r, it, ws,
                          ctypes.c_size_t(nbytes), labels, None, None, None)
    rc, msg = call(E=65)
    assert rc == api.MOE_ERR_UNSUPPORTED and "E=65" in msg
    assert call(r=0)[0] == api.MOE_ERR_UNSUPPORTED
    assert call(r=33)[0] == api.MOE_ERR_UNSUPPORTED
    assert call(it=0)[0] == api.MOE_ERR_ARG
    assert call(d=3, I=5)[0] == api.MOE_ERR_UNSUPPORTED       # 15 bf16 values: not whole 16-byte chunks
    assert call(dtype=api.MOE_I8)[0] == api.MOE_ERR_UNSUPPORTED
    rc, msg = call(nbytes=need - 1)
    assert rc == api.MOE_ERR_WORKSPACE and "workspace" in msg
    assert call(ws=None)[0] == api.MOE_ERR_WORKSPACE
    assert call(ws=MIS)[0] == api.MOE_ERR_ALIGN
    rc, msg = call(labels=None)
    assert rc == api.MOE_ERR_ARG and "labels" in msg


def test_profiling_stack_rejections(L):
    f = ctypes.c_float
    rc, msg = rc_and_msg(L, "moe_profile_route", FAKE, api.MOE_BF16, FAKE, FAKE, None, 16, 64, 8, 2, FAKE, FAKE,
                         None, None)
    assert rc == api.MOE_ERR_ARG and "gate" in msg
    rc, msg = rc_and_msg(L, "moe_profile_route", FAKE, api.MOE_BF16, FAKE, FAKE, None, 16, 64, 8, 2, FAKE, None,
                         FAKE, None)
    assert rc == api.MOE_ERR_ARG and "idx" in msg
    rc, _ = rc_and_msg(L, "moe_profile_route", FAKE, api.MOE_BF16, FAKE, FAKE, None, 16, 64, 8, 9, FAKE, FAKE,
                       FAKE, None)
    assert rc == api.MOE_ERR_UNSUPPORTED                              # k > E
    rc, _ = rc_and_msg(L, "moe_dequant_int8", FAKE, FAKE, 10, 12, api.MOE_BF16, FAKE, None)
    assert rc == api.MOE_ERR_UNSUPPORTED                              # cols % 8
    rc, _ = rc_and_msg(L, "moe_dequant_int8", FAKE, FAKE, 10, 16, api.MOE_I8, FAKE, None)
    assert rc == api.MOE_ERR_UNSUPPORTED
    rc, _ = rc_and_msg(L, "moe_dequant_int8", FAKE, FAKE, -1, 16, api.MOE_BF16, FAKE, None)
    assert rc == api.MOE_ERR_ARG
    rc, _ = rc_and_msg(L, "moe_dequant_int8", FAKE, MIS, 10, 16, api.MOE_BF16, FAKE, None)
    assert rc == api.MOE_ERR_ALIGN
    rc, _ = rc_and_msg(L, "moe_residual_add", FAKE, FAKE, 16, 12, api.MOE_BF16, FAKE, None)
    assert rc == api.MOE_ERR_UNSUPPORTED
    rc, msg = rc_and_msg(L, "moe_residual_add", FAKE, None, 16, 16, api.MOE_BF16, FAKE, None)
    assert rc == api.MOE_ERR_ARG and "Y" in msg
    assert L.moe_residual_add(None, None, 0, 16, api.MOE_BF16, None, None) == 0   # T = 0: nothing to do


def test_quantised_forward_rejections(L):
    def lay(d=2048, I=1408, S_r=64, S_sh=0, tabs=(FAKE,) * 6):
        return api.moe_layer_q8(d, I, S_r, S_sh, *tabs)

    def call(layer, T=4096, k=6, X=FAKE, Xp=FAKE, off=FAKE, H=FAKE, O=FAKE, ws=FAKE, ws_bytes=None):
        if ws_bytes is None:
            ws_bytes = L.moe_grouped_swiglu_fwd_q8_workspace_size(ctypes.byref(layer), T, k)
        return rc_and_msg(L, "moe_grouped_swiglu_fwd_q8", ctypes.byref(layer), X, Xp, off, T, k, H, O, ws,
                          ctypes.c_size_t(ws_bytes), None)

    assert L.moe_grouped_swiglu_fwd_q8_workspace_size(ctypes.byref(lay()), 4096, 6) > 0
    assert L.moe_grouped_swiglu_fwd_q8_workspace_size(None, 4096, 6) == 0
    assert rc_and_msg(L, "moe_grouped_swiglu_fwd_q8", None, FAKE, FAKE, FAKE, 16, 2, FAKE, FAKE, FAKE,
                      ctypes.c_size_t(1 << 20), None)[0] == api.MOE_ERR_ARG
    assert call(lay(d=2040))[0] == api.MOE_ERR_UNSUPPORTED          # d % 16
    assert call(lay(I=1400))[0] == api.MOE_ERR_UNSUPPORTED          # I % 16
    assert call(lay(S_r=0, S_sh=0))[0] == api.MOE_ERR_ARG
    rc, msg = call(lay(tabs=(FAKE, FAKE, FAKE, FAKE, None, FAKE)))
    assert rc == api.MOE_ERR_ARG and "s_up" in msg
    assert call(lay(), k=17)[0] == api.MOE_ERR_ARG
    rc, msg = call(lay(), H=None)
    assert rc == api.MOE_ERR_ARG and "H" in msg
    assert call(lay(), O=MIS)[0] == api.MOE_ERR_ALIGN
    need = L.moe_grouped_swiglu_fwd_q8_workspace_size(ctypes.byref(lay()), 4096, 6)
    assert call(lay(), ws_bytes=need - 1)[0] == api.MOE_ERR_WORKSPACE
    assert call(lay(), T=0, X=None, Xp=None, off=None, H=None, O=None, ws=None)[0] == api.MOE_OK   # nothing to do


def test_validate_routing_rejects_out_of_range_maps(L):
    """The debug-only range check of moe_permute's idx and expert_map (host arrays)."""
    import numpy as np
    idx = np.array([[0, 3], [2, 1], [3, 0]], dtype=np.int32)
    emap = np.array([1, 0, 2, 2], dtype=np.int32)
    assert api.moe_validate_routing(idx, emap, 3) == api.MOE_OK
    assert api.moe_validate_routing(idx, None, 4) == api.MOE_OK        # identity map, S >= E
    bad = idx.copy(); bad[1, 1] = 4
    with pytest.raises(api.MoeError) as e:
        api.moe_validate_routing(bad, emap, 3)
    assert e.value.code == api.MOE_ERR_ARG and "idx[1][1]=4" in str(e.value)
    bad[1, 1] = -1
    with pytest.raises(api.MoeError):
        api.moe_validate_routing(bad, emap, 3)
    bmap = emap.copy(); bmap[3] = 3                                      # slot 3 of 3 slots
    with pytest.raises(api.MoeError) as e:
        api.moe_validate_routing(idx, bmap, 3)
    assert "expert_map[3]=3" in str(e.value)
    with pytest.raises(api.MoeError):
        api.moe_validate_routing(idx, None, 3)                           # identity map needs S >= E
    assert api.moe_validate_routing(np.zeros((0, 2), np.int32), emap, 3) == api.MOE_OK


def test_backward_without_tokens_needs_only_offsets_and_workspace(L):
    """T = 0: the per-token buffers may be NULL; offsets and the workspace are
    what the zeroing of the weight gradients reads, so they stay required."""
    lay = api.moe_layer(2048, 1408, api.MOE_BF16, 40, 2, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)
    need = ctypes.c_size_t(L.moe_grouped_swiglu_bwd_workspace_size(ctypes.byref(lay), 0, 6))
    rc, msg = rc_and_msg(L, "moe_grouped_swiglu_bwd", ctypes.byref(lay), None, None, None, 0, 6, None, None, None,
                         None, None, 0, FAKE, need, None)
    assert rc == api.MOE_ERR_ARG and "offsets" in msg
    rc, msg = rc_and_msg(L, "moe_grouped_swiglu_bwd", ctypes.byref(lay), None, None, FAKE, 0, 6, None, None, None,
                         None, None, 0, None, need, None)
    assert rc == api.MOE_ERR_ARG and "ws" in msg
    # accumulating into dW with no rows: nothing to do, every pointer may be NULL
    rc, _ = rc_and_msg(L, "moe_grouped_swiglu_bwd", ctypes.byref(lay), None, None, None, 0, 6, None, None, None,
                       None, None, 1, None, ctypes.c_size_t(0), None)
    assert rc == api.MOE_OK


def test_binding_rejects_misdescribed_tensors():
    """The binding refuses tensors whose dtype, layout or device the library
    would misread (checked before any library call)."""
    import torch
    i64 = torch.zeros(4, 2, dtype=torch.int64)
    with pytest.raises(ValueError):                                      # host tensor
        api.ptr(i64)
    with pytest.raises(ValueError):                                      # strided view
        api.ptr(torch.zeros(4, 4)[:, ::2])
    assert api.ptr(None) is None and api.ptr(1 << 20) == 1 << 20


def test_noalloc_permute_rejects_tables_above_its_scratch(L):
    """The no-allocation permute refuses, on the host, a count table larger
    than its fixed device scratch (1 MiB)."""
    assert L.moe_permute_noalloc_max_bytes() == 1 << 20
    T, S = 140000, 512
    assert L.moe_permute_workspace_size(T, 8, S) > 1 << 20
    rc, msg = rc_and_msg(L, "moe_permute_noalloc", FAKE, api.MOE_BF16, FAKE, FAKE, FAKE, T, 256, 256, 8, S, FAKE,
                         FAKE, FAKE, FAKE, FAKE, None, None)
    assert rc == api.MOE_ERR_UNSUPPORTED and "scratch" in msg
    rc, msg = rc_and_msg(L, "moe_permute_noalloc", FAKE, api.MOE_BF16, FAKE, FAKE, FAKE, 64, 256, 256, 17, S, FAKE,
                         FAKE, FAKE, FAKE, FAKE, None, None)
    assert rc == api.MOE_ERR_UNSUPPORTED                             # k > 16: validated as moe_permute does
