"""Gate re-routing and permutation (Section 7) alone, through the C ABI, against
the oracle's maps, bit-exact: offsets, perm_token and inv exactly, perm_gate to
fp32 summation order, X_perm rows bit for bit.  The shapes reach both ways the
entry point builds the maps (each block summing the slots x count-blocks table
itself up to 16384 entries, a separate scan launch beyond), the
largest slot count (512), slot maps that fold several experts into one slot (a
token's choices merged into one row), maps that leave slots empty, and the
largest k."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2508_19078_amd import api

from gpu_harness import host, log

pytestmark = pytest.mark.gpu

CASES = {
    # name: (T, d, E, k, map kind, S_routed, dtype)
    "one_block": (100, 64, 8, 2, "identity", 8, torch.bfloat16),
    "fused_256_blocks_folded": (65536, 64, 64, 6, "pairs", 32, torch.bfloat16),
    "scan_274_blocks_gaps": (70000, 16, 64, 8, "even", 128, torch.bfloat16),
    "max_slots_k16": (3000, 32, 256, 16, "odd", 512, torch.bfloat16),
    "fp32_ragged": (257, 24, 16, 4, "pairs", 8, torch.float32),
}


def expert_map_of(kind, E, S):
    e = np.arange(E)
    m = {"identity": e, "pairs": e // 2, "even": 2 * e, "odd": 2 * e + 1}[kind]
    assert m.max() < S
    return m.astype(np.int32)


@pytest.mark.parametrize("name", list(CASES))
def test_permute_maps_and_rows(name):
    T, d, E, k, kind, S, dt = CASES[name]
    log(f"permute {name}: T={T} d={d} E={E} k={k} map={kind} S={S} dtype={dt}")
    rng = np.random.default_rng([4100, T, E, k])
    idx = np.argsort(rng.random((T, E)), axis=1)[:, :k].astype(np.int32)
    gate = rng.random((T, k)).astype(np.float32)
    emap = expert_map_of(kind, E, S)
    X = torch.from_numpy(rng.standard_normal((T, d)).astype(np.float32)).to(dt).cuda()
    dev = "cuda"
    R = T * k
    offsets = torch.zeros(S + 1, dtype=torch.int32, device=dev)
    ptok = torch.zeros(R, dtype=torch.int32, device=dev)
    pgate = torch.zeros(R, dtype=torch.float32, device=dev)
    inv = torch.zeros((T, k), dtype=torch.int32, device=dev)
    Xp = torch.zeros((R, d), dtype=dt, device=dev)
    ws = torch.empty(api.moe_permute_workspace_size(T, k, S), dtype=torch.uint8, device=dev)
    api.moe_permute(X, torch.from_numpy(idx).cuda(), torch.from_numpy(gate).cuda(), torch.from_numpy(emap).cuda(),
                    S, offsets, ptok, pgate, inv, Xp, ws, E=E)
    torch.cuda.synchronize()
    o_off, o_tok, o_gate, o_inv = O.permute_maps(idx, gate, emap, S)
    np.testing.assert_array_equal(host(offsets), o_off)
    N = int(o_off[-1])
    log(f"  {N} rows of {R} choices, {int((np.diff(o_off) == 0).sum())} empty slots")
    np.testing.assert_array_equal(host(ptok)[:N], o_tok)
    np.testing.assert_array_equal(host(inv), o_inv)
    np.testing.assert_allclose(host(pgate)[:N], o_gate, rtol=2e-6)
    np.testing.assert_array_equal(host(Xp[:N]), host(X)[o_tok])
