"""moe_permute_noalloc, the permutation for callers that cannot allocate (its
count table lives in the library's own device scratch), through the C ABI
against moe_permute with a caller workspace on the same inputs: offsets, maps
and every gathered row bit-exact, and the maps equal to the oracle's.  Calls
come in a row on one device, each later one with fewer tokens, so a table left
over from an earlier call would show; the first call takes the path with a
separate scan launch (slots x count blocks above 16384 entries), the later ones
the fused path.  A table above the scratch is rejected before anything is
enqueued."""
import ctypes

import numpy as np
import pytest
import torch

import oracle as O
from paper_2508_19078_amd import api

from gpu_harness import host, log

pytestmark = pytest.mark.gpu


def draw(T, d, E, k, S, seed):
    rng = np.random.default_rng([6060, T, d, E, k, S, seed])
    X = torch.from_numpy(rng.standard_normal((T, d)).astype(np.float32)).to(torch.bfloat16)
    idx = np.argsort(rng.random((T, E)), axis=1)[:, :k].astype(np.int32)
    z = rng.standard_normal((T, k))
    gate = (np.exp(z) / np.exp(z).sum(1, keepdims=True)).astype(np.float32)
    # experts onto S slots: a seeded map that folds some experts together
    emap = rng.integers(0, S, size=E).astype(np.int32)
    emap[:min(E, S)] = rng.permutation(S)[:min(E, S)]
    return X, idx, gate, emap


def outputs(T, d, k, S, dev="cuda"):
    R = T * k
    return dict(offsets=torch.full((S + 1,), -5, dtype=torch.int32, device=dev),
                perm_token=torch.full((R,), -5, dtype=torch.int32, device=dev),
                perm_gate=torch.full((R,), -5.0, dtype=torch.float32, device=dev),
                inv=torch.full((T, k), -5, dtype=torch.int32, device=dev),
                X_perm=torch.zeros((R, d), dtype=torch.bfloat16, device=dev),
                x_sq=torch.full((T,), -5.0, dtype=torch.float32, device=dev))


def one_pair(T, d, E, k, S, seed):
    X, idx, gate, emap = draw(T, d, E, k, S, seed)
    Xd, idd, gd, emd = X.cuda(), torch.from_numpy(idx).cuda(), torch.from_numpy(gate).cuda(), \
        torch.from_numpy(emap).cuda()
    a, b = outputs(T, d, k, S), outputs(T, d, k, S)
    ws = torch.empty(api.moe_permute_workspace_size(T, k, S), dtype=torch.uint8, device="cuda")
    assert api.moe_permute(Xd, idd, gd, emd, S, a["offsets"], a["perm_token"], a["perm_gate"], a["inv"],
                           a["X_perm"], ws, E=E, x_sq=a["x_sq"]) == 0
    assert api.moe_permute_noalloc(Xd, idd, gd, emd, S, b["offsets"], b["perm_token"], b["perm_gate"], b["inv"],
                                   b["X_perm"], E=E, x_sq=b["x_sq"]) == 0
    torch.cuda.synchronize()
    offsets = host(a["offsets"])
    N = int(offsets[-1])
    nblk = -(-T // 256)
    log(f"noalloc permute T={T} d={d} E={E} k={k} S={S}: {N} rows, table {nblk * S} entries "
        f"({'scan launch' if nblk * S > 16384 else 'fused'})")
    for name in ("offsets", "inv"):
        np.testing.assert_array_equal(host(b[name]), host(a[name]), err_msg=name)
    np.testing.assert_array_equal(host(b["perm_token"])[:N], host(a["perm_token"])[:N])
    np.testing.assert_array_equal(host(b["perm_gate"])[:N], host(a["perm_gate"])[:N])
    assert torch.equal(b["X_perm"][:N].view(torch.int16), a["X_perm"][:N].view(torch.int16))
    assert torch.equal(b["x_sq"].view(torch.int32), a["x_sq"].view(torch.int32))
    xs = np.sum(host(Xd).astype(np.float64) ** 2, axis=1)
    np.testing.assert_allclose(host(b["x_sq"]), xs, rtol=1e-5)
    # and both are the oracle's maps
    o_off, o_tok, o_gate, o_inv = O.permute_maps(idx, gate, emap, S)
    np.testing.assert_array_equal(offsets, o_off)
    np.testing.assert_array_equal(host(b["perm_token"])[:N], o_tok)
    np.testing.assert_array_equal(host(b["inv"]), o_inv)
    np.testing.assert_allclose(host(b["perm_gate"])[:N], o_gate, rtol=2e-6)


def test_noalloc_permute_matches_workspace_permute_in_a_row():
    one_pair(40000, 256, 256, 8, 512, 0)      # 157 count blocks x 512 slots: scan launch
    one_pair(5000, 256, 256, 8, 512, 1)       # fewer tokens, fused table sums
    one_pair(700, 136, 64, 6, 40, 2)          # fewer still, another shape


def test_noalloc_permute_rejects_tables_above_its_scratch():
    L = api.lib()
    cap = L.moe_permute_noalloc_max_bytes()
    assert cap == 1 << 20
    T, S = 140000, 512                        # 547 blocks x 512 slots x 4 bytes > 1 MiB
    assert api.moe_permute_workspace_size(T, 8, S) > cap
    fake = 0x100000                           # never dereferenced: rejected on the host
    rc = L.moe_permute_noalloc(fake, api.MOE_BF16, fake, fake, fake, T, 256, 256, 8, S, fake, fake, fake, fake,
                               fake, None, None)
    assert rc == api.MOE_ERR_UNSUPPORTED and b"scratch" in L.moe_last_error()
