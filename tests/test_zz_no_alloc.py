"""The allocation-free attention call (louiskv_sparse_decode_attn_rows_noalloc,
for callers that cannot allocate) against louiskv_sparse_decode_attn_rows with
a workspace, through the C ABI: equal outputs and log-sum-exps bit for bit
(same kernels, same partial layout) on consecutive calls that share the
static scratch array, the second and third with smaller inputs, and the
oracle on a sample; a launch whose partials exceed the array is refused
before anything runs."""
import os
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import oracle  # noqa: E402
from parity_utils import to64  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _L():
    from paper_2510_11292_amd import louiskv
    return louiskv


def _case(seed, dtype, G, H, g, B, PR, W, nl, ls):
    gen = torch.Generator(device=DEV)
    gen.manual_seed(seed)
    S = G * H
    q = torch.randn(G, H * g, 128, generator=gen, device=DEV).mul(1.5).to(dtype)
    kp = torch.randn(S, PR, 128, generator=gen, device=DEV).mul(2).to(dtype)
    vp = torch.randn(S, PR, 128, generator=gen, device=DEV).to(dtype)
    kl = torch.randn(S, W, 128, generator=gen, device=DEV).mul(2).to(dtype)
    vl = torch.randn(S, W, 128, generator=gen, device=DEV).to(dtype)
    rows = torch.stack([torch.randperm(PR, generator=torch.Generator().manual_seed(seed + s))[:B] for s in range(S)])
    rows = rows.to(torch.int32).to(DEV)
    nsel = torch.randint(0, B + 1, (S,), generator=gen, device=DEV, dtype=torch.int32)
    nsel[0] = B
    nsel[-1] = 0
    return q, kp, vp, kl, vl, rows, nsel


# (seed, dtype, groups, kv heads, group size, budget, pool rows, window, live window rows, window start)
CALLS = [
    (11, torch.bfloat16, 1, 8, 4, 2048, 6000, 128, 100, 37),   # 8 slices: split-KV over 9 chunks
    (12, torch.bfloat16, 1, 4, 4, 600, 2000, 64, 64, 0),       # smaller: fewer slices and chunks
    (13, torch.float32, 1, 2, 8, 300, 900, 32, 5, 30),         # smaller again, fp32 kernel
]


def test_noalloc_equals_workspace_call_on_consecutive_calls():
    L = _L()
    for seed, dtype, G, H, g, B, PR, W, nl, ls in CALLS:
        print(f"[no-alloc] seed={seed} dtype={dtype} slices={G * H} budget={B} window={W}", flush=True)
        q, kp, vp, kl, vl, rows, nsel = _case(seed, dtype, G, H, g, B, PR, W, nl, ls)
        need = L.sparse_decode_attn_rows_workspace_size(G * H, g, B, W)
        assert 0 < need <= L.NOALLOC_SCRATCH_BYTES       # the split-KV path, with partials in the array
        out_ref = torch.full((G, H * g, 128), float("nan"), device=DEV)
        lse_ref = torch.full((G, H * g), float("nan"), device=DEV)
        L.sparse_decode_attn_rows(q, H, kp, vp, rows, nsel, kl, vl, ls, nl, out_ref, lse_ref)
        out = torch.full_like(out_ref, float("nan"))
        lse = torch.full_like(lse_ref, float("nan"))
        L.sparse_decode_attn_rows_noalloc(q, H, kp, vp, rows, nsel, kl, vl, ls, nl, out, lse)
        torch.cuda.synchronize()
        assert torch.equal(out, out_ref) and torch.equal(lse, lse_ref), seed
        # and the oracle on two slices (the fullest and a ragged one)
        q64 = to64(q)
        for s in (0, G * H // 2):
            grp, h = divmod(s, H)
            n = int(nsel[s])
            idx = rows[s, :n].long()
            slots = [(ls + i) % W for i in range(nl)]
            kk = np.concatenate([to64(kp[s, idx]), to64(kl[s, slots])])
            vv = np.concatenate([to64(vp[s, idx]), to64(vl[s, slots])])
            o, _ = oracle.attention(q64[grp, h * g:(h + 1) * g], kk, vv, 1 / np.sqrt(128))
            err = np.abs(to64(out[grp, h * g:(h + 1) * g]) - o).max()
            assert err <= (1e-5 * np.abs(o).max() if dtype == torch.float32 else 2e-3), (seed, s, err)


def test_noalloc_refuses_partials_beyond_the_array():
    """512 slices with a 73728-row budget need more partials than the array
    holds: the call returns LOUISKV_ERR_WORKSPACE and leaves the output as it
    was.  (Every slice selects nothing, so the buffers are safe to read even
    by a launch.)"""
    L = _L()
    G, H, g, B, W = 64, 8, 4, 73728, 32
    S = G * H
    assert L.sparse_decode_attn_rows_workspace_size(S, g, B, W) > L.NOALLOC_SCRATCH_BYTES
    q = torch.zeros(G, H * g, 128, dtype=torch.bfloat16, device=DEV)
    kp = torch.zeros(S, 1, 128, dtype=torch.bfloat16, device=DEV)
    kl = torch.zeros(S, W, 128, dtype=torch.bfloat16, device=DEV)
    rows = torch.zeros(S, B, dtype=torch.int32, device=DEV)
    nsel = torch.zeros(S, dtype=torch.int32, device=DEV)
    out = torch.full((G, H * g, 128), 7.0, device=DEV)
    with pytest.raises(L.LouisKVError) as e:
        L.sparse_decode_attn_rows_noalloc(q, H, kp, kp, rows, nsel, kl, kl, 0, 0, out)
    assert e.value.status == 5 and "allocation-free" in str(e.value)
    torch.cuda.synchronize()
    assert torch.all(out == 7.0)
