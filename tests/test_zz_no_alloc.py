"""The workspace-free permutation (ec2moe_permute_noalloc, for callers that cannot allocate)
against ec2moe_permute with a caller workspace, through the C ABI: bit-exact segment
offsets, source rows, inverse permutation and gathered rows, on calls in a row whose
sizes shrink (the library's count array keeps the previous call's contents)."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2508_06024_amd import ec2moe as E
from paper_2508_06024_amd import workload as W
from tests.gpu_common import down, say, up, up_i32

pytestmark = pytest.mark.gpu


def _case(T, M, k, keep, skew, seed):
    rng = np.random.default_rng(seed)
    cand = sorted(rng.choice(M, keep, replace=False).tolist())
    idx, _ = W.gen_routing(T, M, k, cand, seed=seed + 1, skew=skew)
    x = W.f32_to_bf16_bits(rng.standard_normal((T, 128)).astype(np.float32))
    return idx, x


def _noalloc(idx, x, M):
    T, k = idx.shape
    d_idx = up_i32(idx)
    d_x = up(x, W.BF16)
    desc = E.moe_desc(T, M, 1, 128, 128, k, torch.bfloat16)
    seg = torch.full((M + 1,), -7, dtype=torch.int32, device="cuda")
    src = torch.full((T * k,), -7, dtype=torch.int32, device="cuda")
    inv = torch.full((T * k,), -7, dtype=torch.int32, device="cuda")
    xp = torch.zeros((T * k, 128), dtype=torch.bfloat16, device="cuda")
    E.permute_noalloc_into(desc, d_idx, seg, src, inv, x=d_x, x_perm=xp)
    return seg, src, inv, xp, d_idx, d_x


# (T, M, k, candidates, Zipf skew): each call smaller than the one before (120006, 80000, 10000,
# 6000 assignments); the first three
# take the chunked kernels (counts in the library's array), the last the one-workgroup path
CALLS = [(20001, 256, 6, 200, 0.5), (40000, 64, 2, 48, 1.1), (5000, 64, 2, 40, 0.0), (3000, 16, 2, 12, 0.0)]


def test_noalloc_permute_matches_workspace_permute():
    for n, (T, M, k, keep, skew) in enumerate(CALLS):
        say(f"permute_noalloc call {n}: T={T} M={M} k={k}")
        idx, x = _case(T, M, k, keep, skew, seed=100 + n)
        seg, src, inv, xp, d_idx, d_x = _noalloc(idx, x, M)
        wseg, wsrc, winv, wxp = E.permute(d_idx, M, x=d_x)
        torch.cuda.synchronize()
        assert torch.equal(seg, wseg) and torch.equal(src, wsrc) and torch.equal(inv, winv)
        assert torch.equal(xp.view(torch.int16), wxp.view(torch.int16))
        # and the oracle's stable sort
        rseg, rsrc, rinv = O.permute(idx, M)
        np.testing.assert_array_equal(down(seg), rseg)
        np.testing.assert_array_equal(down(src), rsrc)
        np.testing.assert_array_equal(down(inv), rinv)


def test_noalloc_permute_repeats_bit_for_bit():
    """The same input twice, with a different input in between: the leftover counts of the
    other call change nothing."""
    idx_a, x_a = _case(30000, 32, 2, 30, 0.8, seed=7)
    idx_b, x_b = _case(9000, 128, 4, 100, 0.0, seed=8)
    first = _noalloc(idx_a, x_a, 32)[:4]
    _noalloc(idx_b, x_b, 128)
    again = _noalloc(idx_a, x_a, 32)[:4]
    torch.cuda.synchronize()
    for a, b in zip(first, again):
        assert torch.equal(a.view(torch.int32) if a.dtype == torch.int32 else a.view(torch.int16),
                           b.view(torch.int32) if b.dtype == torch.int32 else b.view(torch.int16))
