"""Helpers of the GPU parity tests: device upload of the seeded inputs, the error
metrics, and the routing comparison with its certified near-tie rule."""
from __future__ import annotations

import sys

import numpy as np
import torch

from paper_2508_06024_amd import workload as W

# tolerances: max|gpu - ref| / max|ref| per output tensor
TOL_BF16 = 2e-2
TOL_F32 = 1e-5
# relative gap between consecutive fused probabilities under which the float32 GPU gate
# and the float64 oracle may order two experts differently
NEAR_TIE = 1e-4

DEV = "cuda"


def say(msg: str):
    print(msg, file=sys.stderr, flush=True)


def up(a: np.ndarray, dtype: str) -> torch.Tensor:
    """Stored tensor (uint16 bf16 bits or float32) -> device tensor of the layer dtype."""
    if dtype == W.BF16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(DEV)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def up_i32(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)


def up_f32(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def down(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> exact float64 values (int32 stays int)."""
    t = t.detach()
    if t.dtype == torch.bfloat16:
        return W.to_f64(t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16), W.BF16)
    if t.dtype == torch.int32:
        return t.cpu().numpy()
    return t.float().cpu().numpy().astype(np.float64)


def tol(dtype: str) -> float:
    return TOL_BF16 if dtype == W.BF16 else TOL_F32


def rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = np.max(np.abs(ref)) if ref.size else 0.0
    diff = np.max(np.abs(got - ref)) if ref.size else 0.0
    return float(diff / scale) if scale > 0 else float(diff)


def assert_close(got, ref, tolerance, what=""):
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    e = rel_err(got, ref)
    assert e <= tolerance, f"{what}: max rel error {e:.3e} > {tolerance:.1e}"
    return e


def check_routing(gpu_idx, gpu_w, ref_idx, ref_w, g_ref, cand, k, w_tol=TOL_F32, strict=False):
    """Expert indices must match the oracle bit for bit on every token, except tokens
    whose oracle fused probabilities have a relative gap below NEAR_TIE between
    consecutive ranks 0..k (certified near-ties): there the GPU's j-th pick must carry
    the oracle's j-th largest probability within NEAR_TIE. Weights are compared on the
    tokens routed identically. Returns the number of certified tokens."""
    cand = np.asarray(sorted(cand))
    mism = np.nonzero((gpu_idx != ref_idx).any(axis=1))[0]
    if strict:
        assert mism.size == 0, f"{mism.size} tokens routed differently, first {mism[:5]}"
    for t in mism:
        gs = np.sort(g_ref[t, cand])[::-1]
        nxt = gs[1:k + 1]
        margins = (gs[:nxt.size] - nxt) / gs[:nxt.size]
        assert margins.size and margins.min() < NEAR_TIE, \
            f"token {t}: gpu {gpu_idx[t]} vs oracle {ref_idx[t]} with margins {margins}"
        assert len(set(gpu_idx[t].tolist())) == k
        for j in range(k):
            e = int(gpu_idx[t, j])
            assert e in cand
            assert abs(g_ref[t, e] - gs[j]) <= NEAR_TIE * gs[j], f"token {t} slot {j}"
    same = ~(gpu_idx != ref_idx).any(axis=1)
    if same.any():
        assert_close(gpu_w[same], ref_w[same], w_tol, "topk_w")
    return int(mism.size)
