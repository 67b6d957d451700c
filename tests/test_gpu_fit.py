"""Data-free fitting of the codec projections on the GPU (Eq. 8 with lambda = 0) against
the oracle: the same subspace iteration in float64, the truncated SVD it converges to,
and the Eckart-Young error of one slice."""
import time

import numpy as np
import pytest
import torch

import oracle as O
from paper_2508_06024_amd import ec2moe as E
from paper_2508_06024_amd import workload as W
from tests.gpu_common import down, say, up, up_f32

pytestmark = pytest.mark.gpu


def _slices(c, h, w, r, dt, seed, gap=True):
    """c slices sharing singular vectors, leading r values well above the rest (per-slice
    scales), rounded to the layer dtype; returns (stored, exact float64)."""
    rng = np.random.default_rng(seed)
    n = min(h, w)
    sv = np.concatenate([np.linspace(8.0, 4.0, r), np.linspace(1.0, 0.05, n - r)]) if gap else np.linspace(4, 0.05, n)
    p = W.haar_orthonormal(seed, (1,), h, n)
    q = W.haar_orthonormal(seed, (2,), w, n)
    xs = np.stack([(p * (sv * rng.uniform(0.9, 1.1, n))) @ q.T for _ in range(c)]).astype(np.float32)
    stored = W.f32_to_bf16_bits(xs) if dt == W.BF16 else xs
    return stored, W.to_f64(stored, dt)


def _omega(n, r, seed):
    return np.random.default_rng(seed).standard_normal((n, r)).astype(np.float32)


def _proj(a):
    return a @ a.T


@pytest.mark.parametrize("c,h,w,rh,rw,dt,iters,tol", [
    (1, 128, 256, 16, 32, W.F32, 3, 1e-5),
    (3, 96, 128, 16, 16, W.F32, 5, 1e-5),
    (4, 256, 768, 64, 64, W.BF16, 4, 2e-2),   # the paper-shaped layers' calibration block
    (2, 64, 128, 48, 48, W.F32, 3, 1e-5),     # rank not a multiple of 32
    (1, 320, 384, 256, 256, W.F32, 2, 1e-5),  # the largest rank: every block of the factorisation
])
def test_fit_matches_oracle_iteration(c, h, w, rh, rw, dt, iters, tol):
    say(f"fit c={c} h={h} w={w} r={rh}x{rw} {dt} iters={iters}")
    xs, x64 = _slices(c, h, w, max(rh, rw), dt, seed=c + h)
    ou, ov = _omega(h, rh, 1), _omega(w, rw, 2)
    u, v, status = E.lowrank_fit(up(xs, dt), up_f32(ou), up_f32(ov), iters)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    ru, rv = O.codec_fit_subspace(x64, ou.astype(np.float64), ov.astype(np.float64), iters)
    gu, gv = down(u), down(v)
    for g, ref, name in ((gu, ru, "U"), (gv, rv, "V")):
        e = np.max(np.abs(_proj(g) - _proj(ref)))
        assert e <= tol, f"{name} projector error {e:.2e}"
        o = np.max(np.abs(g.T @ g - np.eye(g.shape[1])))
        assert o <= (1e-5 if dt == W.F32 else 2e-2), f"{name} orthonormality error {o:.2e}"
        say(f"  {name}: projector error {e:.2e}, orthonormality {o:.2e}")


def test_fit_full_size_matches_oracle_iteration():
    """A 4096 x 4096 calibration block at rank 256, one iteration: its Gram products are large
    enough for the 256 x 256 matrix-core tile with float32 output (the only path that uses that
    tile's float32 writer). Projectors against the oracle's iteration on the same bf16 block."""
    h = w = 4096
    r = 256
    rng = np.random.default_rng(21)
    x = (rng.standard_normal((h, w)) * np.linspace(3.0, 0.1, w)).astype(np.float32)[None]
    stored = W.f32_to_bf16_bits(x)
    x64 = W.to_f64(stored, W.BF16)
    ou, ov = _omega(h, r, 8), _omega(w, r, 9)
    u, v, status = E.lowrank_fit(up(stored, W.BF16), up_f32(ou), up_f32(ov), 1)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    ru, rv = O.codec_fit_subspace(x64, ou.astype(np.float64), ov.astype(np.float64), 1)
    for g, ref, name in ((down(u), ru, "U"), (down(v), rv, "V")):
        e = np.max(np.abs(_proj(g) - _proj(ref)))
        say(f"  4096 x 4096, r = 256: {name} projector error {e:.2e}")
        assert e <= 2e-2, f"{name} projector error {e:.2e}"


def test_fit_one_slice_reaches_eckart_young():
    """Enough iterations for the gap: the fitted codec's error is the tail of the spectrum."""
    h, w, r = 512, 384, 32
    xs, x64 = _slices(1, h, w, r, W.F32, seed=9)
    u, v, status = E.lowrank_fit(up(xs, W.F32), up_f32(_omega(h, r, 3)), up_f32(_omega(w, r, 4)), 12)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    gu, gv = down(u), down(v)
    x = x64[0]
    err = np.sum((x - gu @ (gu.T @ x @ gv) @ gv.T) ** 2)
    s = np.linalg.svd(x, compute_uv=False)
    np.testing.assert_allclose(err, np.sum(s[r:] ** 2), rtol=1e-3)
    ru, rv = O.codec_fit_hosvd(x64, r, r)
    assert np.max(np.abs(_proj(gu) - _proj(ru))) < 1e-3


def test_fit_rank_deficient_start_sets_status():
    """A zero start block has no column rank: the Cholesky pivots fail, the kernels finish
    and the status word says so."""
    h, w, r = 64, 128, 16
    xs, _ = _slices(1, h, w, r, W.F32, seed=11)
    u, v, status = E.lowrank_fit(up(xs, W.F32), up_f32(np.zeros((h, r), np.float32)), up_f32(_omega(w, r, 5)), 1)
    torch.cuda.synchronize()
    assert int(status.item()) == 1
    assert np.all(np.isfinite(down(u))) and np.all(np.isfinite(down(v)))


def test_fit_full_size_timing():
    """The Mixtral-shaped calibration block (4096 x 4096, rank 256): orthonormal outputs whose
    projection keeps the block's leading energy; the time is reported."""
    h = w = 4096
    r = 256
    rng = np.random.default_rng(12)
    x = torch.from_numpy(rng.standard_normal((h, w)).astype(np.float32)).to("cuda")
    x = (x @ torch.diag(torch.linspace(3.0, 0.1, w, device="cuda"))).to(torch.bfloat16).contiguous()
    ou, ov = up_f32(_omega(h, r, 6)), up_f32(_omega(w, r, 7))
    E.lowrank_fit(x, ou, ov, 1)  # warm-up
    torch.cuda.synchronize()
    t = time.perf_counter()
    u, v, status = E.lowrank_fit(x, ou, ov, 4)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t) * 1e3
    say(f"  fit 4096x4096 r=256, 4 iterations: {ms:.1f} ms")
    assert int(status.item()) == 0
    uf, vf = u.float(), v.float()
    eye = torch.eye(r, device="cuda")
    assert torch.max(torch.abs(uf.T @ uf - eye)).item() < 3e-2
    assert torch.max(torch.abs(vf.T @ vf - eye)).item() < 3e-2
