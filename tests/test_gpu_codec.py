"""Parity of the low-rank encoder/decoder kernels with the oracle
(Encoder-Decoder based on Low-Rank Compression: Z = U^T X V, X_hat = U_hat Z V_hat^T)."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2508_06024_amd import ec2moe as E
from paper_2508_06024_amd import workload as W
from tests.gpu_common import TOL_F32, assert_close, down, say, tol, up

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", W.CONFIG_ORDER)
def test_codec_matches_oracle_at_full_size(name):
    cfg = W.CONFIGS[name]
    say(f"codec {name}: h={cfg.n_tokens} w={cfg.d_model} r_h={cfg.r_h} r_w={cfg.r_w}")
    inp = W.gen_layer(cfg, experts=False)
    x, u, v = (up(getattr(inp, n), cfg.dtype) for n in ("x", "u", "v"))
    z = E.lowrank_encode(x, u, v)
    xh = E.lowrank_decode(z, u, v)
    torch.cuda.synchronize()
    rz = O.lowrank_encode(inp.f64("x"), inp.f64("u"), inp.f64("v"))
    rxh = O.lowrank_decode(rz, inp.f64("u"), inp.f64("v"))
    ez = assert_close(down(z), rz, TOL_F32, "Z")
    exh = assert_close(down(xh), rxh, tol(cfg.dtype), "X_hat")
    say(f"  Z {ez:.2e}  X_hat {exh:.2e}")


def test_full_rank_codec_round_trips_on_gpu():
    """Square orthogonal U, V (the tiny workload's T=64, d=128 at full rank... r <= 256):
    decode(encode(X)) = X within float32 rounding."""
    cfg = W.CONFIGS["tiny"]
    x = W.gen_call(cfg)[0]
    u = W.haar_orthonormal(5, (1,), 64, 64).astype(np.float32)
    v = W.haar_orthonormal(5, (2,), 128, 128).astype(np.float32)
    z = E.lowrank_encode(up(x, W.F32), up(u, W.F32), up(v, W.F32))
    xh = E.lowrank_decode(z, up(u, W.F32), up(v, W.F32))
    assert_close(down(xh), x.astype(np.float64), 1e-5, "round trip")


@pytest.mark.parametrize("c,h,w,rh,rw,dt", [
    (2, 300, 384, 32, 48, W.BF16),
    (5, 64, 256, 16, 32, W.F32),
    (17, 40, 128, 16, 16, W.BF16),   # more slices than one batch of launches (16)
    (4, 256, 768, 64, 64, W.BF16),   # the paper-shaped layers: 4 sequences of 256 tokens
    (1, 300, 256, 80, 64, W.BF16),   # r_h ending inside the second 64-row block of U^T P
    (2, 260, 128, 208, 112, W.F32),  # ... inside the fourth
    # bf16 layers of whole 64-token, 64-column tiles take the fused encoder:
    (3, 128, 256, 80, 128, W.BF16),   # r_h inside the second 64-row block, two column tiles
    (2, 256, 384, 256, 192, W.BF16),  # three column tiles of a token tile placed on one XCD
    (17, 128, 128, 16, 64, W.BF16),   # two tiles per slice, more slices than one batch
    # one slice of whole 128-token bands with r_h = 128 or 256 takes the decoder's expansion kernel:
    (1, 128, 128, 128, 64, W.BF16),    # one band of two 64-column chunks
    (1, 256, 512, 256, 128, W.BF16),   # with the fused encoder
    (1, 4096, 2176, 128, 64, W.BF16),  # runs of three chunks, the last of each band one chunk (34 chunks)
    # at most 64 tokens per slice take the small-batch encoder and decoder:
    (3, 48, 256, 32, 48, W.BF16),
    (2, 64, 256, 64, 256, W.F32),     # the largest r_h and r_w of that path
])
def test_codec_slices_and_separate_decoder_projections(c, h, w, rh, rw, dt):
    """Several slices coded with one U, V; decoder projections different from the encoder's."""
    say(f"codec slices c={c} h={h} w={w} r={rh}x{rw} {dt}")
    rng = np.random.default_rng(3 + c)
    cast = (lambda a: W.f32_to_bf16_bits(np.asarray(a, np.float32))) if dt == W.BF16 else (lambda a: np.asarray(a, np.float32))
    x = cast(rng.standard_normal((c, h, w)))
    u = cast(W.haar_orthonormal(1, (1,), h, rh))
    v = cast(W.haar_orthonormal(1, (2,), w, rw))
    uh = cast(rng.standard_normal((h, rh)) * 0.1)
    vh = cast(rng.standard_normal((w, rw)) * 0.1)
    z = E.lowrank_encode(up(x, dt), up(u, dt), up(v, dt))
    xh = E.lowrank_decode(z, up(uh, dt), up(vh, dt))
    f = lambda a: W.to_f64(a, dt)
    for s in range(c):
        rz = O.lowrank_encode(f(x[s]), f(u), f(v))
        assert_close(down(z[s]), rz, TOL_F32, f"Z[{s}]")
        assert_close(down(xh[s]), O.lowrank_decode(rz, f(uh), f(vh)), tol(dt), f"X_hat[{s}]")


def test_codec_is_deterministic():
    cfg = W.CONFIGS["small"]
    inp = W.gen_layer(cfg, experts=False)
    x, u, v = (up(getattr(inp, n), cfg.dtype) for n in ("x", "u", "v"))
    z1, z2 = E.lowrank_encode(x, u, v), E.lowrank_encode(x, u, v)
    assert torch.equal(z1, z2)
    assert torch.equal(E.lowrank_decode(z1, u, v), E.lowrank_decode(z2, u, v))
