"""Seeded synthetic workloads for the group-gated MoE layer and the low-rank codec.

This module only draws numbers and lays them out. It holds none of the layer's
arithmetic (no gate, no softmax, no top-k, no FFN, no projection): the CPU oracle
and the HIP path both take their inputs from here, and nothing else is shared
between them.

Shapes follow the paper's problem statement:
  * hidden states X [T][d] (tokens x model width),
  * per-group gate weights W_k stacked into W_local [M][d] with biases b_local [M]
    and the global group gate W_global [K][d], b_global [K]
    (Lightweight Group Gate Network, Eq. 5 and Eq. 6),
  * the hardware-aware candidate set E_local as a bitmask over the M experts
    (Local Expert Selection, Eq. 4),
  * SwiGLU expert weights W_gate_up [M][2H][d] (rows 0..H-1 gate branch, rows
    H..2H-1 up branch) and W_down [M][d][H], or for two-layer ReLU experts (the
    Switch Transformer FFN of the paper's experiments) W_in [M][H][d] in the same
    array and W_down [M][d][H],
  * codec projections U [h][r_h], V [d][r_w] (Encoder-Decoder based on
    Low-Rank Compression, Z = U^T X V), applied to each of the c slices X[s] =
    rows s*h .. (s+1)*h - 1 of X, h = T / c.

Every tensor has its own PCG64 stream, keyed by (seed, tensor tag[, expert]), so
one expert's weights can be regenerated without drawing the others and the
experts can be drawn on several threads. Normals are drawn in float32, scaled in
float64, then rounded to the layer dtype: float32, or bfloat16 by
round-to-nearest-even on the bit pattern. bfloat16 tensors are returned as
uint16 bit patterns.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor
from typing import List, Optional, Sequence

import numpy as np

F32 = "f32"
BF16 = "bf16"

# stream tags (one PCG64 stream per tensor)
_TAG_MASK, _TAG_X, _TAG_WG, _TAG_WL, _TAG_POP, _TAG_WGU, _TAG_WD, _TAG_U, _TAG_V = range(9)


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    """One synthetic MoE layer + codec workload."""
    name: str
    dtype: str            # F32 or BF16: storage and MFMA operand type of every tensor
    n_tokens: int         # T
    d_model: int          # d
    n_experts: int        # M
    n_groups: int         # K (contiguous equal groups of M/K experts)
    ffn_hidden: int       # H
    top_k: int            # k
    r_h: int              # codec rank on the token side
    r_w: int              # codec rank on the feature side
    seed: int
    mask: str             # "fixed", "random", "all" or "per_call"
    n_keep: int = 0       # experts kept by a "random" mask
    masked_out: tuple = ()  # experts removed by a "fixed" mask
    x_dist: str = "normal"  # "normal" (N(0, x_std^2)) or "rms" (N(0,1) rows scaled to unit RMS)
    x_std: float = 1.0
    gate_std: Optional[float] = None  # None -> 1/sqrt(d) (unit-variance logits)
    expert_std: float = 0.02
    zipf_s: float = 0.0   # > 0: gate biases make expert popularity Zipf(s)
    keep_range: tuple = ()  # "per_call": n_keep drawn uniformly from this closed range
    n_calls: int = 1      # "per_call": number of distinct (X, mask) draws timed
    first_call_seed: int = 0
    activation: str = "swiglu"  # expert FFN: "swiglu" or "relu"
    codec_slices: int = 1  # c: X is c slices of h = T / c rows, each coded with the same U, V

    @property
    def group_size(self) -> int:
        return self.n_experts // self.n_groups

    @property
    def w_in_rows(self) -> int:
        """Rows of one expert's input-layer weight (gate and up branches, or W_in)."""
        return self.ffn_hidden if self.activation == "relu" else 2 * self.ffn_hidden

    @property
    def codec_h(self) -> int:
        return self.n_tokens // self.codec_slices

    @property
    def n_assign(self) -> int:
        return self.n_tokens * self.top_k

    def scaled(self, **kw) -> "LayerConfig":
        return dataclasses.replace(self, **kw)


def default_groups(n_experts: int) -> int:
    """K = 2^floor(log2(sqrt(M))): 8 -> 2, 16 -> 4, 64 -> 8 (contiguous equal groups)."""
    k = 1
    while (2 * k) * (2 * k) <= n_experts:
        k *= 2
    return k


CONFIGS = {
    # tiny fp32 layer the oracle finishes instantly
    "tiny": LayerConfig("tiny", F32, 64, 128, 8, 2, 256, 2, 16, 16, seed=0,
                        mask="fixed", masked_out=(2, 7), x_dist="normal", x_std=0.02,
                        gate_std=0.02),
    # small bf16 layer, uniform routing over a random 12 of 16 experts
    "small": LayerConfig("small", BF16, 1024, 1024, 16, 4, 2816, 2, 128, 128, seed=1,
                         mask="random", n_keep=12, x_dist="normal", x_std=1.0,
                         gate_std=None),
    # Mixtral-shaped bf16 layer: 8 experts, d=4096, H=14336, top-2, all experts kept
    "mixtral": LayerConfig("mixtral", BF16, 4096, 4096, 8, 2, 14336, 2, 256, 256, seed=2,
                           mask="all", x_dist="rms", gate_std=0.02),
    # fine-grained layer with Zipf(1.1) expert popularity, 48 of 64 experts kept
    "finegrained": LayerConfig("finegrained", BF16, 8192, 2048, 64, 8, 1408, 6, 128, 128,
                               seed=3, mask="random", n_keep=48, x_dist="rms",
                               gate_std=0.02, zipf_s=1.1),
    # decode-like memory-bound layer; a fresh mask keeping 16..64 experts per call
    "decode": LayerConfig("decode", BF16, 32, 4096, 64, 8, 1536, 8, 32, 64, seed=4,
                          mask="per_call", keep_range=(16, 64), x_dist="rms",
                          gate_std=0.02, n_calls=1000, first_call_seed=4),
}
CONFIG_ORDER = ["tiny", "small", "mixtral", "finegrained", "decode"]


def switch_config(n_experts: int) -> LayerConfig:
    """The paper's experimental setting (Parameter Selection): a batch of 4 sequences of
    256 tokens, top-1 routing, a candidate set capped at 40% of the experts (here exactly
    floor(0.4 M), drawn at random), experts in K = default_groups(M) groups. Experts are
    Switch-style two-layer ReLU FFNs; the paper does not state the model width, so
    d = 768 and H = 3072 are a stated synthetic choice. The codec treats each sequence
    as one slice X[s] of 256 x 768 (X in R^{h x w x c} with h = 256, w = 768, c = 4),
    rank 64 on both sides."""
    M = n_experts
    return LayerConfig(f"switch{M}", BF16, 1024, 768, M, default_groups(M), 3072, 1, 64, 64,
                       seed=100 + M, mask="random", n_keep=(2 * M) // 5, x_dist="rms",
                       gate_std=0.02, activation="relu", codec_slices=4)


for _m in (8, 16, 32, 64):
    CONFIGS[f"switch{_m}"] = switch_config(_m)
SWITCH_ORDER = ["switch8", "switch16", "switch32", "switch64"]
ALL_ORDER = CONFIG_ORDER + SWITCH_ORDER


# ----------------------------------------------------------------------------- bit formats

def f32_to_bf16_bits(a) -> np.ndarray:
    """Round float32 values to bfloat16, nearest-even, returned as uint16 bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(bits) -> np.ndarray:
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def to_f64(a, dtype: str) -> np.ndarray:
    """Exact float64 value of a stored tensor (uint16 bf16 bits or float32)."""
    if dtype == BF16:
        return bf16_bits_to_f32(a).astype(np.float64)
    return np.asarray(a, dtype=np.float32).astype(np.float64)


def _store(a64: np.ndarray, dtype: str) -> np.ndarray:
    a32 = np.asarray(a64, dtype=np.float32)
    return f32_to_bf16_bits(a32) if dtype == BF16 else np.ascontiguousarray(a32)


def mask_words(experts: Sequence[int], n_experts: int) -> List[int]:
    """Bitmask of the candidate experts: bit e of word e // 64."""
    words = [0] * ((n_experts + 63) // 64)
    for e in experts:
        words[int(e) // 64] |= 1 << (int(e) % 64)
    return words


def mask_members(words: Sequence[int], n_experts: int) -> List[int]:
    return [e for e in range(n_experts) if (int(words[e // 64]) >> (e % 64)) & 1]


# ----------------------------------------------------------------------------- generators

def _rng(seed: int, *key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=key)))


def _normal(seed: int, key: tuple, shape, std: float) -> np.ndarray:
    z = _rng(seed, *key).standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        z *= np.float32(std)
    return z


def haar_orthonormal(seed: int, key: tuple, n: int, r: int) -> np.ndarray:
    """n x r matrix with orthonormal columns (r <= n), Haar distributed: QR of a
    standard normal matrix with R's diagonal made positive."""
    assert r <= n
    a = _rng(seed, *key).standard_normal((n, r))
    q, rr = np.linalg.qr(a)
    s = np.sign(np.diag(rr))
    s[s == 0] = 1.0
    return q * s


def _draw_x(cfg: LayerConfig, seed: int, key: tuple) -> np.ndarray:
    shape = (cfg.n_tokens, cfg.d_model)
    if cfg.x_dist == "rms":
        z = _rng(seed, *key).standard_normal(shape, dtype=np.float32).astype(np.float64)
        z /= np.sqrt(np.mean(z * z, axis=1, keepdims=True))
        return z
    return _normal(seed, key, shape, cfg.x_std).astype(np.float64)


def _draw_mask(cfg: LayerConfig, seed: int, key: tuple) -> List[int]:
    M = cfg.n_experts
    if cfg.mask == "all":
        keep = range(M)
    elif cfg.mask == "fixed":
        keep = [e for e in range(M) if e not in cfg.masked_out]
    elif cfg.mask == "random":
        keep = _rng(seed, *key).choice(M, cfg.n_keep, replace=False)
    elif cfg.mask == "per_call":
        rng = _rng(seed, *key)
        lo, hi = cfg.keep_range
        n_keep = int(rng.integers(lo, hi + 1))
        keep = rng.choice(M, n_keep, replace=False)
    else:
        raise ValueError(cfg.mask)
    return mask_words(sorted(int(e) for e in keep), M)


@dataclasses.dataclass
class LayerInputs:
    cfg: LayerConfig
    x: np.ndarray          # [T][d]
    mask: List[int]        # candidate bitmask words
    w_global: np.ndarray   # [K][d]
    b_global: np.ndarray   # [K] float32
    w_local: np.ndarray    # [M][d]
    b_local: np.ndarray    # [M] float32
    w_gate_up: np.ndarray  # [M][2H][d] (SwiGLU) or [M][H][d] (ReLU)
    w_down: np.ndarray     # [M][d][H]
    u: np.ndarray          # [h][r_h], h = T / codec_slices
    v: np.ndarray          # [d][r_w]

    def f64(self, name: str) -> np.ndarray:
        return to_f64(getattr(self, name), self.cfg.dtype)


def zipf_popularity(cfg: LayerConfig, seed: int) -> np.ndarray:
    """Target expert popularity z (sums to 1): z_i proportional to rank_i^-s with a random
    assignment of ranks 1..M to experts."""
    M = cfg.n_experts
    ranks = _rng(seed, _TAG_POP).permutation(M) + 1
    z = ranks.astype(np.float64) ** (-cfg.zipf_s)
    return z / z.sum()


def _zipf_biases(cfg: LayerConfig, seed: int):
    """Biases for which zero gate weights reproduce the popularity z exactly:
    the group softmax gives each group its total popularity and the in-group softmax
    each expert's share of it."""
    z = zipf_popularity(cfg, seed)
    Mk = cfg.group_size
    zg = np.array([z[k * Mk:(k + 1) * Mk].sum() for k in range(cfg.n_groups)])
    b_global = np.log(zg)
    b_local = np.log(z) - np.repeat(np.log(zg), Mk)
    return b_global.astype(np.float32), b_local.astype(np.float32)


def gen_expert(cfg: LayerConfig, e: int, seed: Optional[int] = None):
    """(W_gate_up[e] [2H][d] or W_in[e] [H][d], W_down[e] [d][H]) in storage format."""
    s = cfg.seed if seed is None else seed
    H, d = cfg.ffn_hidden, cfg.d_model
    gu = _normal(s, (_TAG_WGU, e), (cfg.w_in_rows, d), cfg.expert_std)
    dn = _normal(s, (_TAG_WD, e), (d, H), cfg.expert_std)
    if cfg.dtype == BF16:
        return f32_to_bf16_bits(gu), f32_to_bf16_bits(dn)
    return gu, dn


def gen_experts(cfg: LayerConfig, threads: Optional[int] = None):
    M, H, d = cfg.n_experts, cfg.ffn_hidden, cfg.d_model
    st = np.uint16 if cfg.dtype == BF16 else np.float32
    w_gu = np.empty((M, cfg.w_in_rows, d), dtype=st)
    w_dn = np.empty((M, d, H), dtype=st)

    def one(e):
        a, b = gen_expert(cfg, e)
        w_gu[e] = a
        w_dn[e] = b

    n = threads or min(16, len(os.sched_getaffinity(0)))
    with ThreadPoolExecutor(max(1, n)) as ex:
        list(ex.map(one, range(M)))
    return w_gu, w_dn


def gen_call(cfg: LayerConfig, call_seed: Optional[int] = None):
    """The per-call part of a workload: (X, mask). For "per_call" configs each call seed
    gives a fresh X and a fresh mask; otherwise call_seed is ignored."""
    if cfg.mask == "per_call":
        s = cfg.first_call_seed if call_seed is None else call_seed
        x = _draw_x(cfg, s, (1, _TAG_X))
        mask = _draw_mask(cfg, s, (1, _TAG_MASK))
    else:
        x = _draw_x(cfg, cfg.seed, (_TAG_X,))
        mask = _draw_mask(cfg, cfg.seed, (_TAG_MASK,))
    return _store(x, cfg.dtype), mask


def gen_layer(cfg: LayerConfig, call_seed: Optional[int] = None, experts: bool = True,
              threads: Optional[int] = None) -> LayerInputs:
    """All inputs of one layer call. With experts=False the expert weights are left as
    zero-size arrays (for tests of the gate, permutation and codec alone)."""
    s = cfg.seed
    T, d, M, K = cfg.n_tokens, cfg.d_model, cfg.n_experts, cfg.n_groups
    x, mask = gen_call(cfg, call_seed)
    gstd = cfg.gate_std if cfg.gate_std is not None else 1.0 / np.sqrt(d)
    w_global = _normal(s, (_TAG_WG,), (K, d), gstd)
    w_local = _normal(s, (_TAG_WL,), (M, d), gstd)
    if cfg.zipf_s > 0:
        b_global, b_local = _zipf_biases(cfg, s)
    else:
        b_global = np.zeros(K, np.float32)
        b_local = np.zeros(M, np.float32)
    if experts:
        w_gu, w_dn = gen_experts(cfg, threads)
    else:
        st = np.uint16 if cfg.dtype == BF16 else np.float32
        w_gu = np.zeros((0, cfg.w_in_rows, d), st)
        w_dn = np.zeros((0, d, cfg.ffn_hidden), st)
    u = haar_orthonormal(s, (_TAG_U,), cfg.codec_h, cfg.r_h)
    v = haar_orthonormal(s, (_TAG_V,), d, cfg.r_w)
    return LayerInputs(cfg, x, mask, _store(w_global, cfg.dtype), b_global,
                       _store(w_local, cfg.dtype), b_local, w_gu, w_dn,
                       _store(u, cfg.dtype), _store(v, cfg.dtype))


def gen_routing(T: int, M: int, k: int, cand: Sequence[int], seed: int,
                skew: float = 0.0):
    """Seeded routing for stage tests of the permutation, experts and combine:
    k distinct candidate experts per token (optionally Zipf-skewed toward the low
    candidates) and positive weights that sum to 1 per token. Returns
    (idx int32 [T][k], w float32 [T][k])."""
    rng = _rng(seed, 99)
    cand = np.asarray(sorted(cand), dtype=np.int64)
    assert len(cand) >= k
    if skew > 0:
        p = (np.arange(1, len(cand) + 1, dtype=np.float64)) ** (-skew)
        p /= p.sum()
    else:
        p = None
    idx = np.empty((T, k), np.int32)
    for t in range(T):
        idx[t] = cand[rng.choice(len(cand), k, replace=False, p=p)]
    w = rng.random((T, k)).astype(np.float64) + 0.05
    w /= w.sum(axis=1, keepdims=True)
    return idx, w.astype(np.float32)
