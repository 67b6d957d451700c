"""Algorithmic work of each kernel of the step, and MI355X peaks.

Counts are what the method must compute or move (no padding, no re-reads): bf16 or
fp32 operands read once, intermediates written once and read once, weights of the
experts that received at least one row read once.
"""
from __future__ import annotations

import hashlib
import json
import os

import numpy as np

# MI355X published peaks
PEAK_HBM_GBS = 8000.0
PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}

_HERE = os.path.dirname(os.path.abspath(__file__))
_ROOT = os.path.dirname(_HERE)


def expert_rows(idx: np.ndarray, n_experts: int) -> np.ndarray:
    return np.bincount(np.asarray(idx).ravel(), minlength=n_experts)


def kernel_work(cfg, rows_per_expert: np.ndarray) -> dict:
    """{kernel: (flop, bytes)} for one step of the layer at this routing."""
    s = 2 if cfg.dtype == "bf16" else 4
    T, d, M, K, H, k = cfg.n_tokens, cfg.d_model, cfg.n_experts, cfg.n_groups, cfg.ffn_hidden, cfg.top_k
    A = T * k
    act = int(np.count_nonzero(rows_per_expert))
    rh, rw = cfg.r_h, cfg.r_w
    c = getattr(cfg, "codec_slices", 1)
    h = T // c
    work = {
        "gate": (2.0 * T * d * (M + K), T * d * s + (M + K) * d * s + 8.0 * T * k),
        "expert_down": (2.0 * A * H * d, act * 1.0 * d * H * s + A * H * s + A * d * s),
        "combine": (2.0 * A * d, A * d * s + 8.0 * T * k + T * d * s),
        "permute": (0.0, 4.0 * A + 12.0 * A),
        # per slice: X V then U^T (X V); U and V read once for all slices
        "encode": (2.0 * T * d * rw + 2.0 * rh * rw * T, T * d * s + (h * rh + d * rw) * s + 4.0 * c * rh * rw),
        # per slice: V Z^T then U (V Z^T)^T
        "decode": (c * 2.0 * d * rw * rh + 2.0 * T * rh * d, T * d * s + (h * rh + d * rw) * s + 4.0 * c * rh * rw),
    }
    if getattr(cfg, "activation", "swiglu") == "relu":
        work["expert_in_relu"] = (2.0 * A * d * H, act * 1.0 * H * d * s + A * d * s + A * H * s)
    else:
        work["expert_gate_up"] = (4.0 * A * d * H, act * 2.0 * H * d * s + A * d * s + A * H * s)
    return work


# Profile name of each library launch on the layer path -> the stage whose algorithmic work
# (kernel_work) it shares. A split-K "<name>_tail" or "<name>_reduce" launch belongs to the
# stage of <name>.
STAGE_OF_KERNEL = {
    "gate": "gate", "gate_split": "gate",
    "perm_onepass": "permute", "perm_count": "permute", "perm_scan": "permute", "perm_scatter": "permute",
    "gather_rows": "permute",
    "transpose": "encode", "codec_xv": "encode", "codec_utp": "encode", "codec_encode": "encode",
    "codec_encode_part": "encode", "codec_encode_finish": "encode",
    "codec_z_bf16": "decode", "codec_prep": "decode", "codec_vzt": "decode", "codec_uw": "decode",
    "codec_decode": "decode",
    "expert_gate_up": "expert_gate_up", "expert_in_relu": "expert_in_relu", "expert_down": "expert_down",
    "combine": "combine",
}


def stage_of(name: str):
    """Stage of a launch's profile name, or None for launches outside the layer step."""
    for suf in ("_tail", "_reduce"):
        if name.endswith(suf):
            name = name[: -len(suf)]
    return STAGE_OF_KERNEL.get(name)


def source_digest(*names: str) -> str:
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(_HERE, "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch recorded from rocprofv3 counters for this kernel and
    workload, or None if absent or taken on a different kernel source."""
    path = os.path.join(_ROOT, "profiles", f"{kernel}_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_digest") != source_digest(*rec.get("sources", [])):
        return None
    return rec.get("hbm_bytes_per_launch")
