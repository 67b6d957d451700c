"""The algorithmic work that the benchmark's roofline figures divide by: hand-computed
counts for the Mixtral-shaped layer (SwiGLU experts, Eq. 1) and the codec."""
import numpy as np

from paper_2508_06024_amd import roofline as R
from paper_2508_06024_amd import workload as W


def test_mixtral_gate_up_and_down_work():
    cfg = W.CONFIGS["mixtral"]  # T 4096, d 4096, 8 experts, H 14336, top-2, bf16
    w = R.kernel_work(cfg, np.full(8, 1024))
    # gate-up: 4 A d H flop (two products of 2 A d H), A = 8192
    assert w["expert_gate_up"][0] == 4 * 8192 * 4096 * 14336 == 1_924_145_348_608
    # bytes: 8 experts' [2H][d] bf16 weights, the A gathered token rows, the A x H act rows
    assert w["expert_gate_up"][1] == 8 * 2 * 14336 * 4096 * 2 + 8192 * 4096 * 2 + 8192 * 14336 * 2 == 2_181_038_080
    assert w["expert_down"] == (2 * 8192 * 14336 * 4096, 8 * 4096 * 14336 * 2 + 8192 * 14336 * 2 + 8192 * 4096 * 2)
    # combine: read the A output rows, the routing (idx + weight, 8 bytes per slot), write T rows
    assert w["combine"][1] == 8192 * 4096 * 2 + 8 * 4096 * 2 + 4096 * 4096 * 2


def test_only_experts_with_rows_count_their_weights():
    cfg = W.CONFIGS["mixtral"]
    rows = np.array([2048, 2048, 1024, 1024, 1024, 1024, 0, 0])
    full = R.kernel_work(cfg, np.full(8, 1024))
    some = R.kernel_work(cfg, rows)
    weights = 2 * 14336 * 4096 * 2
    assert full["expert_gate_up"][1] - some["expert_gate_up"][1] == 2 * weights
    assert full["expert_gate_up"][0] == some["expert_gate_up"][0]  # flops follow the assignments


def test_codec_work():
    cfg = W.CONFIGS["mixtral"]  # one slice of 4096 x 4096, r 256 x 256
    w = R.kernel_work(cfg, np.full(8, 1024))
    # encode: X V (2 T d r_w) then U^T P (2 r_h r_w T); X, U, V read once, Z written in float32
    assert w["encode"] == (2 * 4096 * 4096 * 256 + 2 * 256 * 256 * 4096,
                           4096 * 4096 * 2 + (4096 * 256 + 4096 * 256) * 2 + 4 * 256 * 256)
    # gate: the logits of M + K rows; X and the gate weights read once, the routing written
    assert w["gate"] == (2 * 4096 * 4096 * 10, 4096 * 4096 * 2 + 10 * 4096 * 2 + 8 * 4096 * 2)


def test_every_layer_launch_has_a_stage():
    """Each profile name the library gives a launch (the ProfileScope literals and the GEMM
    names set in the sources) maps to a stage with algorithmic work, so the per-stage
    figures of bench.py cover every kernel of the step. Fitting and the generic GEMM name
    are outside the layer step."""
    import os
    import re
    csrc = os.path.join(os.path.dirname(R.__file__), "csrc")
    names = set()
    for f in os.listdir(csrc):
        text = open(os.path.join(csrc, f)).read()
        for line in text.splitlines():
            if "ProfileScope prof(" in line or re.search(r"\.name = ", line):
                names.update(re.findall(r'"([a-z_0-9]+)"', line))
    names -= {"gemm"}
    names = {n for n in names if not n.startswith("fit_")}
    assert {"codec_encode", "codec_vzt", "expert_gate_up", "gate"} <= names
    stages = set(R.kernel_work(W.CONFIGS["mixtral"], np.ones(8, np.int64))) | {"expert_in_relu"}
    for n in sorted(names):
        assert R.stage_of(n) in stages, n
        assert R.stage_of(n + "_tail") == R.stage_of(n)
