"""The oracle's pins catch plausible mistakes: each case plants one mistake in a copy of the
oracle (on the CPU, in a temporary directory) and runs the pins against it there, which must
then fail. A planted edit that no longer matches the oracle's text is an error of this test.
The planner's pins load the library's host entry points (no GPU work)."""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PLANNER_PINS = "not library and not zero_capability"  # the planner pins that need no library

# mistakes planted in oracle/planner_oracle.py (Eq. 2-4, 9-11)
PLANNER_MUTATIONS = [
    ("capability without the bandwidth term (Eq. 3)",
     '+ params["w_power"] * state["power"] + params["w_bandwidth"] * state["bandwidth"])',
     '+ params["w_power"] * state["power"])'),
    ("the cap keeps the experts of largest f",
     "key=lambda i: (complexity[i] / cap, i))[:limit]", "key=lambda i: (-complexity[i] / cap, i))[:limit]"),
    ("tasks taken in ascending priority (Eq. 11)",
     "order = sorted(range(n), key=lambda i: (-prio[i], i))", "order = sorted(range(n), key=lambda i: (prio[i], i))"),
    ("end placement ignores the priority threshold",
     'if load_end + complexity[i] <= params["t_end"] and prio[i] >= params["beta"]:',
     'if load_end + complexity[i] <= params["t_end"]:'),
    ("communication charged to end-side tasks (Eq. 9)",
     "(0.0 if end else comm[i])", "comm[i]"),
]

# (what the mistake is, text of the oracle, planted replacement)
MUTATIONS = [
    ("gate and up branches swapped (SwiGLU)",
     "act = silu(h[:, :H]) * h[:, H:]", "act = silu(h[:, H:]) * h[:, :H]"),
    ("sign of the SiLU exponent",
     "return z / (1.0 + np.exp(-z))", "return z / (1.0 + np.exp(z))"),
    ("ReLU dropped from the Switch experts",
     "return np.maximum(h, 0.0) @", "return h @"),
    ("local biases dropped (Eq. 5)",
     "local_logits = x @ np.asarray(w_local, np.float64).T + np.asarray(b_local, np.float64)",
     "local_logits = x @ np.asarray(w_local, np.float64).T"),
    ("group biases dropped (Eq. 6)",
     "group_logits = x @ np.asarray(w_global, np.float64).T + np.asarray(b_global, np.float64)",
     "group_logits = x @ np.asarray(w_global, np.float64).T"),
    ("group softmax over every group, empty ones included (Eq. 4, 6)",
     "p_group = softmax(group_logits_t[active])", "p_group = softmax(group_logits_t)[active]"),
    ("candidate mask ignored (Eq. 4)",
     "cand_in_group = [[i for i in grp if i in cand] for grp in groups]",
     "cand_in_group = [list(grp) for grp in groups]"),
    ("group probability left out of the fusion (Eq. 7)",
     "g[i] = p_group[a] * pl", "g[i] = pl"),
    ("exact ties go to the higher expert index",
     "order = sorted(cand, key=lambda i: (-g_row[i], i))", "order = sorted(cand, key=lambda i: (-g_row[i], -i))"),
    ("selected weights not renormalised",
     "w[t] = w[t] / w[t].sum()", "w[t] = w[t]"),
    ("top-G groups stop before they hold k candidates",
     "if len(kept) >= top_groups and held >= min_candidates:", "if len(kept) >= top_groups:"),
    ("permutation sorted without keeping the input order inside a segment",
     'order = np.argsort(flat, kind="stable")', 'order = np.argsort(flat, kind="quicksort")'),
    ("top-G ranking ties to the higher group index",
     "order = sorted(range(len(active)), key=lambda a: (-p_group[a], active[a]))",
     "order = sorted(range(len(active)), key=lambda a: (-p_group[a], -active[a]))"),
    ("unequal groups start one expert late",
     "starts = np.concatenate([[0], np.cumsum(group_sizes)])", "starts = np.concatenate([[1], 1 + np.cumsum(group_sizes)])"),
    ("inverse permutation taken as the permutation itself",
     "inv_perm[order] = np.arange(flat.size, dtype=np.int32)", "inv_perm[:] = order"),
    ("combine without the gate weights (Eq. 1)",
     "y += w[:, j:j + 1] * y_perm[inv_perm.reshape(T, k)[:, j]]", "y += y_perm[inv_perm.reshape(T, k)[:, j]]"),
    ("encoder without U^T",
     "return np.asarray(u, np.float64).T @ np.asarray(x, np.float64) @ np.asarray(v, np.float64)",
     "return np.asarray(x, np.float64) @ np.asarray(v, np.float64)"),
    ("decoder with V_hat where its transpose belongs",
     "@ np.asarray(z, np.float64) @ np.asarray(v_hat, np.float64).T", "@ np.asarray(z, np.float64) @ np.asarray(v_hat, np.float64)"),
    ("fit: R's diagonal left with either sign (basis not the positive-diagonal QR)",
     "    return q * s\n", "    return q\n"),
    ("fit: the Gram matrices of the two sides swapped (Eq. 8)",
     "return iterate(a, omega_u), iterate(b, omega_v)", "return iterate(b, omega_u), iterate(a, omega_v)"),
    ("fit: V from the mode-1 unfolding",
     "v = np.linalg.svd(_unfold_cols(xs), full_matrices=False)[0][:, :r_w]",
     "v = np.linalg.svd(_unfold_rows(xs), full_matrices=False)[0][:, :r_w]"),
    ("fit: one power step fewer than asked",
     "        for _ in range(iters):\n            q = orthonormal_basis(g @ q)",
     "        for _ in range(iters - 1):\n            q = orthonormal_basis(g @ q)"),
    ("experts run on X instead of the reconstruction X_hat",
     "y = moe_forward(x_hat, idx, w, w_gate_up, w_down, activation)", "y = moe_forward(x, idx, w, w_gate_up, w_down, activation)"),
]


def _tree(tmp, mutation, module="ec2moe_oracle.py", pins="test_oracle_pins.py"):
    """A copy of what the pins import, with the mistake planted in the oracle."""
    dst = os.path.join(tmp, "tree")
    shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(dst, "oracle"),
                    ignore=shutil.ignore_patterns("__pycache__"))
    shutil.copytree(os.path.join(ROOT, "paper_2508_06024_amd"), os.path.join(dst, "paper_2508_06024_amd"),
                    ignore=shutil.ignore_patterns("__pycache__", "_build", "csrc"))
    shutil.copytree(os.path.join(ROOT, "tests"), os.path.join(dst, "tests"),
                    ignore=shutil.ignore_patterns("__pycache__", "test_*.py"))
    shutil.copy(os.path.join(ROOT, "tests", pins), os.path.join(dst, "tests"))
    path = os.path.join(dst, "oracle", module)
    with open(path) as f:
        src = f.read()
    _, old, new = mutation
    assert src.count(old) == 1, f"planted edit does not match the oracle once: {old!r}"
    with open(path, "w") as f:
        f.write(src.replace(old, new))
    return dst


def _run_pins(tree, pins="test_oracle_pins.py", select=None):
    env = dict(os.environ, PYTHONDONTWRITEBYTECODE="1", OMP_NUM_THREADS="1", OPENBLAS_NUM_THREADS="1")
    cmd = [sys.executable, "-m", "pytest", f"tests/{pins}", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu"]
    if select:
        cmd += ["-k", select]
    return subprocess.run(cmd, cwd=tree, env=env, capture_output=True, text=True, timeout=300)


def test_unmodified_copy_passes(tmp_path):
    """The copied tree is sound: with no mistake planted every pin passes there."""
    tree = _tree(os.path.join(tmp_path, "a"), ("none", "def softmax(v):", "def softmax(v):"))
    r = _run_pins(tree)
    assert r.returncode == 0, r.stdout[-2000:]
    tree = _tree(os.path.join(tmp_path, "b"), ("none", "def capability(", "def capability("), "planner_oracle.py",
                 "test_planner.py")
    r = _run_pins(tree, "test_planner.py", PLANNER_PINS)
    assert r.returncode == 0 and "passed" in r.stdout, r.stdout[-2000:]


def test_every_planted_mistake_fails_a_pin(tmp_path):
    cases = [(m, "ec2moe_oracle.py", "test_oracle_pins.py", None) for m in MUTATIONS]
    cases += [(m, "planner_oracle.py", "test_planner.py", PLANNER_PINS) for m in PLANNER_MUTATIONS]

    def one(i):
        m, module, pins, select = cases[i]
        tree = _tree(os.path.join(tmp_path, str(i)), m, module, pins)
        return m[0], _run_pins(tree, pins, select)
    with ThreadPoolExecutor(max_workers=4) as ex:
        results = list(ex.map(one, range(len(cases))))
    survived = [name for name, r in results if r.returncode == 0]
    assert not survived, f"mistakes no pin catches: {survived}"
    for name, r in results:
        assert "failed" in r.stdout or "error" in r.stdout.lower(), f"{name}: {r.stdout[-500:]}"
