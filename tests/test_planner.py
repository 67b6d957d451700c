"""The end-side planner: hardware-aware local expert selection (Eq. 2-4, with the 40%
candidate cap of Parameter Selection) and the route-aware greedy scheduler (Eq. 9-11).
The oracle is pinned by hand-worked examples and invariants; the library's host entry
points (no GPU work) must match it exactly on seeded random instances."""
import json
import math
import os
import time

import numpy as np
import pytest

import oracle.planner_oracle as PO
from paper_2508_06024_amd import ec2moe as E
from paper_2508_06024_amd import workload as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "planner_hand.json")


def _hand():
    with open(GOLDEN) as f:
        return json.load(f)


def _state(d):
    return E.DeviceState(d["cpu"], d["mem"], d["power"], d["bandwidth"])


def _sel(d):
    return E.SelectionParams(d["w_cpu"], d["w_mem"], d["w_power"], d["w_bandwidth"], d["epsilon"], d["max_fraction"])


def _sched(d):
    return E.ScheduleParams(*(d[n] for n in ("alpha", "beta", "epsilon", "t_end", "load_end", "load_cloud",
                                             "speed_end", "speed_cloud")))


# ----------------------------------------------------------------------------- oracle pins

def test_selection_hand_example():
    c = _hand()["selection"]
    assert PO.select_candidates(c["state"], c["params"], c["complexity"]) == c["selected"]
    assert PO.select_candidates(c["state"], dict(c["params"], max_fraction=1.0), c["complexity"]) == c["selected_uncapped"]


def test_selection_hand_example_with_every_capability_term():
    c = _hand()["selection_all_terms"]
    assert PO.capability(c["state"], c["params"]) == c["capability"]
    assert PO.select_candidates(c["state"], c["params"], c["complexity"]) == c["selected"]
    assert PO.select_candidates(c["state"], dict(c["params"], max_fraction=1.0), c["complexity"]) == c["selected_uncapped"]


def test_schedule_hand_example():
    c = _hand()["schedule"]
    loc, order, obj, le, lc = PO.schedule_tasks(c["params"], c["complexity"], c["comm"])
    assert loc == c["location"] and order == c["order"]
    assert obj == c["objective"] and le == c["load_end"] and lc == c["load_cloud"]


def _random_selection(rng, M):
    state = {k: float(rng.uniform(0, 4)) for k in ("cpu", "mem", "power", "bandwidth")}
    params = {k: float(rng.uniform(0, 2)) for k in ("w_cpu", "w_mem", "w_power", "w_bandwidth")}
    params.update(epsilon=float(rng.uniform(0.2, 2.0)), max_fraction=float(rng.choice([0.25, 0.4, 1.0])))
    complexity = [float(v) for v in rng.gamma(2.0, 2.0, M)]
    return state, params, complexity


@pytest.mark.parametrize("seed", range(20))
def test_selection_invariants(seed):
    rng = np.random.default_rng(seed)
    M = int(rng.choice([8, 16, 33, 64, 256]))
    state, params, v = _random_selection(rng, M)
    T = PO.capability(state, params)
    sel = PO.select_candidates(state, params, v)
    uncapped = PO.select_candidates(state, dict(params, max_fraction=1.0), v)
    assert uncapped == [i for i in range(M) if v[i] <= params["epsilon"] * T or v[i] / T <= params["epsilon"]]
    assert len(sel) <= math.floor(params["max_fraction"] * M) and set(sel) <= set(uncapped)
    if len(uncapped) > len(sel):  # the cap keeps the least complex experts
        assert max(v[i] for i in sel) <= min(v[i] for i in set(uncapped) - set(sel)) if sel else True
    # a more capable device never loses an expert (no cap)
    richer = {k: 2 * x for k, x in state.items()}
    assert set(uncapped) <= set(PO.select_candidates(richer, dict(params, max_fraction=1.0), v))


@pytest.mark.parametrize("seed", range(20))
def test_schedule_invariants(seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(1, 300))
    C = [float(x) for x in rng.gamma(2.0, 1.0, n)]
    comm = [float(x) for x in rng.gamma(1.5, 1.0, n)]
    p = dict(alpha=float(rng.uniform(0, 1)), beta=float(rng.uniform(0, 3)), epsilon=1e-3,
             t_end=float(rng.uniform(5, 100)), load_end=float(rng.uniform(0, 4)), load_cloud=0.0,
             speed_end=1.0, speed_cloud=float(rng.uniform(1, 8)))
    loc, order, obj, le, lc = PO.schedule_tasks(p, C, comm)
    prio = [C[i] / (comm[i] + p["epsilon"]) for i in range(n)]
    assert sorted(order) == list(range(n))
    assert all(prio[a] >= prio[b] for a, b in zip(order, order[1:]))
    assert all(prio[i] >= p["beta"] for i in range(n) if loc[i] == 0)
    assert le <= max(p["t_end"], p["load_end"]) + 1e-9
    assert math.isclose(le - p["load_end"] + lc - p["load_cloud"], sum(C), rel_tol=1e-12)
    # beta above every priority: everything in the cloud, objective = alpha C/s_cloud + (1-alpha) Comm
    loc2, _, obj2, _, _ = PO.schedule_tasks(dict(p, beta=max(prio) + 1), C, comm)
    assert all(x == 1 for x in loc2)
    assert math.isclose(obj2, sum(p["alpha"] * C[i] / p["speed_cloud"] + (1 - p["alpha"]) * comm[i]
                                  for i in range(n)), rel_tol=1e-12)


# ----------------------------------------------------------------------------- library vs oracle

def test_library_matches_hand_examples():
    c = _hand()
    for key in ("selection", "selection_all_terms"):
        s = c[key]
        words, n = E.select_candidates(_state(s["state"]), _sel(s["params"]), s["complexity"])
        assert W.mask_members(words, len(s["complexity"])) == s["selected"] and n == len(s["selected"])
    t = c["schedule"]
    loc, order, (obj, le, lc) = E.schedule_tasks(_sched(t["params"]), t["complexity"], t["comm"])
    assert loc.tolist() == t["location"] and order.tolist() == t["order"]
    assert (obj, le, lc) == (t["objective"], t["load_end"], t["load_cloud"])


@pytest.mark.parametrize("seed", range(30))
def test_library_selection_matches_oracle(seed):
    rng = np.random.default_rng(1000 + seed)
    M = int(rng.integers(1, 257))
    state, params, v = _random_selection(rng, M)
    if seed % 5 == 0:  # exact ties of f at the cap
        v = [float(rng.choice([1.0, 2.0, 3.0])) for _ in range(M)]
    words, n = E.select_candidates(E.DeviceState(**state), E.SelectionParams(**params), v)
    ref = PO.select_candidates(state, params, v)
    assert W.mask_members(words, M) == ref and n == len(ref)
    assert len(words) == (M + 63) // 64


@pytest.mark.parametrize("seed", range(30))
def test_library_schedule_matches_oracle(seed):
    rng = np.random.default_rng(2000 + seed)
    n = int(rng.integers(0, 2000))
    C = [float(x) for x in rng.gamma(2.0, 1.0, n)]
    comm = [float(x) for x in rng.gamma(1.5, 1.0, n)]
    if seed % 4 == 0:  # many equal priorities
        C = [float(rng.integers(1, 4)) for _ in range(n)]
        comm = [float(rng.integers(0, 3)) for _ in range(n)]
    p = dict(alpha=float(rng.uniform(0, 1)), beta=float(rng.uniform(0, 3)), epsilon=0.5,
             t_end=float(rng.uniform(5, 500)), load_end=float(rng.uniform(0, 4)), load_cloud=1.0,
             speed_end=1.0, speed_cloud=float(rng.uniform(1, 8)))
    loc, order, (obj, le, lc) = E.schedule_tasks(E.ScheduleParams(**p), C, comm)
    rloc, rorder, robj, rle, rlc = PO.schedule_tasks(p, C, comm)
    assert loc.tolist() == rloc and order.tolist() == rorder
    assert (obj, le, lc) == (robj, rle, rlc)  # the same double operations in the same order


def test_library_rejects_bad_inputs():
    s = _hand()["selection"]
    with pytest.raises(E.Ec2moeError):
        E.select_candidates(_state(s["state"]), _sel(dict(s["params"], max_fraction=1.5)), s["complexity"])
    with pytest.raises(E.Ec2moeError):
        E.select_candidates(_state(s["state"]), _sel(s["params"]), [1.0, -1.0])
    with pytest.raises(E.Ec2moeError):
        E.select_candidates(_state(s["state"]), _sel(s["params"]), [1.0] * 257)
    t = _hand()["schedule"]
    with pytest.raises(E.Ec2moeError):
        E.schedule_tasks(_sched(dict(t["params"], epsilon=0.0)), t["complexity"], t["comm"])
    with pytest.raises(E.Ec2moeError):
        E.schedule_tasks(_sched(t["params"]), [1.0, float("nan")], [0.0, 0.0])
    loc, order, summary = E.schedule_tasks(_sched(t["params"]), [], [])
    assert loc.size == 0 and summary[1] == t["params"]["load_end"]


def test_zero_capability_selects_nothing_and_feeds_the_gate_format():
    words, n = E.select_candidates(E.DeviceState(0, 0, 0, 0), E.SelectionParams(1, 1, 1, 1, 1.0, 0.4), [0.0] * 70)
    assert n == 0 and words == [0, 0]
    # the selection is a candidate mask of the gate: Parameter Selection's workloads
    rng = np.random.default_rng(7)
    for M in (8, 16, 32, 64):
        v = [float(x) for x in rng.gamma(2.0, 2.0, M)]
        words, n = E.select_candidates(E.DeviceState(4, 4, 4, 4), E.SelectionParams(1, 1, 1, 1, 1.0, 0.4), v)
        assert n <= int(0.4 * M) and len(W.mask_members(words, M)) == n
