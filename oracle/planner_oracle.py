"""CPU oracle of the end-side planner: hardware-aware local expert selection (Local
Expert Selection, Eq. 2-4) and the route-aware greedy pipeline scheduler (Route-Aware
Heuristic Pipeline Scheduling, Eq. 9-11).

TEST INFRASTRUCTURE, NOT PRODUCT CODE: only the test suite may import it. It shares no
code with the library. The paper leaves H, f and the thresholds open; the readings are:
  * H (Eq. 3): T_capability = w_cpu cpu + w_mem mem + w_power power + w_bandwidth bandwidth;
  * f (Eq. 4): f(V_i, T) = V_i / T; T <= 0 selects nothing;
  * the candidate cap (Parameter Selection: at most 40% of the experts): keep the
    floor(max_fraction M) qualifying experts of smallest f, ties to the lower index;
  * the greedy order of Eq. 11: descending priority P = C / (Comm + eps) of Eq. 10, ties
    to the lower index; a task placed on the end device adds C to Load_end, one placed
    in the cloud adds C to Load_cloud;
  * Eq. 9: ExecTime = C / speed of the chosen side; Comm is paid by cloud tasks only.
"""
from __future__ import annotations

import math


def capability(state, params):
    """Eq. 3 with the linear H."""
    return (params["w_cpu"] * state["cpu"] + params["w_mem"] * state["mem"]
            + params["w_power"] * state["power"] + params["w_bandwidth"] * state["bandwidth"])


def select_candidates(state, params, complexity):
    """Eq. 4 and the cap: the sorted list of selected expert indices."""
    cap = capability(state, params)
    if not cap > 0:
        return []
    ok = [i for i, v in enumerate(complexity) if v / cap <= params["epsilon"]]
    limit = math.floor(params["max_fraction"] * len(complexity))
    if len(ok) > limit:
        ok = sorted(ok, key=lambda i: (complexity[i] / cap, i))[:limit]
    return sorted(ok)


def schedule_tasks(params, complexity, comm):
    """Eq. 9-11: (location per task: 0 end / 1 cloud, processing order, objective,
    final Load_end, final Load_cloud)."""
    n = len(complexity)
    prio = [complexity[i] / (comm[i] + params["epsilon"]) for i in range(n)]
    order = sorted(range(n), key=lambda i: (-prio[i], i))
    load_end, load_cloud = params["load_end"], params["load_cloud"]
    loc = [None] * n
    for i in order:
        if load_end + complexity[i] <= params["t_end"] and prio[i] >= params["beta"]:
            loc[i] = 0
            load_end += complexity[i]
        else:
            loc[i] = 1
            load_cloud += complexity[i]
    objective = 0.0
    for i in range(n):
        end = loc[i] == 0
        exec_time = complexity[i] / (params["speed_end"] if end else params["speed_cloud"])
        objective += params["alpha"] * exec_time + (1.0 - params["alpha"]) * (0.0 if end else comm[i])
    return loc, order, objective, load_end, load_cloud
