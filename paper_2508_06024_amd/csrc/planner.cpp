// Host planner of the end side: hardware-aware local expert selection (Local Expert
// Selection, Eq. 2-4) producing the candidate mask the gate consumes, and the greedy
// route-aware pipeline scheduler (Route-Aware Heuristic Pipeline Scheduling, Eq. 9-11).
// Plain host code: no GPU work. Contracts in include/ec2moe.h.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <numeric>
#include <vector>

#include "internal.h"

namespace ec2moe {
namespace {

ec2moe_status invalid(const char* what) { return report_error(EC2MOE_ERR_INVALID_ARGUMENT, what); }

bool finite_nonneg(double v) { return std::isfinite(v) && v >= 0.0; }

}  // namespace
}  // namespace ec2moe

using namespace ec2moe;

extern "C" {

ec2moe_status ec2moe_select_candidates(const ec2moe_device_state* state, const ec2moe_selection_params* params,
                                       const double* complexity, int32_t n_experts, uint64_t* mask_out,
                                       int32_t* n_selected) {
    if (!state || !params || !complexity || !mask_out || !n_selected) return invalid("NULL argument");
    if (n_experts < 1 || n_experts > 256) return invalid("n_experts must be in [1, 256]");
    const double s[4] = {state->cpu, state->mem, state->power, state->bandwidth};
    const double wt[4] = {params->w_cpu, params->w_mem, params->w_power, params->w_bandwidth};
    for (int i = 0; i < 4; ++i)
        if (!finite_nonneg(s[i]) || !finite_nonneg(wt[i])) return invalid("device state and H weights must be finite and >= 0");
    if (!finite_nonneg(params->epsilon)) return invalid("epsilon must be finite and >= 0");
    if (!(params->max_fraction >= 0.0 && params->max_fraction <= 1.0)) return invalid("max_fraction must be in [0, 1]");
    for (int i = 0; i < n_experts; ++i)
        if (!finite_nonneg(complexity[i])) return invalid("expert complexities must be finite and >= 0");

    // Eq. 3: T_capability = H(S_device), a weighted sum in the order cpu, mem, power, bandwidth
    const double cap = wt[0] * s[0] + wt[1] * s[1] + wt[2] * s[2] + wt[3] * s[3];
    const int words = (n_experts + 63) / 64;
    std::fill(mask_out, mask_out + words, uint64_t(0));
    *n_selected = 0;
    if (!(cap > 0.0)) return report_error(EC2MOE_OK, "");
    // Eq. 4: f(V_i, T) = V_i / T <= epsilon
    std::vector<std::pair<double, int>> ok;
    for (int i = 0; i < n_experts; ++i) {
        const double f = complexity[i] / cap;
        if (f <= params->epsilon) ok.emplace_back(f, i);
    }
    // the candidate cap: the floor(max_fraction * M) experts of smallest f, ties to the lower index
    const size_t limit = static_cast<size_t>(std::floor(params->max_fraction * n_experts));
    if (ok.size() > limit) {
        std::stable_sort(ok.begin(), ok.end(), [](const auto& a, const auto& b) { return a.first < b.first; });
        ok.resize(limit);
    }
    for (const auto& e : ok) mask_out[e.second >> 6] |= uint64_t(1) << (e.second & 63);
    *n_selected = static_cast<int32_t>(ok.size());
    return report_error(EC2MOE_OK, "");
}

ec2moe_status ec2moe_schedule_tasks(const ec2moe_schedule_params* params, const double* complexity,
                                    const double* comm, int32_t n_tasks, int32_t* location, int32_t* order,
                                    double* summary) {
    if (!params) return invalid("params is NULL");
    if (n_tasks < 0) return invalid("n_tasks < 0");
    if (n_tasks > 0 && (!complexity || !comm || !location)) return invalid("NULL argument");
    const ec2moe_schedule_params& p = *params;
    if (!(p.alpha >= 0.0 && p.alpha <= 1.0)) return invalid("alpha must be in [0, 1]");
    if (!std::isfinite(p.beta)) return invalid("beta must be finite");
    if (!(std::isfinite(p.epsilon) && p.epsilon > 0.0)) return invalid("epsilon must be finite and > 0");
    if (!std::isfinite(p.t_end) || !finite_nonneg(p.load_end) || !finite_nonneg(p.load_cloud))
        return invalid("t_end and the initial loads must be finite (loads >= 0)");
    if (!(std::isfinite(p.speed_end) && p.speed_end > 0.0 && std::isfinite(p.speed_cloud) && p.speed_cloud > 0.0))
        return invalid("speeds must be finite and > 0");
    for (int i = 0; i < n_tasks; ++i)
        if (!finite_nonneg(complexity[i]) || !finite_nonneg(comm[i]))
            return invalid("task complexities and communication costs must be finite and >= 0");

    // Eq. 10: priorities; tasks taken in descending priority, equal priorities in index order
    std::vector<double> prio(n_tasks);
    for (int i = 0; i < n_tasks; ++i) prio[i] = complexity[i] / (comm[i] + p.epsilon);
    std::vector<int32_t> ord(n_tasks);
    std::iota(ord.begin(), ord.end(), 0);
    std::stable_sort(ord.begin(), ord.end(), [&](int32_t a, int32_t b) { return prio[a] > prio[b]; });
    // Eq. 11: greedy placement against the end device's threshold
    double load_end = p.load_end, load_cloud = p.load_cloud;
    for (int32_t i : ord) {
        if (load_end + complexity[i] <= p.t_end && prio[i] >= p.beta) {
            location[i] = 0;
            load_end += complexity[i];
        } else {
            location[i] = 1;
            load_cloud += complexity[i];
        }
    }
    // Eq. 9: the weighted cost of the placement, summed in task order
    double objective = 0.0;
    for (int i = 0; i < n_tasks; ++i) {
        const bool end = location[i] == 0;
        const double exec = complexity[i] / (end ? p.speed_end : p.speed_cloud);
        objective += p.alpha * exec + (1.0 - p.alpha) * (end ? 0.0 : comm[i]);
    }
    if (order) std::copy(ord.begin(), ord.end(), order);
    if (summary) {
        summary[0] = objective;
        summary[1] = load_end;
        summary[2] = load_cloud;
    }
    return report_error(EC2MOE_OK, "");
}

}  // extern "C"
