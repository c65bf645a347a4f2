// Plan-bundle annotations and load-driven variant switching (host only).
//
// Annotations (Sec. 4.4; Algorithm gen attaches per-model demand and an
// estimated quality to every variant; Sec. 5.2 names the model with the
// largest share of the planned demand the variant's dominant model): the
// nominal durations of a plan's LLM-node calls summed per model class, the
// dominant class, and the chance that no node makes an impact-weighted error
// (product of 1 - v (1 - q)).
//
// Switching (Sec. 5.2, "Switching plan variants"): a state machine over load
// samples that scans later variants when the active variant's dominant model
// is overloaded and returns to the lowest-index calm variant when load
// subsides, with a quality tolerance and a dwell time.
#include <cmath>
#include <cstdint>
#include <vector>

#include "dyplan.h"

namespace {

bool is_llm(const dy_problem& p, int n) { return !p.objective || !p.objective->is_tool || p.objective->is_tool[n] == 0; }

}  // namespace

extern "C" {

int dy_bundle_annotate(const dy_problem* prob, const int32_t* model, int32_t n_models, const int32_t* impl,
                       double* model_demand, int32_t* dominant, double* quality) {
    if (!prob || !model || !impl || !model_demand || !dominant || !quality || n_models < 1) return DY_EINVAL;
    const int N = prob->n_nodes, R = prob->max_radix;
    if (N < 1 || N > DY_MAX_NODES || !prob->radix || !prob->p || !prob->tau || !prob->w) return DY_EINVAL;
    for (int n = 0; n < N; ++n) {
        if (impl[n] < 0 || impl[n] >= prob->radix[n] || impl[n] >= R) return DY_EINVAL;
        const int32_t m = model[(size_t)n * R + impl[n]];
        if (is_llm(*prob, n) && (m < 0 || m >= n_models)) return DY_EINVAL;
    }
    for (int m = 0; m < n_models; ++m) model_demand[m] = 0.0;
    double q = 1.0;
    bool llm = false;
    for (int n = 0; n < N; ++n) {
        if (!is_llm(*prob, n)) continue;
        llm = true;
        const size_t e = (size_t)n * R + impl[n];
        model_demand[model[e]] += (double)prob->tau[e];
        // 1 - v (1 - q), operation by operation
        double t = 1.0 - (double)prob->p[e];
        t = (double)prob->w[n] * t;
        q = q * (1.0 - t);
    }
    int32_t dom = -1;
    if (llm) {
        dom = 0;
        for (int m = 1; m < n_models; ++m)
            if (model_demand[m] > model_demand[dom]) dom = m;
    }
    *dominant = dom;
    *quality = q;
    return DY_OK;
}

int dy_switch_simulate(const dy_variant* v, int32_t n_variants, int32_t n_models, const double* times,
                       const double* loads, int32_t n_steps, const dy_switch_rules* r, int32_t* active,
                       int32_t* n_switches) {
    if (!v || !times || !loads || !r || !active || n_variants < 1 || n_models < 1 || n_steps < 0) return DY_EINVAL;
    for (int j = 0; j < n_variants; ++j)
        if (v[j].dominant < -1 || v[j].dominant >= n_models || std::isnan(v[j].quality)) return DY_EINVAL;
    int cur = 0, switches = 0;
    bool switched = false;
    double last = 0.0;
    for (int s = 0; s < n_steps; ++s) {
        const double* L = loads + (size_t)s * n_models;
        auto load = [&](int j) { return v[j].dominant < 0 ? 0.0 : L[v[j].dominant]; };
        auto keeps_quality = [&](int j) { return v[cur].quality - v[j].quality <= r->tolerance; };
        int next = cur;
        if (!(switched && times[s] - last < r->dwell)) {
            const double lc = load(cur);
            if (lc > r->high) {
                // overloaded: first later variant on another, calmer dominant model
                for (int j = cur + 1; j < n_variants; ++j) {
                    const double lj = load(j);
                    if (v[j].dominant != v[cur].dominant && !(lj > r->high) && lj <= lc - r->margin &&
                        keeps_quality(j)) {
                        next = j;
                        break;
                    }
                }
            } else {
                // load subsided: lowest-index variant below the low threshold
                for (int j = 0; j < cur; ++j)
                    if (load(j) < r->low && keeps_quality(j)) {
                        next = j;
                        break;
                    }
            }
        }
        if (next != cur) {
            cur = next;
            last = times[s];
            switched = true;
            ++switches;
        }
        active[s] = cur;
    }
    if (n_switches) *n_switches = switches;
    return DY_OK;
}

}  // extern "C"
