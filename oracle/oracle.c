/*
 * Plan-scoring oracle: a plain, slow, single-threaded fp64 CPU reference for
 * scoring workflow physical plans and selecting one plan per pressure level.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or call
 * this file; only the test suite, the smoke check and the benchmark's CPU
 * baseline leg use it.  It shares no code with the GPU library.
 *
 * What it computes (for a plan pi that gives node n implementation i_n):
 *
 *  corr(pi)   = prod_n (1 - w_n (1 - p_{n,i_n}))                      [1]
 *               The vulnerability-weighted correctness.  The paper weights a
 *               node's residual error r = 1 - q by its vulnerability v
 *               (Sec. 4.3, f = v * r); here each node keeps the workflow
 *               correct unless it errs AND the error is impactful, which gives
 *               the product of (1 - v r) over nodes.
 *  CP_k(pi)   = longest path of the DAG where node n lasts
 *               tau_{n,i_n} / (1 - rho_{k, b(n,i_n)})                 [2]
 *               Serial dependencies add and a join waits for its latest
 *               predecessor (Sec. 4.3 "Accounting for parallel branches");
 *               for fixed assignments the ILP's completion time equals this
 *               longest path (eq. admission-constraints).  The pressure factor
 *               1/(1 - rho) is the backend latency multiplier of the workload
 *               recipes.
 *  demand(pi) = sum_n tau_{n,i_n} * size_{n,i_n}                      [3]
 *               The nominal-duration demand annotation (Sec. 4.4, D_tau,
 *               weighted by model size).
 *  select_k   = argmax corr over plans with CP_k <= SLO, ties to the lowest
 *               plan index; none if no plan is feasible.              [4]
 *               One pressure-specialised variant per level (Sec. 4.4,
 *               Algorithm gen: one solve per level).
 *
 * Arithmetic is IEEE fp64 on the fp32 inputs widened exactly, in this fixed
 * order and with no fused multiply-add (build with -ffp-contract=off):
 *   corr:   c = 1; for n = 0..N-1: t = 1 - p; t = w * t; c = c * (1 - t)
 *   CP_k:   for n = 0..N-1: lat = tau / (1 - rho); f_n = lat + max_{u in pred(n)} f_u
 *           (0 if no predecessor); CP = max over sinks of f_n
 *   demand: d = 0; for n = 0..N-1: d = d + tau * size
 * Plan index: mixed radix, node 0 most significant.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_MAX_NODES 64

typedef struct {
    int32_t n_nodes;
    int32_t n_edges;
    const int32_t* edges;     /* [n_edges][2], u < v */
    const int32_t* radix;     /* [n_nodes] */
    int32_t max_radix;        /* row stride of the tables */
    const float* p;           /* [n_nodes][max_radix] */
    const float* tau;         /* [n_nodes][max_radix] */
    const float* size;        /* [n_nodes][max_radix] */
    const int32_t* backend;   /* [n_nodes][max_radix] */
    const float* w;           /* [n_nodes] */
    int32_t n_levels;
    int32_t n_backends;
    const float* rho;         /* [n_levels][n_backends] */
    float slo;
} or_problem;

typedef struct {
    int64_t index;            /* -1 when no plan is feasible */
    int32_t feasible;
    double corr, cp, demand;  /* NaN when no plan is feasible */
} or_choice;

/* Predecessor lists, rebuilt by each entry point (plain O(N*E) scan). */
typedef struct {
    int32_t count[OR_MAX_NODES];
    int32_t list[OR_MAX_NODES][OR_MAX_NODES];
    int32_t is_sink[OR_MAX_NODES];
} or_graph;

static int or_build_graph(const or_problem* pb, or_graph* g) {
    int N = pb->n_nodes;
    if (N < 1 || N > OR_MAX_NODES) return -1;
    for (int n = 0; n < N; ++n) {
        g->count[n] = 0;
        g->is_sink[n] = 1;
    }
    for (int e = 0; e < pb->n_edges; ++e) {
        int u = pb->edges[2 * e], v = pb->edges[2 * e + 1];
        if (u < 0 || v >= N || u >= v) return -2;
        g->list[v][g->count[v]++] = u;
        g->is_sink[u] = 0;
    }
    return 0;
}

/* Plan index -> implementation per node (node N-1 is the least significant digit). */
void or_decode(const or_problem* pb, uint64_t index, int32_t* impl) {
    for (int n = pb->n_nodes - 1; n >= 0; --n) {
        uint64_t r = (uint64_t)pb->radix[n];
        impl[n] = (int32_t)(index % r);
        index /= r;
    }
}

/* [1] vulnerability-weighted correctness */
double or_corr(const or_problem* pb, const int32_t* impl) {
    double c = 1.0;
    for (int n = 0; n < pb->n_nodes; ++n) {
        double p = (double)pb->p[n * pb->max_radix + impl[n]];
        double w = (double)pb->w[n];
        double t = 1.0 - p;
        t = w * t;
        c = c * (1.0 - t);
    }
    return c;
}

/* [2] critical path at level k; level < 0 means no pressure (every rho = 0) */
static double or_cp_g(const or_problem* pb, const or_graph* g, const int32_t* impl, int level) {
    double f[OR_MAX_NODES];
    double cp = 0.0;
    for (int n = 0; n < pb->n_nodes; ++n) {
        int i = impl[n];
        double tau = (double)pb->tau[n * pb->max_radix + i];
        double rho = 0.0;
        if (level >= 0) rho = (double)pb->rho[level * pb->n_backends + pb->backend[n * pb->max_radix + i]];
        double lat = tau / (1.0 - rho);
        double m = 0.0;
        for (int j = 0; j < g->count[n]; ++j) {
            double fu = f[g->list[n][j]];
            if (fu > m) m = fu;
        }
        f[n] = lat + m;
    }
    int first = 1;
    for (int n = 0; n < pb->n_nodes; ++n) {
        if (!g->is_sink[n]) continue;
        if (first || f[n] > cp) cp = f[n];
        first = 0;
    }
    return cp;
}

double or_cp(const or_problem* pb, const int32_t* impl, int32_t level) {
    or_graph g;
    if (or_build_graph(pb, &g) != 0) return NAN;
    return or_cp_g(pb, &g, impl, level);
}

/* [3] nominal demand */
double or_demand(const or_problem* pb, const int32_t* impl) {
    double d = 0.0;
    for (int n = 0; n < pb->n_nodes; ++n) {
        int k = n * pb->max_radix + impl[n];
        d = d + (double)pb->tau[k] * (double)pb->size[k];
    }
    return d;
}

/* ---- selection [4] --------------------------------------------------------- */

typedef struct {
    const or_problem* pb;
    or_graph g;
    or_choice* out;
    int32_t* impl;
} or_sel;

static void or_sel_init(or_sel* s, const or_problem* pb, or_choice* out, int32_t* impl) {
    s->pb = pb;
    s->out = out;
    s->impl = impl;
    for (int k = 0; k < pb->n_levels; ++k) {
        out[k].index = -1;
        out[k].feasible = 0;
        out[k].corr = NAN;
        out[k].cp = NAN;
        out[k].demand = NAN;
    }
}

/* Offer one plan; plans must be offered in increasing index order so that a
 * strictly greater correctness is needed to replace the current best. */
static void or_sel_offer(or_sel* s, int64_t index) {
    const or_problem* pb = s->pb;
    double slo = (double)pb->slo;
    double corr = or_corr(pb, s->impl);
    double demand = -1.0;
    for (int k = 0; k < pb->n_levels; ++k) {
        double cp = or_cp_g(pb, &s->g, s->impl, k);
        if (!(cp <= slo)) continue;
        or_choice* b = &s->out[k];
        if (b->index < 0 || corr > b->corr) {
            if (demand < 0.0) demand = or_demand(pb, s->impl);
            b->index = index;
            b->feasible = 1;
            b->corr = corr;
            b->cp = cp;
            b->demand = demand;
        }
    }
}

/* Select over plan indices [begin, begin + count). */
int32_t or_select_range(const or_problem* pb, uint64_t begin, uint64_t count, or_choice* out) {
    int32_t impl[OR_MAX_NODES];
    or_sel s;
    or_sel_init(&s, pb, out, impl);
    if (or_build_graph(pb, &s.g) != 0) return -1;
    for (uint64_t j = 0; j < count; ++j) {
        or_decode(pb, begin + j, impl);
        or_sel_offer(&s, (int64_t)(begin + j));
    }
    return 0;
}

/* Select over rows: row r holds the implementation id of node n in byte
 * rows[r * stride + n]; its plan index is index_base + r. */
int32_t or_select_rows(const or_problem* pb, const uint8_t* rows, uint64_t count, uint64_t stride,
                       uint64_t index_base, or_choice* out) {
    int32_t impl[OR_MAX_NODES];
    or_sel s;
    or_sel_init(&s, pb, out, impl);
    if (or_build_graph(pb, &s.g) != 0) return -1;
    for (uint64_t r = 0; r < count; ++r) {
        for (int n = 0; n < pb->n_nodes; ++n) impl[n] = rows[r * stride + (uint64_t)n];
        or_sel_offer(&s, (int64_t)(index_base + r));
    }
    return 0;
}

/* ---- per-plan scores --------------------------------------------------------
 * corr[j], cp[j * K + k], demand[j], feas[j] (bit k set when CP_k <= SLO). */
static void or_score_one(const or_problem* pb, const or_graph* g, const int32_t* impl, uint64_t j,
                         double* corr, double* cp, double* demand, uint32_t* feas) {
    int K = pb->n_levels;
    uint32_t bits = 0;
    corr[j] = or_corr(pb, impl);
    demand[j] = or_demand(pb, impl);
    for (int k = 0; k < K; ++k) {
        double c = or_cp_g(pb, g, impl, k);
        cp[j * (uint64_t)K + (uint64_t)k] = c;
        if (c <= (double)pb->slo && k < 32) bits |= 1u << k;
    }
    feas[j] = bits;
}

int32_t or_score_range(const or_problem* pb, uint64_t begin, uint64_t count, double* corr, double* cp,
                       double* demand, uint32_t* feas) {
    int32_t impl[OR_MAX_NODES];
    or_graph g;
    if (or_build_graph(pb, &g) != 0) return -1;
    for (uint64_t j = 0; j < count; ++j) {
        or_decode(pb, begin + j, impl);
        or_score_one(pb, &g, impl, j, corr, cp, demand, feas);
    }
    return 0;
}

int32_t or_score_rows(const or_problem* pb, const uint8_t* rows, uint64_t count, uint64_t stride,
                      double* corr, double* cp, double* demand, uint32_t* feas) {
    int32_t impl[OR_MAX_NODES];
    or_graph g;
    if (or_build_graph(pb, &g) != 0) return -1;
    for (uint64_t j = 0; j < count; ++j) {
        for (int n = 0; n < pb->n_nodes; ++n) impl[n] = rows[j * stride + (uint64_t)n];
        or_score_one(pb, &g, impl, j, corr, cp, demand, feas);
    }
    return 0;
}

/* Score an explicit list of plan indices (for sampled checks at full size). */
int32_t or_score_indices(const or_problem* pb, const uint64_t* index, uint64_t count, double* corr,
                         double* cp, double* demand, uint32_t* feas) {
    int32_t impl[OR_MAX_NODES];
    or_graph g;
    if (or_build_graph(pb, &g) != 0) return -1;
    for (uint64_t j = 0; j < count; ++j) {
        or_decode(pb, index[j], impl);
        or_score_one(pb, &g, impl, j, corr, cp, demand, feas);
    }
    return 0;
}

/* ---- the workload SLO: 1.5 x the lower median of the unpressured CP --------
 * The exact lower median (0-based rank floor((n-1)/2)) is found in two passes:
 * a histogram of the top `bits` bits of the fp64 pattern (CP >= 0, so the
 * pattern orders like the value), then the values inside the chosen bucket. */

static double or_cp0(const or_problem* pb, const or_graph* g, const int32_t* impl) {
    return or_cp_g(pb, g, impl, -1);
}

static uint64_t or_bits(double x) {
    uint64_t b;
    memcpy(&b, &x, sizeof b);
    return b;
}

/* kind 0: plan indices [begin, begin+count); kind 1: rows */
static int or_cp0_at(const or_problem* pb, const or_graph* g, int kind, const uint8_t* rows, uint64_t stride,
                     uint64_t begin, uint64_t j, int32_t* impl, double* out) {
    if (kind == 0) {
        or_decode(pb, begin + j, impl);
    } else {
        for (int n = 0; n < pb->n_nodes; ++n) impl[n] = rows[j * stride + (uint64_t)n];
    }
    *out = or_cp0(pb, g, impl);
    return 0;
}

int32_t or_cp0_hist(const or_problem* pb, int32_t kind, const uint8_t* rows, uint64_t stride, uint64_t begin,
                    uint64_t count, int32_t bits, uint64_t* hist) {
    int32_t impl[OR_MAX_NODES];
    or_graph g;
    if (or_build_graph(pb, &g) != 0 || bits < 1 || bits > 30) return -1;
    for (uint64_t j = 0; j < count; ++j) {
        double v;
        or_cp0_at(pb, &g, kind, rows, stride, begin, j, impl, &v);
        hist[or_bits(v) >> (64 - bits)] += 1;
    }
    return 0;
}

/* Collect CP values whose top `bits` bits equal `bucket`; returns how many
 * there were (only the first `cap` are stored). */
int64_t or_cp0_collect(const or_problem* pb, int32_t kind, const uint8_t* rows, uint64_t stride,
                       uint64_t begin, uint64_t count, int32_t bits, uint64_t bucket, double* out, uint64_t cap) {
    int32_t impl[OR_MAX_NODES];
    or_graph g;
    if (or_build_graph(pb, &g) != 0 || bits < 1 || bits > 30) return -1;
    uint64_t got = 0;
    for (uint64_t j = 0; j < count; ++j) {
        double v;
        or_cp0_at(pb, &g, kind, rows, stride, begin, j, impl, &v);
        if ((or_bits(v) >> (64 - bits)) == bucket) {
            if (got < cap) out[got] = v;
            ++got;
        }
    }
    return (int64_t)got;
}

/* CP at no pressure for every plan in a range (small cases). */
int32_t or_cp0_range(const or_problem* pb, int32_t kind, const uint8_t* rows, uint64_t stride, uint64_t begin,
                     uint64_t count, double* out) {
    int32_t impl[OR_MAX_NODES];
    or_graph g;
    if (or_build_graph(pb, &g) != 0) return -1;
    for (uint64_t j = 0; j < count; ++j) or_cp0_at(pb, &g, kind, rows, stride, begin, j, impl, &out[j]);
    return 0;
}
