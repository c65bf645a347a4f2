/*
 * Oracle for the paper's additive plan objective (Sec. 4.3-4.4): a plain,
 * slow, single-threaded fp64 CPU reference.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or call
 * this file; only the test suite, the smoke check and the benchmark's CPU
 * baseline leg use it.  It shares no code with the GPU library.
 *
 * For a plan pi that gives node n implementation i_n (Sec. 4.3, eq.
 * admission-objective and eq. admission-constraints; Sec. 4.4, eq.
 * variant-objective):
 *
 *  reach(n) = 1 + beta * e * (|R(n)| - 1) / (|V| - 1), R(n) = n and every node
 *             reachable from it; reach = 1 for a one-node workflow.      [R]
 *  u_{n,i}  = reach(n) q_{n,i} - lambda_f v_n (1 - q_{n,i}) - lambda_c c_{n,i}
 *             for an LLM node (the impact-weighted error f = v r, r = 1 - q);
 *             tool nodes contribute no quality or cost term.          [U]
 *  T(pi)    = longest path of the DAG with node n lasting its nominal duration
 *             tau_{n,i_n} (tool nodes included): the ILP's completion time
 *             for fixed assignments.                                   [T]
 *  D(pi)    = sum over LLM nodes of tau_{n,i_n} (D_tau).               [D]
 *  J_k(pi)  = sum_{LLM n} u_{n,i_n} - lambda_l T(pi) - lambda_ld L_k D(pi)
 *                                                                      [J]
 *  select_k = argmax_pi J_k, ties to the lowest plan index.            [S]
 *
 * Arithmetic: IEEE fp64 on the fp32 inputs widened exactly, no fused
 * multiply-add, in this order:
 *   reach: t = beta * e; t = t * (|R|-1); t = t / (|V|-1); reach = 1 + t
 *   u:     a = reach * q; b = 1 - q; b = v * b; b = lambda_f * b; a = a - b;
 *          b = lambda_c * c; a = a - b
 *   U = 0; for n in node order, LLM nodes: U = U + u
 *   T:     f_n = tau + max_{pred} f_u (0 with no predecessor); T = max over sinks
 *   D = 0; for n in node order, LLM nodes: D = D + tau
 *   J:     j = lambda_l * T; j = U - j; m = lambda_ld * L_k; m = m * D; j = j - m
 * Plan index: mixed radix, node 0 most significant.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OP_MAX_NODES 64
#define OP_MAX_LEVELS 64

typedef struct {
    int32_t n_nodes;
    int32_t n_edges;
    const int32_t* edges;     /* [n_edges][2], u < v */
    const int32_t* radix;     /* [n_nodes] */
    int32_t max_radix;        /* row stride of the tables */
    const float* q;           /* [n_nodes][max_radix] local quality */
    const float* tau;         /* [n_nodes][max_radix] nominal duration */
    const float* cost;        /* [n_nodes][max_radix] call cost */
    const float* v;           /* [n_nodes] vulnerability */
    const int32_t* is_tool;   /* [n_nodes] or NULL (every node an LLM node) */
    float lambda_f, lambda_c, lambda_l, lambda_ld, beta, effort;
    int32_t n_levels;
    const float* levels;      /* [n_levels] L_k */
} op_problem;

typedef struct {
    int64_t index;            /* the argmax plan */
    int32_t feasible;         /* 1 (the objective has no hard constraint) */
    double j, t, d;           /* its J_k, T and D */
} op_choice;

typedef struct {
    int32_t n;
    int32_t npred[OP_MAX_NODES];
    int32_t pred[OP_MAX_NODES][OP_MAX_NODES];
    int32_t sink[OP_MAX_NODES];
    double reach[OP_MAX_NODES];
} op_graph;

/* Predecessor lists, sinks and reach weights, by plain scans of the edge list. */
static int op_build(const op_problem* pb, op_graph* g) {
    const int N = pb->n_nodes;
    if (N < 1 || N > OP_MAX_NODES || pb->n_levels < 1 || pb->n_levels > OP_MAX_LEVELS) return -1;
    g->n = N;
    int32_t adj[OP_MAX_NODES][OP_MAX_NODES];
    memset(adj, 0, sizeof adj);
    for (int n = 0; n < N; ++n) {
        g->npred[n] = 0;
        g->sink[n] = 1;
    }
    for (int e = 0; e < pb->n_edges; ++e) {
        int u = pb->edges[2 * e], w = pb->edges[2 * e + 1];
        if (u < 0 || w >= N || u >= w) return -1;
        if (adj[u][w]) continue; /* a repeated edge is one edge */
        adj[u][w] = 1;
        g->pred[w][g->npred[w]++] = u;
        g->sink[u] = 0;
    }
    /* [R]: |R(n)| by a depth-first walk from n over the adjacency matrix */
    for (int n = 0; n < N; ++n) {
        int seen[OP_MAX_NODES] = {0}, stack[OP_MAX_NODES], top = 0, size = 0;
        stack[top++] = n;
        seen[n] = 1;
        while (top > 0) {
            int x = stack[--top];
            ++size;
            for (int y = 0; y < N; ++y)
                if (adj[x][y] && !seen[y]) {
                    seen[y] = 1;
                    stack[top++] = y;
                }
        }
        if (N == 1) {
            g->reach[n] = 1.0;
        } else {
            double t = (double)pb->beta * (double)pb->effort;
            t = t * (double)(size - 1);
            t = t / (double)(N - 1);
            g->reach[n] = 1.0 + t;
        }
    }
    return 0;
}

static int op_llm(const op_problem* pb, int n) { return pb->is_tool == NULL || pb->is_tool[n] == 0; }

/* [U] one node's utility */
static double op_u(const op_problem* pb, const op_graph* g, int n, int i) {
    const int k = n * pb->max_radix + i;
    double q = (double)pb->q[k];
    double a = g->reach[n] * q;
    double b = 1.0 - q;
    b = (double)pb->v[n] * b;
    b = (double)pb->lambda_f * b;
    a = a - b;
    b = (double)pb->lambda_c * (double)pb->cost[k];
    a = a - b;
    return a;
}

/* U, T, D of a plan */
static void op_terms(const op_problem* pb, const op_graph* g, const int32_t* impl, double* U, double* T,
                     double* D) {
    double f[OP_MAX_NODES];
    double u = 0.0, d = 0.0, t = 0.0;
    int first = 1;
    for (int n = 0; n < g->n; ++n) {
        const double tau = (double)pb->tau[n * pb->max_radix + impl[n]];
        if (op_llm(pb, n)) {
            u = u + op_u(pb, g, n, impl[n]);
            d = d + tau;
        }
        double m = 0.0;
        for (int j = 0; j < g->npred[n]; ++j)
            if (f[g->pred[n][j]] > m) m = f[g->pred[n][j]];
        f[n] = tau + m;
        if (g->sink[n] && (first || f[n] > t)) {
            t = f[n];
            first = 0;
        }
    }
    *U = u;
    *T = t;
    *D = d;
}

/* [J] */
static double op_j(const op_problem* pb, int k, double U, double T, double D) {
    double j = (double)pb->lambda_l * T;
    j = U - j;
    double m = (double)pb->lambda_ld * (double)pb->levels[k];
    m = m * D;
    return j - m;
}

static void op_decode(const op_problem* pb, uint64_t index, int32_t* impl) {
    for (int n = pb->n_nodes - 1; n >= 0; --n) {
        const uint64_t r = (uint64_t)pb->radix[n];
        impl[n] = (int32_t)(index % r);
        index /= r;
    }
}

/* reach weights (tests) */
int32_t op_reach(const op_problem* pb, double* out) {
    op_graph g;
    if (op_build(pb, &g) != 0) return -1;
    for (int n = 0; n < pb->n_nodes; ++n) out[n] = g.reach[n];
    return 0;
}

/* per-plan U, T, D and J[k] for plans given by implementation vectors */
int32_t op_eval(const op_problem* pb, const int32_t* impl, double* U, double* T, double* D, double* J) {
    op_graph g;
    if (op_build(pb, &g) != 0) return -1;
    op_terms(pb, &g, impl, U, T, D);
    for (int k = 0; k < pb->n_levels; ++k) J[k] = op_j(pb, k, *U, *T, *D);
    return 0;
}

static void op_offer(const op_problem* pb, const op_graph* g, const int32_t* impl, int64_t index,
                     op_choice* out) {
    double U, T, D;
    op_terms(pb, g, impl, &U, &T, &D);
    for (int k = 0; k < pb->n_levels; ++k) {
        const double j = op_j(pb, k, U, T, D);
        /* plans arrive in increasing index order: only a strictly greater J replaces */
        if (out[k].index < 0 || j > out[k].j) {
            out[k].index = index;
            out[k].feasible = 1;
            out[k].j = j;
            out[k].t = T;
            out[k].d = D;
        }
    }
}

static void op_init(const op_problem* pb, op_choice* out) {
    for (int k = 0; k < pb->n_levels; ++k) {
        out[k].index = -1;
        out[k].feasible = 0;
        out[k].j = out[k].t = out[k].d = NAN;
    }
}

/* [S] over plan indices [begin, begin + count) */
int32_t op_select_range(const op_problem* pb, uint64_t begin, uint64_t count, op_choice* out) {
    op_graph g;
    int32_t impl[OP_MAX_NODES];
    op_init(pb, out);
    if (op_build(pb, &g) != 0) return -1;
    for (uint64_t j = 0; j < count; ++j) {
        op_decode(pb, begin + j, impl);
        op_offer(pb, &g, impl, (int64_t)(begin + j), out);
    }
    return 0;
}

/* [S] over rows (byte n of row r = implementation of node n; index = index_base + r) */
int32_t op_select_rows(const op_problem* pb, const uint8_t* rows, uint64_t count, uint64_t stride,
                       uint64_t index_base, op_choice* out) {
    op_graph g;
    int32_t impl[OP_MAX_NODES];
    op_init(pb, out);
    if (op_build(pb, &g) != 0) return -1;
    for (uint64_t r = 0; r < count; ++r) {
        for (int n = 0; n < pb->n_nodes; ++n) impl[n] = rows[r * stride + (uint64_t)n];
        op_offer(pb, &g, impl, (int64_t)(index_base + r), out);
    }
    return 0;
}

/* per-plan U[j], T[j], D[j], J[j * K + k] over a range (kind 0) or rows (kind 1) */
int32_t op_score(const op_problem* pb, int32_t kind, const uint8_t* rows, uint64_t stride, uint64_t begin,
                 uint64_t count, double* U, double* T, double* D, double* J) {
    op_graph g;
    int32_t impl[OP_MAX_NODES];
    if (op_build(pb, &g) != 0) return -1;
    const int K = pb->n_levels;
    for (uint64_t j = 0; j < count; ++j) {
        if (kind == 0)
            op_decode(pb, begin + j, impl);
        else
            for (int n = 0; n < pb->n_nodes; ++n) impl[n] = rows[j * stride + (uint64_t)n];
        op_terms(pb, &g, impl, &U[j], &T[j], &D[j]);
        for (int k = 0; k < K; ++k) J[j * (uint64_t)K + (uint64_t)k] = op_j(pb, k, U[j], T[j], D[j]);
    }
    return 0;
}
