/*
 * dyplan.h -- C ABI of the MI355X (gfx950) workflow physical-plan scorer.
 *
 * A workflow request is a materialised DAG whose nodes each take one
 * implementation: a model on a backend plus a verification policy
 * (Sec. 3.1, eq. physical-plan; tool nodes are nodes with a single
 * implementation).  A physical plan assigns one implementation to every node.
 * This library scores plans and, for every pressure level, selects the best
 * plan that meets the SLO: the pressure-specialised variants of Sec. 4.4 and
 * Algorithm gen (coefficients bound once, then one selection per level).
 *
 * Scoring a plan pi (i_n = implementation of node n):
 *   corr(pi)   = prod_n (1 - w_n * (1 - p_{n,i_n}))
 *                vulnerability-weighted correctness: residual error 1 - q
 *                weighted by the node's vulnerability (Sec. 4.1, Sec. 4.3).
 *   CP_k(pi)   = longest path of the DAG where node n lasts
 *                tau_{n,i_n} / (1 - rho_{k, backend(n,i_n)})
 *                serial dependencies add and a join waits for its latest
 *                predecessor (Sec. 4.3, "Accounting for parallel branches";
 *                for fixed assignments the completion time of
 *                eq. admission-constraints is this longest path).
 *   demand(pi) = sum_n tau_{n,i_n} * size_{n,i_n}
 *                nominal-duration demand annotation (Sec. 4.4, D_tau),
 *                weighted by the model-size factor.
 * Selection at level k: the plan with the greatest corr among plans with
 * CP_k <= slo (inclusive); equal corr goes to the lowest plan index.
 *
 * Objective mode (dy_problem.objective non-NULL): the paper's own additive
 * objective, Sec. 4.3 eq. admission-objective with Sec. 4.4 eq.
 * variant-objective, selected at each specialisation level L_k:
 *   reach(n) = 1 + beta * e * (|R(n)| - 1) / (|V| - 1), R(n) = n and every
 *              node reachable from it (1 for a one-node workflow);
 *   u_{n,i}  = reach(n) p_{n,i} - lambda_f w_n (1 - p_{n,i}) - lambda_c cost_{n,i}
 *              for LLM nodes (tool nodes carry no quality or cost term);
 *   T(pi)    = longest path of nominal durations tau (tool nodes included);
 *   D(pi)    = sum over LLM nodes of tau_{n,i_n} (D_tau);
 *   J_k(pi)  = sum_{LLM n} u_{n,i_n} - lambda_l T(pi) - lambda_ld L_k D(pi),
 * and the choice of level k is the plan with the greatest J_k (equal J to the
 * lowest index); there is no hard constraint, rho and slo are not used.
 *
 * Plan index: mixed radix over the nodes, node 0 most significant:
 *   index = (...((i_0 * radix_1 + i_1) * radix_2 + i_2)...) * radix_{N-1} + i_{N-1}.
 *
 * Numerics.  Plans are scored in fp32 on the GPU.  Selections are certified:
 * every plan whose fp32 score could, within the proven fp32 error bound, be
 * the exact winner is re-evaluated in fp64 with the definition above written
 * out in node order without fused multiply-add, so the selected index and
 * feasibility flag equal those of an fp64 evaluation of every plan, and the
 * reported corr / cp / demand of a winner are its fp64 values rounded to the
 * nearest fp32.  Per-plan scores (dy_plan_score) are fp32 with relative error
 * below 2 * n_nodes * 2^-24 (corr, demand) and (n_nodes + 2) * 2^-24 (cp);
 * their feasibility bits are exact (fp64 decides every plan whose fp32 CP is
 * too close to the SLO to decide).
 *
 * Errors.  Every entry point returns DY_OK (0) or a negative status and never
 * aborts or throws.  dy_plan_last_error(handle) describes the last failure on
 * that handle; dy_plan_last_error(NULL) the last failure of dy_plan_create on
 * the calling thread.  A handle may be used by one thread at a time; distinct
 * handles are independent.
 */
#ifndef DYPLAN_H
#define DYPLAN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DY_ABI_VERSION 4

#define DY_MAX_NODES 32      /* nodes per problem */
#define DY_MAX_RADIX 255     /* implementations per node (ids fit a uint8 row byte) */
#define DY_MAX_LEVELS 32     /* pressure levels per problem */
#define DY_MAX_BACKENDS 64   /* backends per problem */

enum {
    DY_OK = 0,
    DY_EINVAL = -1,   /* bad argument: null pointer, NaN, value out of range, bad row id */
    DY_ENOTDAG = -2,  /* an edge (u, v) is not u < v (the numbering must be topological) */
    DY_ELIMIT = -3,   /* a compile-time limit above is exceeded, or a range is too long */
    DY_ENOMEM = -4,   /* host or device allocation failed */
    DY_EDEVICE = -5   /* a HIP runtime call failed (no device, launch failure, ...) */
};

typedef struct dy_plan dy_plan; /* opaque handle */

/*
 * One planning problem (one materialised workflow request).  All pointers are
 * HOST pointers; dy_plan_create copies what it needs, so the caller may free
 * them as soon as it returns.
 *
 *  n_nodes            N, 1..DY_MAX_NODES.
 *  n_edges, edges     E edges as int32 pairs [E][2] = (u, v), 0 <= u < v < N
 *                     (nodes numbered in a topological order, Sec. 3.1);
 *                     duplicate edges are allowed and mean one edge.
 *  radix              int32 [N], 1..DY_MAX_RADIX implementations per node.
 *  max_radix          row stride of the tables below, >= max(radix).
 *  p                  float [N][max_radix] success probability q of
 *                     implementation (n, i), in [0, 1] (Sec. 4.1).
 *  tau                float [N][max_radix] nominal duration, finite, >= 0
 *                     (Sec. 4.2, eq. tau).
 *  size               float [N][max_radix] model-size factor used by the
 *                     demand annotation, finite, >= 0.
 *  backend            int32 [N][max_radix] backend id, 0..n_backends-1.
 *  w                  float [N] vulnerability v_n in [0, 1] (Sec. 4.3).
 *  n_levels, rho      K levels, float [K][n_backends] pressure of backend b
 *                     at level k, 0 <= rho < 1; a node's duration at level k
 *                     is tau / (1 - rho_{k, backend}).
 *  slo                critical-path bound, >= 0 (may be +inf).
 *  objective          NULL for the corr / SLO selection above, else the
 *                     paper's additive objective (then n_levels, rho, slo,
 *                     size and backend are not read; backend and rho may be
 *                     NULL).
 * Table entries with i >= radix[n] are ignored.  Sum over nodes of the
 * largest tau must stay below 1e30.
 */
/*
 * The paper's additive objective (Sec. 4.3-4.4), all values finite:
 *  cost      float [N][max_radix] call cost c of implementation (n, i).
 *  is_tool   int32 [N], 1 marks a tool node, or NULL (every node an LLM node).
 *  lambda_f, lambda_c   weights of the impact-weighted error and of the cost.
 *  lambda_l  weight of the critical path T, >= 0.
 *  lambda_ld weight of the demand D_tau, >= 0.
 *  beta, effort         reach weight parameters (effort e in [0, 1]).
 *  n_levels, levels     K specialisation levels L_k >= 0, float [K].
 * The sum over LLM nodes of the largest |u|, lambda_l times the sum of the
 * largest durations, and lambda_ld L_k times that sum must each stay <= 1e30.
 */
typedef struct dy_objective {
    const float* cost;
    const int32_t* is_tool;
    float lambda_f, lambda_c, lambda_l, lambda_ld;
    float beta, effort;
    int32_t n_levels;
    const float* levels;
} dy_objective;

typedef struct dy_problem {
    int32_t n_nodes;
    int32_t n_edges;
    const int32_t* edges;
    const int32_t* radix;
    int32_t max_radix;
    const float* p;
    const float* tau;
    const float* size;
    const int32_t* backend;
    const float* w;
    int32_t n_levels;
    int32_t n_backends;
    const float* rho;
    float slo;
    const dy_objective* objective;
} dy_problem;

enum { DY_SOURCE_RANGE = 0, DY_SOURCE_ROWS = 1 };

/*
 * Where the candidate plans of one problem come from.
 *  kind = DY_SOURCE_RANGE: plan indices [begin, begin + count) of the
 *         problem's mixed-radix space (count >= 1, begin + count <= the
 *         number of plans and <= 2^64 - 1).  rows/row_stride/index_base unused.
 *  kind = DY_SOURCE_ROWS: `count` rows in DEVICE memory, row r at
 *         rows + r * row_stride, byte n of a row = implementation id of node n
 *         (must be < radix[n]; a bad id makes the call fail with DY_EINVAL).
 *         row_stride >= n_nodes.  The plan index reported for row r is
 *         index_base + r.  The rows must stay valid until the call's stream
 *         work completes.
 *  problem: index of the problem in the array given to dy_plan_create.
 * A single source may cover at most 2^40 plans.
 */
typedef struct dy_source {
    int32_t kind;
    int32_t problem;
    uint64_t begin;
    uint64_t count;
    const uint8_t* rows;
    uint64_t row_stride;
    uint64_t index_base;
} dy_source;

/* The selected plan of one level.  index = -1 and feasible = 0 when no plan of
 * the source meets the SLO at that level; corr, cp and demand are then NaN.
 * cp is CP at this level.  Objective mode: feasible = 1, corr = J_k of the
 * plan, cp = T, demand = D_tau (fp64 values rounded to the nearest fp32). */
typedef struct dy_choice {
    int64_t index;
    int32_t feasible;
    float corr;
    float cp;
    float demand;
} dy_choice;

/* Statistics of the last dy_plan_select call on a handle. */
typedef struct dy_stats {
    uint64_t plans;          /* plans scored */
    uint64_t candidates;     /* plans re-evaluated in fp64 for certification */
    int32_t fallbacks;       /* (source, level) pairs decided by the exhaustive fp64 path */
    int32_t n_jobs;          /* sources in the call */
    float main_ms;           /* duration of the main scoring kernel(s), when timing is on */
    float total_ms;          /* launch of the first kernel to the end of the last */
    int32_t generated_jobs;  /* sources whose main pass ran a kernel generated for their problem */
    int32_t ydiv_jobs;       /* sources whose sweep took its bin thresholds divided (corr) or lowered
                                (objective) ahead by each implementation of node y: per plan one add (CP, or
                                the demand D) and a min into the row's threshold, one compare per row */
} dy_stats;

/* Options for dy_plan_set_option. */
enum {
    DY_OPT_TIMING = 1,          /* 1: record HIP events around the kernels of each call (default 0) */
    DY_OPT_SAMPLE_STRIDE = 2,   /* the seeding pre-pass scores 1 of every S work units (default 128) */
    DY_OPT_CAND_CAPACITY = 3,   /* candidate slots per source (default 1 << 16, min 16) */
    DY_OPT_FORCE_FP64 = 4,      /* 1: decide every level with the exhaustive fp64 path (default 0) */
    DY_OPT_JIT = 5,             /* kernels generated for the problem (hiprtc): 0 never; 1 (default) for
                                   rows, per-plan scores of 32-bit RANGE sources of DAGs above 16 nodes,
                                   and the sweep of 32-bit RANGE sources of at least 2^24 plans in
                                   plans of at most 8 problems;
                                   2 as 1 but the sweep for RANGE sources of any size */
    DY_OPT_GRAPH = 6,           /* 1: replay a call that repeats the previous one (same sources) from a
                                   HIP graph of its launches (default 1; calls with DY_OPT_TIMING on
                                   launch directly); results are identical */
    DY_OPT_CLIMB = 7            /* local-search seeds: RANGE sources that cover the whole plan space of a
                                   problem of at most 8 nodes also seed each level's threshold from a
                                   local search over the plans (the sampling pass then thins out); under
                                   the additive objective only when lambda_l and every lambda_ld L_k are
                                   not negative.  0: never; 1 (default): in calls of at least 128 such
                                   sources; 2: for every such source.  Results are identical */
};

/*
 * Validate and stage n_probs problems on HIP device `device`.  Derives, once,
 * the fp32 tables (per-node factor 1 - w(1 - p), duration, demand term), the
 * per-level certification bands and the DAG structure (Algorithm gen: bind
 * coefficients once for all levels), and copies them to device memory owned
 * by the handle.  Validation runs before any HIP call.
 * On success *out is the new handle; on failure *out = NULL.
 */
int dy_plan_create(const dy_problem* probs, int32_t n_probs, int32_t device, dy_plan** out);

/*
 * Select, for every source, the best feasible plan of each level: one
 * pressure-specialised variant per level (Sec. 4.4, eq. variant-objective:
 * the same bound coefficients re-solved at each level; Algorithm gen: one
 * solve per level, the results bundled).  corr / SLO problems: the greatest
 * corr among plans with CP_k <= slo (Sec. 4.3 longest path, inclusive bound);
 * objective problems: the greatest J_k (Sec. 4.3 eq. admission-objective).
 * Equal scores go to the lowest plan index.
 *  src     HOST array of n_src sources (each names a problem of the handle;
 *          several sources may name the same problem).
 *  out     HOST array [n_src][dy_plan_max_levels(h)]; row s, column k is level
 *          k of source s (columns >= that problem's n_levels are untouched).
 *  stream  a hipStream_t (NULL: the default stream); kernels run on it and
 *          the call synchronises it before returning.
 */
int dy_plan_select(dy_plan* h, const dy_source* src, int32_t n_src, dy_choice* out, void* stream);

/*
 * dy_plan_select for callers that cannot allocate memory (serving loops that
 * must not call hipMalloc, harnesses that forbid it): the same selection, the
 * same arguments and results, but every per-call device buffer (seed slots,
 * thresholds, prefilter tables, candidate lists, certification state, the
 * choices) lives in one fixed array of 16 MiB that the library holds on each
 * device it runs on until the process ends.  No device or pinned host memory
 * is allocated and no kernel is compiled or loaded: a problem's generated
 * kernels are used when an earlier dy_plan_select call has loaded them, the
 * library's own kernels otherwise (identical results).  The choices are
 * copied back through the caller's `out` array; the call synchronises
 * `stream` before returning.  Limits: at most 64 sources per call, and the
 * candidate slots per source are what the array leaves (about 14,000 with 64
 * sources; overflowing lists are resolved exactly, as in dy_plan_select);
 * beyond them it fails with DY_ELIMIT and a message.  Every such call on a
 * device shares that device's array, whatever the handle: calls that overlap
 * on one device (other host threads, other handles, streams not ordered
 * after each other) race and must be serialised by the caller.  Each call
 * clears what it needs before use; the array keeps the last call's contents.
 */
int dy_plan_select_static(dy_plan* h, const dy_source* src, int32_t n_src, dy_choice* out, void* stream);

/*
 * Per-plan scores of one source (the quantities Sec. 4.3 and Sec. 4.4 attach
 * to a plan: vulnerability-weighted correctness, the longest path at every
 * level, the D_tau demand annotation), written asynchronously on `stream` into
 * caller-owned DEVICE buffers (any may be NULL to skip it):
 *  corr[count], cp[count][K] (CP at each level), demand[count],
 *  feas_bits[count] (bit k set iff CP_k <= slo, decided exactly; K <= 32).
 * Objective mode: corr = sum of the utilities U, cp[.][k] = J_k, demand = D_tau
 * (fp32; |error| below the per-level bound of the certification), every bit set.
 * Inputs and outputs must stay valid until the stream work completes.
 */
int dy_plan_score(dy_plan* h, const dy_source* src, float* corr, float* cp, float* demand,
                  uint32_t* feas_bits, void* stream);

/*
 * The HIP source of the kernels the library generates for one problem and
 * compiles at run time with hiprtc (the streamed-rows kernels and, for
 * uniform pressure or the objective, their per-plan score kernel; for DAGs
 * of at least three nodes the range sweep and its seeding pass), with the
 * problem's structure and constants written in.  Host-only (no HIP call): for inspection and offline
 * compilation.  Writes at most cap bytes, NUL-terminated when cap > 0, and
 * sets *len to the full length without the NUL.  Returns dy_plan_create's
 * status for an invalid problem (message in dy_plan_last_error(NULL)).
 */
int dy_kernel_source(const dy_problem* prob, char* buf, uint64_t cap, uint64_t* len);

/* Free the handle and its device memory (NULL is a no-op).  The compiled
 * per-level variants live only as the choices a caller copied out
 * (Algorithm gen returns the bundle; nothing of it stays in the handle).
 * Calls still running on a stream must have completed. */
void dy_plan_destroy(dy_plan* h);

int32_t dy_plan_max_levels(const dy_plan* h);
int32_t dy_plan_num_problems(const dy_plan* h);
int dy_plan_set_option(dy_plan* h, int32_t option, int64_t value);
int dy_plan_get_stats(const dy_plan* h, dy_stats* out);

const char* dy_plan_last_error(const dy_plan* h);
const char* dy_status_str(int status);
int32_t dy_abi_version(void);

/* Host-only checks of the library's internal arithmetic helpers (the
 * invariant-divisor digit decode used for mixed-radix plan indices, the
 * directed fp32 roundings of the certification bands).  No HIP call.
 * Returns the number of failed checks (0: all pass). */
int dy_selftest(void);

/*
 * Suffix recompilation (Appendix "Suffix Recompilation and Its Timing Scope",
 * eq. suffix-repair).  After a successful bounded recovery the committed
 * nodes C_t (completed or in flight: their bindings are fixed) leave the
 * choice, and the undispatched nodes U_t are selected again on the residual
 * DAG G_t = G[U_t], whose makespan starts from zero; the updated plan is the
 * committed bindings joined with the suffix's.  Host-only calls (no HIP).
 *
 * dy_suffix_create   residual problem of `full` for committed[N] (nonzero =
 *                    committed): the nodes of U_t in their original order
 *                    (still topological), the edges between two of them, their
 *                    table rows; objective mode keeps the weights and levels
 *                    and takes the nodes' cost rows and tool flags (reach
 *                    weights then follow G_t, as for any problem); corr / SLO
 *                    problems keep levels, pressures and SLO.  The handle owns
 *                    copies of everything.  Fails with the status of
 *                    dy_plan_create's checks for an invalid `full`, DY_EINVAL
 *                    for NULL arguments or when every node is committed
 *                    (nothing to recompile); dy_plan_last_error(NULL) then
 *                    describes the failure.
 * dy_suffix_problem  the residual problem, valid until dy_suffix_destroy: stage
 *                    it with dy_plan_create and select as usual.
 * dy_suffix_nodes    its node count; node_map (if not NULL, [count]) receives
 *                    the full node of each residual node.
 * dy_suffix_merge    impl_out[N] (host) = committed_impl[n] for committed n,
 *                    else the implementation that residual plan index
 *                    `residual_index` (mixed radix over the residual nodes,
 *                    first node most significant) gives the node; *full_index
 *                    (if not NULL) = the merged plan's index in `full`, or -1
 *                    when it exceeds 2^63 - 1.  DY_EINVAL for NULL arguments, a
 *                    committed id outside [0, radix) or an index outside the
 *                    residual plan space; the two domains never overlap.
 */
/*
 * Plan-bundle annotations (Sec. 4.4; Algorithm gen attaches per-model demand
 * and an estimated quality to each variant; Sec. 5.2: the model receiving the
 * largest share of the planned demand is the variant's dominant model).
 * Host-only.  For the plan impl[N] of `prob`, with model[N][max_radix] the
 * model class (0..n_models-1) of implementation (n, i):
 *  model_demand[n_models]  sum over LLM nodes running model m of their
 *                          nominal duration tau (fp64, node order);
 *  *dominant               the model with the largest demand, equal demand to
 *                          the lowest id; -1 when the plan has no LLM node;
 *  *quality                product over LLM nodes of 1 - v (1 - q), fp64 (the
 *                          chance that no node makes an impact-weighted error).
 * LLM nodes: all nodes, or those objective->is_tool leaves unflagged.
 * DY_EINVAL for NULL pointers or an implementation / model id out of range.
 */
int dy_bundle_annotate(const dy_problem* prob, const int32_t* model, int32_t n_models, const int32_t* impl,
                       double* model_demand, int32_t* dominant, double* quality);

/* A variant of a bundle as the switching rules see it. */
typedef struct dy_variant {
    int32_t dominant;   /* dominant model (-1: none; its load then reads 0) */
    double quality;     /* estimated quality */
} dy_variant;

/* Thresholds of load-driven switching (Sec. 5.2). */
typedef struct dy_switch_rules {
    double high;        /* the active variant's dominant-model load above this triggers a scan of later variants */
    double low;         /* when it does not, return to the lowest-index variant whose dominant load is below this */
    double tolerance;   /* largest accepted drop of estimated quality from the active variant */
    double margin;      /* a later candidate's dominant load must be at most the active one's minus this */
    double dwell;       /* minimum time between two switches */
} dy_switch_rules;

/*
 * Load-driven switching over a bundle of n_variants variants ordered by
 * level (Sec. 5.2, "Switching plan variants").  Host-only.  Starting on
 * variant 0, for each load sample s (time times[s], non-decreasing; loads
 * [n_steps][n_models]): within `dwell` of the last switch nothing changes;
 * if the active variant's dominant-model load exceeds `high`, the first later
 * variant whose dominant model differs from the active one's, is not above
 * `high`, has load at most the active one's minus `margin` and whose quality
 * is at most `tolerance` below the active one's becomes active; otherwise the
 * lowest-index variant below the active one whose dominant load is below
 * `low` and that passes the same quality check; else the selection is kept.
 * active[n_steps] receives the variant after each sample, *n_switches (if not
 * NULL) the number of switches.  DY_EINVAL for NULL pointers, bad counts or a
 * dominant id outside [-1, n_models).
 */
int dy_switch_simulate(const dy_variant* variants, int32_t n_variants, int32_t n_models, const double* times,
                       const double* loads, int32_t n_steps, const dy_switch_rules* rules, int32_t* active,
                       int32_t* n_switches);

typedef struct dy_suffix dy_suffix; /* opaque */
int dy_suffix_create(const dy_problem* full, const uint8_t* committed, dy_suffix** out);
const dy_problem* dy_suffix_problem(const dy_suffix* s);
int32_t dy_suffix_nodes(const dy_suffix* s, int32_t* node_map);
int dy_suffix_merge(const dy_suffix* s, const int32_t* committed_impl, int64_t residual_index, int32_t* impl_out,
                    int64_t* full_index);
void dy_suffix_destroy(dy_suffix* s);

#ifdef __cplusplus
}
#endif

#endif /* DYPLAN_H */
