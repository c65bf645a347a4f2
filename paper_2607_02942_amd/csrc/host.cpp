// Host side of the plan scorer: validation, one-time table derivation
// (Algorithm gen binds coefficients once for every level), certification
// bands, device staging and the orchestration of a selection call.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstddef>
#include <cstdio>
#include <cstring>
#include <functional>
#include <new>
#include <string>
#include <vector>

#include "dyplan.h"
#include "dyplan_internal.h"

namespace dyp {
hipError_t launch_init(JobDev* d_jobs, int njobs, hipStream_t s);
hipError_t launch_table(JobDev* d_jobs, int njobs, hipStream_t s);
hipError_t launch_sample_sweep(const JobDev* d_jobs, int n, bool has_s2, bool obj, uint64_t max_samples,
                               int npre_max, int npre_c, int kmax, hipStream_t s);
hipError_t launch_sweep(const JobDev* d_jobs, int n, bool has_s2, bool obj, uint64_t max_units, int npre_max,
                        int npre_c, int ry, bool b256, bool rad12, int pat, hipStream_t s);
hipError_t launch_sample_generic(const JobDev* d_jobs, int n, uint64_t max_samples, int ncol, hipStream_t s);
hipError_t launch_scan(const JobDev* d_jobs, int n, uint64_t max_units, int ncol, hipStream_t s);
hipError_t launch_certify(const JobDev* d_jobs, int njobs, int waves, int kmax, int nmax, int nrmax, hipStream_t s);
hipError_t launch_exhaust(const JobDev* d_jobs, int njobs, uint64_t max_units, hipStream_t s);
hipError_t launch_reseed(const JobDev* d_jobs, int njobs, hipStream_t s);
hipError_t launch_seed_cands(const JobDev* d_jobs, int njobs, int kmax, int nmax, hipStream_t s);
hipError_t launch_climb(const JobDev* d_jobs, int njobs, int kmax, int modes, int entries, int nodes,
                         hipStream_t s);
hipError_t static_scratch(int device, char** ptr, size_t* bytes);
struct JitRows {
    hipModule_t mod = nullptr;
    hipFunction_t scan = nullptr;
    hipFunction_t scan_u = nullptr;
    hipFunction_t sample = nullptr;
    hipFunction_t score_rows = nullptr;
    hipFunction_t sweep = nullptr;
    hipFunction_t seed = nullptr;
};
bool jit_rows_get(int device, const ProbDev& D, JitRows* out, std::string* err);
std::string jit_rows_source(const ProbDev& D);
hipError_t launch_score(const JobDev& job, uint64_t units, float* corr, float* cp, float* dem, uint32_t* feas,
                        int n_nodes, int n_entries, int ry, bool simple, bool obj, hipStream_t s);
}  // namespace dyp

using namespace dyp;

namespace {

thread_local std::string g_create_error;

constexpr uint64_t kMaxSourcePlans = 1ull << 40;
constexpr size_t kCandPoolBytes = 1ull << 30;    // candidate slots shared by the sources of one call
constexpr uint64_t kMinSamples = 4096;           // the adaptive stride keeps at least this many samples
constexpr int kDirectResults = 64;                // up to this many sources, results go straight to host memory
constexpr int kStaticSources = 64;                // sources per dy_plan_select_static call at most
constexpr uint32_t kStaticMinCand = 1024;         // candidate slots per source it needs at least
constexpr int kClimbNodes = 8;                    // local-search seeds for problems of at most this many nodes
constexpr int kClimbMinSources = 128;             // ... in calls of at least this many such sources (DY_OPT_CLIMB 1)
// ROWS sources of at least kSplitRows rows under per-backend pressure
// (generated kernels) are scored in two shares: the first 1/kSplitShare of the
// rows, then the candidates gathered so far re-seed the thresholds
// (k_seed_cands), then the rest.  The sampled seeds then only serve the first
// share, so they are sparser (stride up to kSplitStride).  Under per-backend
// pressure the prefilter works on the unpressured CP and passes most rows
// unless the thresholds are near the optimum; under uniform pressure the
// sampled seeds already abandon most rows early and a second share measured
// no gain.
constexpr uint64_t kSweepRunMin = 1ull << 20;    // library sweep: runs of blocks per thread for groups of this many blocks
constexpr uint64_t kSplitRows = 1ull << 22;
constexpr uint64_t kSplitShare = 32;
constexpr uint64_t kSplitStride = 512;
constexpr double kU = 0x1p-24;                    // fp32 unit roundoff

struct HostProb {
    int n = 0, k = 0, b = 0, rmax = 0;
    int npre = 0, rx = 1, ry = 1;
    bool uniform = true, has_s2 = false;
    bool obj = false;           // the paper's additive objective instead of corr / SLO
    uint64_t n_plans = 0;       // saturated
    bool plans_saturated = false;
};

struct Scratch {
    size_t jobs = 0;            // sources the buffers hold
    bool clean = false;         // every job slot's seeds, counters and flags are zero (no k_init needed)
    uint32_t* sync = nullptr;   // [jobs] certification block counters
    uint32_t cap = 0;           // candidate slots per source
    int kmax = 0;
    char* d = nullptr;
    size_t bytes = 0;
    JobDev* d_jobs = nullptr;
    JobDev* d_fb = nullptr;
    uint32_t* scert = nullptr;
    float* thr = nullptr;
    uint32_t* table = nullptr;
    uint32_t* table2 = nullptr;
    uint32_t* ncand = nullptr;
    int32_t* flags = nullptr;
    dy_choice* out = nullptr;
    uint64_t* fb_corr = nullptr;
    uint64_t* fb_index = nullptr;
    double* cert_c = nullptr;
    uint64_t* cert_i = nullptr;
    double* cert_cp = nullptr;
    double* cert_d = nullptr;
    Cand* cand = nullptr;
    size_t res_bytes = 0;       // out, ncand and flags are one contiguous region (one copy back)
    // pinned host mirrors
    JobDev* h_jobs = nullptr;   // the job array last uploaded
    JobDev* h_fb = nullptr;
    char* h_res = nullptr;      // pinned, host-coherent result region (choices, counters, flags)
    char* d_hres = nullptr;     // its device address: certification writes it directly
    size_t res_ncand_off = 0, res_flags_off = 0;
    dy_choice* h_out = nullptr;
    uint32_t* h_ncand = nullptr;
    int32_t* h_flags = nullptr;
    uint32_t* h_done = nullptr;  // pinned, host-coherent: one completion word per source
    uint32_t* d_done = nullptr;  // its device address
    size_t uploaded = 0;        // jobs of h_jobs present on the device (0: none)
};

uint32_t f2u(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    return u;
}

float round_down(double x) {
    float f = (float)x;
    if ((double)f > x) f = std::nextafter(f, -INFINITY);
    return f;
}

float round_up(double x) {
    float f = (float)x;
    if ((double)f < x) f = std::nextafter(f, INFINITY);
    return f;
}

Magic make_magic(uint64_t d) {
    Magic g{0u, 0u, 0u, (uint32_t)d};
    int l = 0;
    while ((1ull << l) < d) ++l;
    unsigned __int128 num = ((unsigned __int128)1 << 32) * (unsigned __int128)((1ull << l) - d);
    g.m = (uint32_t)(num / d + 1);
    g.sh1 = l < 1 ? (uint32_t)l : 1u;
    g.sh2 = l > 1 ? (uint32_t)(l - 1) : 0u;
    return g;
}

uint32_t magic_div(uint32_t x, const Magic& g) {
    uint32_t t = (uint32_t)(((uint64_t)g.m * x) >> 32);
    return (t + ((x - t) >> g.sh1)) >> g.sh2;
}

uint64_t sat_mul(uint64_t a, uint64_t b, bool* sat) {
    unsigned __int128 r = (unsigned __int128)a * b;
    if (r > (unsigned __int128)UINT64_MAX) {
        *sat = true;
        return UINT64_MAX;
    }
    return (uint64_t)r;
}

bool finite_f(float x) { return std::isfinite(x); }

int fail(std::string* err, int status, const char* fmt, int a = 0, int b = 0, int c = 0) {
    char buf[256];
    std::snprintf(buf, sizeof buf, fmt, a, b, c);
    *err = buf;
    return status;
}

// Objective mode: reach(n) = 1 + beta e (|R(n)| - 1) / (|V| - 1), R(n) = n and
// every node reachable from it (Sec. 4.3, the reach weight of the utility);
// the fp64 operations in the order the definition writes them.
void obj_reach(const dy_problem& pb, double* reach) {
    const int N = pb.n_nodes;
    uint32_t desc[DY_MAX_NODES];
    for (int n = N - 1; n >= 0; --n) {
        desc[n] = 1u << n;
        for (int e = 0; e < pb.n_edges; ++e)
            if (pb.edges[2 * e] == n) desc[n] |= desc[pb.edges[2 * e + 1]];
    }
    const dy_objective& o = *pb.objective;
    for (int n = 0; n < N; ++n) {
        if (N == 1) {
            reach[n] = 1.0;
            continue;
        }
        double t = (double)o.beta * (double)o.effort;
        t = t * (double)(__builtin_popcount(desc[n]) - 1);
        t = t / (double)(N - 1);
        reach[n] = 1.0 + t;
    }
}

bool obj_is_llm(const dy_problem& pb, int n) { return !pb.objective->is_tool || pb.objective->is_tool[n] == 0; }

// u = reach q - lambda_f v (1 - q) - lambda_c c of an LLM node's implementation
// (Sec. 4.3, eq. admission-objective: quality weighted by reach, minus the
// impact-weighted error f = v r with r = 1 - q, minus the weighted cost), in fp64,
// one operation per statement.
double obj_u(const dy_problem& pb, double reach, int n, size_t e) {
    const dy_objective& o = *pb.objective;
    const double q = (double)pb.p[e];
    double a = reach * q;
    double b = 1.0 - q;
    b = (double)pb.w[n] * b;
    b = (double)o.lambda_f * b;
    a = a - b;
    b = (double)o.lambda_c * (double)o.cost[e];
    a = a - b;
    return a;
}

int validate_objective(const dy_problem& pb, int idx, double sum_tau, std::string* err) {
    const dy_objective& o = *pb.objective;
    if (!o.cost || !o.levels) return fail(err, DY_EINVAL, "problem %d: objective cost or levels is NULL", idx);
    if (o.n_levels < 1) return fail(err, DY_EINVAL, "problem %d: objective n_levels must be >= 1", idx);
    if (o.n_levels > DY_MAX_LEVELS)
        return fail(err, DY_ELIMIT, "problem %d: objective n_levels %d exceeds %d", idx, o.n_levels, DY_MAX_LEVELS);
    if (!finite_f(o.lambda_f) || !finite_f(o.lambda_c) || !finite_f(o.beta))
        return fail(err, DY_EINVAL, "problem %d: objective weights must be finite", idx);
    if (!(o.lambda_l >= 0.0f && finite_f(o.lambda_l)) || !(o.lambda_ld >= 0.0f && finite_f(o.lambda_ld)))
        return fail(err, DY_EINVAL, "problem %d: lambda_l and lambda_ld must be finite and >= 0", idx);
    if (!(o.effort >= 0.0f && o.effort <= 1.0f))
        return fail(err, DY_EINVAL, "problem %d: effort not in [0, 1]", idx);
    double lmax = 0.0;
    for (int k = 0; k < o.n_levels; ++k) {
        if (!(o.levels[k] >= 0.0f && finite_f(o.levels[k])))
            return fail(err, DY_EINVAL, "problem %d: level %d must be finite and >= 0", idx, k);
        lmax = std::max(lmax, (double)o.levels[k]);
    }
    const int N = pb.n_nodes;
    double reach[DY_MAX_NODES];
    obj_reach(pb, reach);
    double su = 0.0;
    for (int n = 0; n < N; ++n) {
        if (o.is_tool && o.is_tool[n] != 0 && o.is_tool[n] != 1)
            return fail(err, DY_EINVAL, "problem %d: is_tool[%d] must be 0 or 1", idx, n);
        if (!std::isfinite(reach[n])) return fail(err, DY_EINVAL, "problem %d: reach weight of node %d overflows", idx, n);
        double mu = 0.0;
        for (int i = 0; i < pb.radix[n]; ++i) {
            const size_t e = (size_t)n * pb.max_radix + i;
            if (!finite_f(o.cost[e]))
                return fail(err, DY_EINVAL, "problem %d: cost[%d][%d] must be finite", idx, n, i);
            if (obj_is_llm(pb, n)) mu = std::max(mu, std::fabs(obj_u(pb, reach[n], n, e)));
        }
        su += mu;
    }
    if (!(su <= 1e30)) return fail(err, DY_EINVAL, "problem %d: utilities too large", idx);
    if ((double)o.lambda_l * sum_tau > 1e30 || (double)o.lambda_ld * lmax * sum_tau > 1e30)
        return fail(err, DY_EINVAL, "problem %d: weighted latency or demand too large", idx);
    return DY_OK;
}

int validate_problem(const dy_problem& pb, int idx, std::string* err) {
    const int N = pb.n_nodes;
    const bool obj = pb.objective != nullptr;
    if (N < 1) return fail(err, DY_EINVAL, "problem %d: n_nodes must be >= 1", idx);
    if (N > DY_MAX_NODES) return fail(err, DY_ELIMIT, "problem %d: n_nodes %d exceeds %d", idx, N, DY_MAX_NODES);
    if (pb.n_edges < 0) return fail(err, DY_EINVAL, "problem %d: negative n_edges", idx);
    if (pb.n_edges > 0 && !pb.edges) return fail(err, DY_EINVAL, "problem %d: edges is NULL", idx);
    if (pb.n_edges > DY_MAX_NODES * DY_MAX_NODES)
        return fail(err, DY_ELIMIT, "problem %d: too many edges", idx);
    if (!pb.radix || !pb.p || !pb.tau || !pb.w || (!obj && (!pb.size || !pb.backend || !pb.rho)))
        return fail(err, DY_EINVAL, "problem %d: a table pointer is NULL", idx);
    if (!obj) {
        if (pb.n_levels < 1) return fail(err, DY_EINVAL, "problem %d: n_levels must be >= 1", idx);
        if (pb.n_levels > DY_MAX_LEVELS)
            return fail(err, DY_ELIMIT, "problem %d: n_levels %d exceeds %d", idx, pb.n_levels, DY_MAX_LEVELS);
        if (pb.n_backends < 1) return fail(err, DY_EINVAL, "problem %d: n_backends must be >= 1", idx);
        if (pb.n_backends > DY_MAX_BACKENDS)
            return fail(err, DY_ELIMIT, "problem %d: n_backends %d exceeds %d", idx, pb.n_backends,
                        DY_MAX_BACKENDS);
    }
    int rmax = 0;
    for (int n = 0; n < N; ++n) {
        if (pb.radix[n] < 1) return fail(err, DY_EINVAL, "problem %d: radix[%d] < 1", idx, n);
        if (pb.radix[n] > DY_MAX_RADIX)
            return fail(err, DY_ELIMIT, "problem %d: radix[%d] exceeds %d", idx, n, DY_MAX_RADIX);
        rmax = std::max(rmax, pb.radix[n]);
    }
    if (pb.max_radix < rmax || pb.max_radix > (1 << 16))
        return fail(err, DY_EINVAL, "problem %d: max_radix %d must be in [max radix, 65536]", idx, pb.max_radix);
    for (int e = 0; e < pb.n_edges; ++e) {
        int u = pb.edges[2 * e], v = pb.edges[2 * e + 1];
        if (u < 0 || v < 0 || u >= N || v >= N)
            return fail(err, DY_EINVAL, "problem %d: edge %d names a node out of range", idx, e);
        if (u >= v)
            return fail(err, DY_ENOTDAG, "problem %d: edge %d is not (u, v) with u < v (topological numbering)", idx, e);
    }
    double sum_tau = 0.0, sum_dem = 0.0;
    for (int n = 0; n < N; ++n) {
        float w = pb.w[n];
        if (!(w >= 0.0f && w <= 1.0f)) return fail(err, DY_EINVAL, "problem %d: w[%d] not in [0, 1]", idx, n);
        double mt = 0.0, md = 0.0;
        for (int i = 0; i < pb.radix[n]; ++i) {
            size_t e = (size_t)n * pb.max_radix + i;
            float p = pb.p[e], t = pb.tau[e];
            if (!(p >= 0.0f && p <= 1.0f))
                return fail(err, DY_EINVAL, "problem %d: p[%d][%d] not in [0, 1]", idx, n, i);
            if (!finite_f(t) || t < 0.0f)
                return fail(err, DY_EINVAL, "problem %d: tau[%d][%d] must be finite and >= 0", idx, n, i);
            mt = std::max(mt, (double)t);
            if (obj) continue;
            float s = pb.size[e];
            int b = pb.backend[e];
            if (!finite_f(s) || s < 0.0f)
                return fail(err, DY_EINVAL, "problem %d: size[%d][%d] must be finite and >= 0", idx, n, i);
            if (b < 0 || b >= pb.n_backends)
                return fail(err, DY_EINVAL, "problem %d: backend[%d][%d] out of range", idx, n, i);
            md = std::max(md, (double)t * (double)s);
        }
        sum_tau += mt;
        sum_dem += md;
    }
    if (sum_tau > 1e30) return fail(err, DY_EINVAL, "problem %d: durations too large", idx);
    if (obj) return validate_objective(pb, idx, sum_tau, err);
    for (int k = 0; k < pb.n_levels; ++k)
        for (int b = 0; b < pb.n_backends; ++b) {
            float r = pb.rho[k * pb.n_backends + b];
            if (!(r >= 0.0f && r < 1.0f))
                return fail(err, DY_EINVAL, "problem %d: rho[%d][%d] not in [0, 1)", idx, k, b);
            if (sum_tau / (1.0 - (double)r) > 1e30)
                return fail(err, DY_EINVAL, "problem %d: durations too large at level %d", idx, k);
        }
    if (sum_dem > 1e30) return fail(err, DY_EINVAL, "problem %d: demand terms too large", idx);
    if (!(pb.slo >= 0.0f)) return fail(err, DY_EINVAL, "problem %d: slo must be >= 0 (and not NaN)", idx);
    return DY_OK;
}

// fp32 longest path with one duration per node (the kernels' recurrence).
float cp32(int N, const uint32_t* pred, uint32_t sinks, const float* d) {
    float f[DY_MAX_NODES];
    float best = 0.0f;
    for (int n = 0; n < N; ++n) {
        float m = 0.0f;
        for (int u = 0; u < n; ++u)
            if (pred[n] >> u & 1u) m = std::max(m, f[u]);
        f[n] = d[n] + m;
        if (sinks >> n & 1u) best = std::max(best, f[n]);
    }
    return best;
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace

// The kernel family that scores a source.
// Sources of one call are launched in groups: the prefix-shared sweep (RANGE,
// uniform pressure; with or without a second sink term; corr / SLO or the
// additive objective), the generic per-plan path, and the generated rows kernels.
enum Group { G_SWEEP = 0, G_SWEEP_S2 = 1, G_OSWEEP = 2, G_OSWEEP_S2 = 3, G_GENERIC = 4, G_JIT = 5 };
constexpr int kGroups = 6, kSweepGroups = 4;

struct PassPlan {
    int n[kGroups] = {};                  // sources per group, stored in group order
    uint64_t units[G_JIT] = {};           // largest main-pass work of the group
    uint64_t samples[G_JIT] = {};         // largest seeding-pass work of the group
    int npre[kSweepGroups] = {};
    int ry[kSweepGroups] = {};            // R_y shared by every source of a sweep group, else -1
    int npre_c[kSweepGroups] = {};        // prefix length shared by every source of a sweep group, else -1
    int pat[kSweepGroups] = {};           // largest prefix-row table (npre x rmax entries) of a sweep group
    int ydiv_jit[kSweepGroups] = {};      // generated sweeps on thresholds divided (corr) or lowered (objective) by y's terms
    int sample_lib[kSweepGroups] = {};    // library-sweep sources the sampling pass seeds (see launch_seed)
    int njit[kSweepGroups] = {};          // trailing sources of the group that run their generated sweep
    bool b256[kSweepGroups] = {true, true, true, true};  // every library-sweep source has the 256-bin table
    bool rad12[kSweepGroups] = {true, true, true, true}; // ... and 12 implementations per prefix node, 32-bit blocks
    int kmax = 1;                         // most levels of any source
    int climb_e = 0;                      // largest sum of radices of a source that climbs
    int climb_n = 0;                      // most nodes of a source that climbs
    int ncol = 1;                         // most nodes of any source of the generic group
    int before(int g) const {             // jobs stored ahead of group g
        int t = 0;
        for (int q = 0; q < g; ++q) t += n[q];
        return t;
    }
};

// What a selection call derives from its sources and the handle's state
// before launching: the group of every source, the launch order, the job
// array and the launch plan.  A call whose sources and state equal the
// previous call's reuses it (for 4,096 sources deriving it takes about 130
// microseconds of host time, during which the device would wait).
struct CallPlan {
    bool valid = false;
    // the key: sources, candidate slots, scratch, options, generated-kernel states
    std::vector<dy_source> src;
    uint64_t cap = 0;
    const void* scratch = nullptr;
    int64_t opts[6] = {};
    std::vector<int> jit_state;
    // the derived plan
    std::vector<int> grp, order;
    std::vector<JobDev> jobs;
    PassPlan pp;
    int n3 = 0;
    uint64_t plans = 0, all_units = 0;
    bool any_split = false, any_climb = false;
    int climb_modes = 0;
};

struct dy_plan {
    int device = 0;
    int kmax = 0;
    int nmax = 0, nrmax = 0;          // most nodes and node-table entries (N x R_max) of any problem
    std::vector<HostProb> hp;
    std::vector<ProbDev> hdesc;       // host copies of the device descriptors
    std::vector<int> jit_state;       // per problem: 0 untried, 1 ready, -1 unavailable
    std::vector<JitRows> jit;
    int use_jit = 1;
    int cus = 0;                      // compute units of the device
    char* d_arena = nullptr;
    ProbDev* d_probs = nullptr;
    Scratch sc;
    int timing = 0;
    uint32_t sample_stride = 128;   // upper bound of the adaptive stride, or the fixed stride when set
    bool stride_fixed = false;
    uint32_t cand_cap = 1u << 16;
    int force_fp64 = 0;
    int use_climb = 1;                // local-search seeds: 0 never, 1 for calls of many sources, 2 always
    std::vector<char> st_host;        // host copies of dy_plan_select_static's jobs and results
    hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};
    // A call that repeats the previous one (same job array, scratch clear) is
    // replayed from a HIP graph of its launches: one submission instead of one
    // per kernel, which on gfx950 costs more host time than the short kernels
    // of a selection run.  Captured on an internal stream, launched on the
    // caller's.
    // Calls with timing on always launch directly: events recorded inside a
    // captured graph are not updated by its replays on this runtime.
    int use_graph = 1;
    hipStream_t cap_stream = nullptr;
    hipGraphExec_t graph = nullptr;
    CallPlan call;                    // the last dy_plan_select call's plan
    dy_stats stats{};
    std::string err;
};

namespace {

struct DeviceGuard {
    int prev = -1;
    bool ok = false;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        ok = hipSetDevice(dev) == hipSuccess;
    }
    ~DeviceGuard() {
        if (prev >= 0) (void)hipSetDevice(prev);
    }
};

int hip_fail(std::string* err, hipError_t e, const char* what) {
    *err = std::string(what) + ": " + hipGetErrorString(e);
    return e == hipErrorOutOfMemory ? DY_ENOMEM : DY_EDEVICE;
}

void free_scratch(Scratch& s) {
    if (s.d) (void)hipFree(s.d);
    if (s.h_jobs) (void)hipHostFree(s.h_jobs);
    if (s.h_fb) (void)hipHostFree(s.h_fb);
    if (s.h_res) (void)hipHostFree(s.h_res);
    if (s.h_done) (void)hipHostFree(s.h_done);
    s = Scratch{};
}

// Lays the per-call buffers of njobs sources (cap candidate slots each) out
// from device address d (null: only the size); returns the bytes they span.
size_t layout_scratch(Scratch& s, char* d, size_t njobs, uint32_t cap, int km) {
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = align_up(off, 256);
        off = o + bytes;
        return o;
    };
    size_t o_jobs = take(njobs * sizeof(JobDev));
    size_t o_fb = take(njobs * sizeof(JobDev));
    size_t o_scert = take(njobs * KMAX * NSLOT * sizeof(uint32_t));
    size_t o_cc = take(njobs * KMAX * CERT_WAVES * sizeof(double));
    size_t o_ci = take(njobs * KMAX * CERT_WAVES * sizeof(uint64_t));
    size_t o_cp = take(njobs * KMAX * CERT_WAVES * sizeof(double));
    size_t o_cd = take(njobs * KMAX * CERT_WAVES * sizeof(double));
    size_t o_thr = take(njobs * KMAX * sizeof(float));
    size_t o_table = take(njobs * NBINS * sizeof(uint32_t));
    size_t o_table2 = take(njobs * NBINS2 * sizeof(uint32_t));
    const size_t res_out = 0;
    const size_t res_ncand = align_up(njobs * km * sizeof(dy_choice), 8);
    const size_t res_flags = res_ncand + njobs * sizeof(uint32_t);
    const size_t res_bytes = res_flags + njobs * sizeof(int32_t);
    size_t o_res = take(res_bytes);
    size_t o_fbc = take(njobs * KMAX * sizeof(uint64_t));
    size_t o_fbi = take(njobs * KMAX * sizeof(uint64_t));
    size_t o_sync = take(njobs * sizeof(uint32_t));
    size_t o_cand = take(njobs * (size_t)cap * sizeof(Cand));
    off = align_up(off, 256);
    s.res_bytes = res_bytes;
    s.res_ncand_off = res_ncand;
    s.res_flags_off = res_flags;
    if (!d) return off;
    s.d = d;
    s.bytes = off;
    s.jobs = njobs;
    s.cap = cap;
    s.kmax = km;
    s.d_jobs = (JobDev*)(d + o_jobs);
    s.d_fb = (JobDev*)(d + o_fb);
    s.scert = (uint32_t*)(d + o_scert);
    s.cert_c = (double*)(d + o_cc);
    s.cert_i = (uint64_t*)(d + o_ci);
    s.cert_cp = (double*)(d + o_cp);
    s.cert_d = (double*)(d + o_cd);
    s.thr = (float*)(d + o_thr);
    s.table = (uint32_t*)(d + o_table);
    s.table2 = (uint32_t*)(d + o_table2);
    s.out = (dy_choice*)(d + o_res + res_out);
    s.ncand = (uint32_t*)(d + o_res + res_ncand);
    s.flags = (int32_t*)(d + o_res + res_flags);
    s.sync = (uint32_t*)(d + o_sync);
    s.fb_corr = (uint64_t*)(d + o_fbc);
    s.fb_index = (uint64_t*)(d + o_fbi);
    s.cand = (Cand*)(d + o_cand);
    s.clean = false;  // the next call clears the scratch first
    return off;
}

int ensure_scratch(dy_plan* h, size_t njobs, uint32_t cap) {
    Scratch& s = h->sc;
    if (s.d && s.jobs >= njobs && s.cap >= cap && s.kmax == h->kmax) return DY_OK;
    free_scratch(s);
    const int km = h->kmax;
    const size_t off = layout_scratch(s, nullptr, njobs, cap, km);
    char* d = nullptr;
    hipError_t e = hipMalloc((void**)&d, off);
    if (e != hipSuccess) return hip_fail(&h->err, e, "hipMalloc(scratch)");
    layout_scratch(s, d, njobs, cap, km);
    const size_t res_bytes = s.res_bytes;
    if ((e = hipHostMalloc((void**)&s.h_jobs, njobs * sizeof(JobDev), hipHostMallocDefault)) != hipSuccess ||
        (e = hipHostMalloc((void**)&s.h_fb, njobs * sizeof(JobDev), hipHostMallocDefault)) != hipSuccess ||
        (e = hipHostMalloc((void**)&s.h_res, res_bytes, hipHostMallocMapped | hipHostMallocCoherent)) !=
            hipSuccess ||
        (e = hipHostGetDevicePointer((void**)&s.d_hres, s.h_res, 0)) != hipSuccess ||
        (e = hipHostMalloc((void**)&s.h_done, njobs * sizeof(uint32_t), hipHostMallocMapped | hipHostMallocCoherent)) !=
            hipSuccess ||
        (e = hipHostGetDevicePointer((void**)&s.d_done, s.h_done, 0)) != hipSuccess) {
        free_scratch(s);
        return hip_fail(&h->err, e, "hipHostMalloc(scratch)");
    }
    s.h_out = (dy_choice*)(s.h_res);
    s.h_ncand = (uint32_t*)(s.h_res + s.res_ncand_off);
    s.h_flags = (int32_t*)(s.h_res + s.res_flags_off);
    s.uploaded = 0;
    return DY_OK;
}

// The per-call buffers of dy_plan_select_static: laid out in the library's
// fixed device array of this device (kStaticBytes, no allocation), with the
// host-side copies in buffers the handle allocated at creation.  The
// candidate slots per source are what the array has left, at most `cap`.
int static_view(dy_plan* h, size_t njobs, uint32_t cap, Scratch* s) {
    if (njobs > (size_t)kStaticSources) {
        h->err = "dy_plan_select_static: more than " + std::to_string(kStaticSources) +
                 " sources in one call (the fixed scratch array holds that many)";
        return DY_ELIMIT;
    }
    char* base = nullptr;
    size_t bytes = 0;
    const hipError_t e = static_scratch(h->device, &base, &bytes);
    if (e != hipSuccess) return hip_fail(&h->err, e, "hipGetSymbolAddress(scratch)");
    const int km = h->kmax;
    const size_t fixed = layout_scratch(*s, nullptr, njobs, 0, km) + 256;
    const uint64_t fit = fixed < bytes ? (bytes - fixed) / (njobs * sizeof(Cand)) : 0;
    const uint32_t c = (uint32_t)std::min<uint64_t>(cap, fit);
    if (c < kStaticMinCand) {
        h->err = "dy_plan_select_static: the fixed scratch array is too small for this call";
        return DY_ELIMIT;
    }
    layout_scratch(*s, base, njobs, c, km);
    if (s->bytes > bytes) {
        h->err = "dy_plan_select_static: scratch layout exceeds the fixed array";
        return DY_ELIMIT;
    }
    s->h_jobs = (JobDev*)h->st_host.data();
    s->h_fb = s->h_jobs + kStaticSources;
    s->h_res = (char*)(s->h_fb + kStaticSources);
    s->h_out = (dy_choice*)s->h_res;
    s->h_ncand = (uint32_t*)(s->h_res + s->res_ncand_off);
    s->h_flags = (int32_t*)(s->h_res + s->res_flags_off);
    return DY_OK;
}

// Builds the device image of every problem: ProbDev descriptors + tables.
// Objective mode: tables of the per-node terms and the certification bounds.
// An fp32 estimate of a plan's J_k (sums of the fp32-rounded terms in node
// order, the longest path in fp32, then the weights) differs from the fp64
// evaluation of the definition by at most E_k = (N + 6) u A_k (1 + 2^-10) +
// (3N + 8) 2^-149 (1 + lambda_l + m_k), with A_k = sum of the largest |u| +
// lambda_l T_max + m_k D_max, m_k = lambda_ld L_k: the sums of N terms err by
// (N - 1) u of their magnitude, each rounded term and weight product by u more,
// and fp64 adds (N + 3) 2^-53; the last term covers subnormal roundings.
void stage_objective(const dy_problem& pb, ProbDev& D, float2* at, float2* atx, float* dz, float* dem, float* lat,
                     double* a64, double* lat64, double* dem64) {
    const dy_objective& o = *pb.objective;
    const int N = pb.n_nodes, R = pb.max_radix, K = o.n_levels;
    double reach[DY_MAX_NODES];
    obj_reach(pb, reach);
    D.obj = 1;
    D.llm = 0;
    float dlo = 0.0f, dhi = 0.0f;  // fp32 D of the plans with the smallest / largest d everywhere (node order)
    float tmx[DY_MAX_NODES];
    double su = 0.0, dsum = 0.0;
    for (int n = 0; n < N; ++n) {
        const bool llm = obj_is_llm(pb, n);
        if (llm) D.llm |= 1u << n;
        float dmn = INFINITY, dmx = 0.0f;
        double mu = 0.0;
        tmx[n] = 0.0f;
        for (int i = 0; i < pb.radix[n]; ++i) {
            const size_t e2 = (size_t)n * R + i;
            const float tau = pb.tau[e2] == 0.0f ? 0.0f : pb.tau[e2];
            const double u = llm ? obj_u(pb, reach[n], n, e2) : 0.0;
            const float d = llm ? tau : 0.0f;
            a64[e2] = u;
            dem64[e2] = (double)d;
            lat64[e2] = (double)tau;
            at[e2] = make_float2((float)u, tau);
            dem[e2] = d;
            lat[e2] = tau;
            mu = std::max(mu, std::fabs(u));
            dmn = std::min(dmn, d);
            dmx = std::max(dmx, d);
            tmx[n] = std::max(tmx[n], tau);
        }
        su += mu;
        dsum += (double)dmx;
        dlo = dlo + dmn;
        dhi = dhi + dmx;
    }
    *atx = make_float2(0.0f, 0.0f);
    *dz = 0.0f;
    // longest path with every node at its longest duration, fp64
    double f[DY_MAX_NODES], tmax = 0.0;
    for (int n = 0; n < N; ++n) {
        double m = 0.0;
        for (int v = 0; v < n; ++v)
            if (D.pred[n] >> v & 1u) m = std::max(m, f[v]);
        f[n] = (double)tmx[n] + m;
        if (D.sinks >> n & 1u) tmax = std::max(tmax, f[n]);
    }
    D.cp_lo_bits = f2u(dlo);
    D.cp_hi_bits = f2u(dhi);
    D.lam_l = o.lambda_l;
    D.lam_l64 = (double)o.lambda_l;
    const double grow = 1.0 + 0x1p-20;  // magnitudes of fp32 sums exceed the fp64 ones by < N u
    for (int k = 0; k < K; ++k) {
        const double m = (double)o.lambda_ld * (double)o.levels[k];  // 24 x 24 bits: exact
        D.m64[k] = m;
        D.m32[k] = (float)m;
        const double A = (su + D.lam_l64 * tmax + m * dsum) * grow;
        const double E = (N + 6) * kU * A * (1.0 + 0x1p-10) + (3.0 * N + 8.0) * 0x1p-149 * (1.0 + D.lam_l64 + m);
        D.err2[k] = 2.0 * E * (1.0 + 0x1p-40);
        D.lvl_order[k] = k;
    }
    // Offsets of the sweep's shifted thresholds, per implementation j of y
    // (the last node): c_j >= u_j - lambda_l tau_j + E_s.  A plan's fp32 G and
    // its row's fp32 R = fma(-lambda_l, M, ux) take four roundings between
    // them (tau_j + M, ux + u_j, the fma of G, that of R), each of a value of
    // magnitude below A_0 = sum of the largest |u| + lambda_l T_max (fp32 sums
    // inflated by grow), the first scaled by lambda_l: E_s = 4 u A_0 (1 +
    // 2^-10) plus (4 + 4 lambda_l) 2^-149 for subnormal results.  lambda_l
    // tau_j is exact in fp64 (24 x 24 bits); the sum's own rounding is covered
    // by the 2^-50 margin before rounding up.
    const double A0 = (su + D.lam_l64 * tmax) * grow;
    const double Es = 4.0 * kU * A0 * (1.0 + 0x1p-10) + (4.0 + 4.0 * D.lam_l64) * 0x1p-149;
    const int ry = std::min(pb.radix[N - 1], 64);
    for (int i = 0; i < 64; ++i) {
        float c = 0.0f;
        if (i < ry) {
            const float2 v = at[(size_t)(N - 1) * R + i];
            const double w = (double)v.x - D.lam_l64 * (double)v.y;
            c = round_up(w + Es + (std::fabs(w) + Es) * 0x1p-50);
        }
        D.ysub[i] = c;
    }
}

// dry: derive the descriptors and tables on the host only (no HIP call); the
// descriptors' table pointers then point into a host image that is discarded.
int stage_problems(dy_plan* h, const dy_problem* probs, int32_t n_probs, std::string* err, bool dry = false) {
    struct Layout {
        size_t at, atx, dz, dem, lat, a64, lat64, dem64;
    };
    std::vector<Layout> lay(n_probs);
    size_t off = align_up((size_t)n_probs * sizeof(ProbDev), 256);
    auto take = [&](size_t bytes) {
        size_t o = align_up(off, 256);
        off = o + bytes;
        return o;
    };
    h->hp.resize(n_probs);
    h->kmax = 0;
    h->nmax = 0;
    h->nrmax = 0;
    for (int j = 0; j < n_probs; ++j) {
        const dy_problem& pb = probs[j];
        const size_t NR = (size_t)pb.n_nodes * pb.max_radix;
        // objective mode: one latency level (nominal durations)
        const int KL = pb.objective ? 1 : pb.n_levels;
        Layout& L = lay[j];
        L.at = take(NR * sizeof(float2));
        L.atx = take(sizeof(float2));
        L.dz = take(sizeof(float));
        L.dem = take(NR * sizeof(float));
        L.lat = take((size_t)KL * NR * sizeof(float));
        L.a64 = take(NR * sizeof(double));
        L.lat64 = take((size_t)KL * NR * sizeof(double));
        L.dem64 = take(NR * sizeof(double));
        h->kmax = std::max(h->kmax, pb.objective ? pb.objective->n_levels : pb.n_levels);
        h->nmax = std::max(h->nmax, (int)pb.n_nodes);
        h->nrmax = std::max(h->nrmax, (int)NR);
    }
    std::vector<char> img(off, 0);
    hipError_t e = hipSuccess;
    if (!dry) {
        e = hipMalloc((void**)&h->d_arena, off);
        if (e != hipSuccess) {
            h->d_arena = nullptr;
            return hip_fail(err, e, "hipMalloc(tables)");
        }
        h->d_probs = (ProbDev*)h->d_arena;
    }
    ProbDev* descs = (ProbDev*)img.data();
    for (int j = 0; j < n_probs; ++j) {
        const dy_problem& pb = probs[j];
        const Layout& L = lay[j];
        const bool obj = pb.objective != nullptr;
        const int N = pb.n_nodes, R = pb.max_radix;
        const int K = obj ? pb.objective->n_levels : pb.n_levels, B = obj ? 1 : pb.n_backends;
        ProbDev& D = descs[j];
        std::memset(&D, 0, sizeof D);
        HostProb& H = h->hp[j];
        D.n = N;
        D.k = K;
        D.b = B;
        D.rmax = R;
        // structure
        uint32_t succ = 0;
        for (int e2 = 0; e2 < pb.n_edges; ++e2) {
            int u = pb.edges[2 * e2], v = pb.edges[2 * e2 + 1];
            D.pred[v] |= 1u << u;
            succ |= 1u << u;
        }
        const uint32_t all = N == 32 ? 0xffffffffu : ((1u << N) - 1u);
        D.sinks = all & ~succ;
        D.npre = N >= 2 ? N - 2 : 0;
        D.xnode = N >= 2 ? N - 2 : -1;
        D.ynode = N - 1;
        D.rx = N >= 2 ? pb.radix[N - 2] : 1;
        D.ry = pb.radix[N - 1];
        D.edge_xy = (N >= 2 && (D.pred[N - 1] >> (N - 2) & 1u)) ? 1 : 0;
        D.x_sink = N >= 2 ? (int)((D.sinks >> (N - 2)) & 1u) : 1;
        D.pre_sinks = D.npre > 0 ? (D.sinks & ((1u << D.npre) - 1u)) : 0u;
        for (int n = 0; n < N; ++n) {
            D.radix[n] = pb.radix[n];
            D.rmag[n] = make_magic((uint64_t)pb.radix[n]);
        }
        // place values of prefix nodes inside a block index (product of later prefix radices)
        for (int n = 0; n < D.npre; ++n) {
            bool sat = false;
            uint64_t pv = 1;
            for (int m = n + 1; m < D.npre; ++m) pv = sat_mul(pv, (uint64_t)pb.radix[m], &sat);
            D.pv64[n] = sat ? UINT64_MAX : pv;
            D.pv_big[n] = (sat || pv > 0xffffffffull) ? 1u : 0u;
            D.pvmag[n] = D.pv_big[n] ? Magic{0, 0, 0, 0} : make_magic(pv);
        }
        bool sat = false;
        uint64_t np = 1;
        for (int n = 0; n < N; ++n) np = sat_mul(np, (uint64_t)pb.radix[n], &sat);
        D.n_plans = np;
        H.n_plans = np;
        H.plans_saturated = sat;
        // pressure: uniform when every used backend of a level has the same rho
        uint64_t used = 0;
        if (!obj)
            for (int n = 0; n < N; ++n)
                for (int i = 0; i < pb.radix[n]; ++i) used |= 1ull << pb.backend[(size_t)n * R + i];
        bool uniform = true;
        std::vector<double> rho_k(K, 0.0), rho_lo(K, 0.0), rho_hi(K, 0.0);
        for (int k = 0; k < K && !obj; ++k) {
            bool first = true;
            float r0 = 0.0f, rl = 0.0f, rh = 0.0f;
            for (int b = 0; b < B; ++b) {
                if (!(used >> b & 1ull)) continue;
                float r = pb.rho[k * B + b];
                if (first) {
                    r0 = rl = rh = r;
                    first = false;
                } else {
                    if (f2u(r) != f2u(r0)) uniform = false;
                    rl = std::min(rl, r);
                    rh = std::max(rh, r);
                }
            }
            rho_k[k] = (double)r0;
            rho_lo[k] = (double)rl;
            rho_hi[k] = (double)rh;
        }
        D.uniform = uniform ? 1 : 0;
        D.slo = obj ? INFINITY : (double)pb.slo;
        const double slo = D.slo;
        // certification bands (fp32 CP error <= (N-1) u relative, fp64 oracle error
        // ~ (N+3) 2^-53; the margin (N+1) u covers both, (N+2) u with rounded latencies)
        for (int k = 0; k < K; ++k) {
            if (obj) {  // no hard constraint: every plan is feasible at every level
                D.lo[k] = INFINITY;
                D.hi[k] = INFINITY;
                D.mk[k] = 1.0f;
            } else if (uniform) {
                const double th = slo * (1.0 - rho_k[k]);
                D.lo[k] = round_down(th * (1.0 - (N + 1) * kU));
                D.hi[k] = round_up(th * (1.0 + (N + 1) * kU));
                D.mk[k] = (float)(1.0 / (1.0 - rho_k[k]));
            } else {
                // CP_k <= CP_0 / (1 - largest rho of the level) and >= CP_0 / (1 - smallest):
                // bands on the unpressured CP, widened like the per-level ones
                D.lo[k] = round_down(slo * (1.0 - rho_hi[k]) * (1.0 - (N + 2) * kU));
                D.hi[k] = round_up(slo * (1.0 - rho_lo[k]) * (1.0 + (N + 2) * kU));
                D.mk[k] = 1.0f;
            }
        }
        D.glo = round_down(slo * (1.0 - (N + 2) * kU));
        D.ghi = round_up(slo * (1.0 + (N + 2) * kU));
        // tables
        float2* at = (float2*)(img.data() + L.at);
        float* dem = (float*)(img.data() + L.dem);
        float* lat = (float*)(img.data() + L.lat);
        double* a64 = (double*)(img.data() + L.a64);
        double* lat64 = (double*)(img.data() + L.lat64);
        double* dem64 = (double*)(img.data() + L.dem64);
        float2* atx = (float2*)(img.data() + L.atx);
        if (obj) {
            stage_objective(pb, D, at, atx, (float*)(img.data() + L.dz), dem, lat, a64, lat64, dem64);
        } else {
        float dmin[DY_MAX_NODES], dmax[DY_MAX_NODES];
        for (int n = 0; n < N; ++n) {
            double w = (double)pb.w[n];
            dmin[n] = INFINITY;
            dmax[n] = 0.0f;
            for (int i = 0; i < pb.radix[n]; ++i) {
                size_t e2 = (size_t)n * R + i;
                // the definition's per-node terms in fp64, operation by operation
                double t = 1.0 - (double)pb.p[e2];
                t = w * t;
                const double a = 1.0 - t;
                const float tau = pb.tau[e2] == 0.0f ? 0.0f : pb.tau[e2];
                const double d = (double)tau * (double)pb.size[e2];
                a64[e2] = a;
                dem64[e2] = d;
                at[e2] = make_float2((float)a, tau);
                dem[e2] = (float)d;
                dmin[n] = std::min(dmin[n], tau);
                dmax[n] = std::max(dmax[n], tau);
                for (int k = 0; k < K; ++k) {
                    const double r = (double)pb.rho[k * B + pb.backend[e2]];
                    const double l = (double)tau / (1.0 - r);
                    lat64[(size_t)k * N * R + e2] = l;
                    lat[(size_t)k * N * R + e2] = (float)l;
                }
            }
        }
        *atx = make_float2(1.0f, 0.0f);
        // fp32 bounds of the unpressured CP (the recurrence is monotone in every duration)
        // tail bounds: exact products and sums in fp64, then widened by 2^-18
        // relative (more than N <= 32 fp32 roundings) and rounded outward
        {
            double tail = 1.0;
            D.corr_tail[N] = 1.0f;
            for (int n = N - 1; n >= 0; --n) {
                float amax = 0.0f;
                for (int i = 0; i < pb.radix[n]; ++i) amax = std::max(amax, at[(size_t)n * R + i].x);
                tail *= (double)amax;
                D.corr_tail[n] = round_up(tail * (1.0 + 0x1p-18));
            }
            double rest[DY_MAX_NODES];
            for (int n = N - 1; n >= 0; --n) {
                double best = INFINITY;
                for (int v = n + 1; v < N; ++v)
                    if (D.pred[v] >> n & 1u) best = std::min(best, (double)dmin[v] + rest[v]);
                rest[n] = std::isinf(best) ? 0.0 : best;
                D.lat_tail[n] = round_down(rest[n] * (1.0 - 0x1p-18));
            }
        }
        const float clo = cp32(N, D.pred, D.sinks, dmin);
        const float chi = cp32(N, D.pred, D.sinks, dmax);
        D.cp_lo_bits = f2u(clo);
        D.cp_hi_bits = f2u(chi);
        }
        int s = 2;
        while (s < 31 && ((D.cp_hi_bits >> s) - (D.cp_lo_bits >> s)) > 62u) ++s;
        D.bin_shift = s;
        // the generated sweep bins the CP at 2^18 patterns per bin into 256 bins
        // (one masked half-word read forms the LDS offset) when they cover it
        D.jsh = ((D.cp_hi_bits >> 18) - (D.cp_lo_bits >> 18)) <= (uint32_t)(NBINS2 - 2) ? 18 : 0;
        // seeding pass: levels by decreasing band, and per bin how many of them
        // every CP in the bin certainly meets (decided by the bin's largest CP)
        std::vector<int> order(K);
        for (int k = 0; k < K; ++k) order[k] = k;
        if (uniform)
            std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return D.lo[x] > D.lo[y]; });
        for (int k = 0; k < K; ++k) D.lvl_order[k] = order[k];
        const uint32_t blo = D.cp_lo_bits >> s;
        for (int lane = 0; lane < NBINS && !obj; ++lane) {
            const uint64_t B = blo + (((uint32_t)lane - blo) & 63u);
            uint64_t top = ((B + 1) << s) - 1;
            if (top > 0x7f7fffffull) top = 0x7f7fffffull;
            float U;
            const uint32_t tb = (uint32_t)top;
            std::memcpy(&U, &tb, 4);
            uint32_t j = 0;
            for (int k = 0; k < K; ++k)
                if (D.lo[k] >= U) ++j;
            D.jtab[lane] = j;
        }
        char* base = dry ? img.data() : h->d_arena;
        D.at = (const float2*)(base + L.at);
        D.atx = N >= 2 ? (const float2*)(base + L.at) + (size_t)(N - 2) * R : (const float2*)(base + L.atx);
        D.aty = (const float2*)(base + L.at) + (size_t)(N - 1) * R;
        D.dem = (const float*)(base + L.dem);
        D.lat = (const float*)(base + L.lat);
        D.a64 = (const double*)(base + L.a64);
        D.lat64 = (const double*)(base + L.lat64);
        D.dem64 = (const double*)(base + L.dem64);
        D.ay_max = 0.0f;
        D.ty_min = INFINITY;
        for (int i = 0; i < pb.radix[N - 1]; ++i) {
            const float2 v = ((const float2*)(img.data() + L.at))[(size_t)(N - 1) * R + i];
            D.ay_max = std::max(D.ay_max, v.x);
            D.ty_min = std::min(D.ty_min, v.y);
        }
        {
            const int ry = std::min(pb.radix[N - 1], 64);
            const float2* ay = (const float2*)(img.data() + L.at) + (size_t)(N - 1) * R;
            std::vector<int> ord(ry);
            for (int i = 0; i < ry; ++i) ord[i] = i;
            std::stable_sort(ord.begin(), ord.end(), [&](int u, int v) { return ay[u].x > ay[v].x; });
            for (int i = 0; i < 64; ++i) D.yord[i] = (uint8_t)(i < ry ? ord[i] : 0);
            // reciprocal factors of y, rounded down with a margin of 2^-22
            // relative (two fp32 roundings, 2^-24 each, plus this fp64 one)
            for (int i = 0; i < 64; ++i) {
                float r = 0.0f;
                if (i < ry && (double)ay[i].x >= 0x1p-20) {
                    const double v = 1.0 / ((double)ay[i].x * (1.0 + 0x1p-22));
                    r = (float)v;
                    if ((double)r > v) r = std::nextafter(r, 0.0f);
                }
                D.yinv[i] = r;
            }
        }
        for (int k = 0; k < KMAX; ++k) {
            float m = INFINITY;
            if (!obj && k < K) {
                const float* ly = (const float*)(img.data() + L.lat) + ((size_t)k * N + (N - 1)) * R;
                for (int i = 0; i < pb.radix[N - 1]; ++i) m = std::min(m, ly[i]);
            }
            D.lymin[k] = m;
        }
        D.demx = N >= 2 ? D.dem + (size_t)(N - 2) * R : (const float*)(base + L.dz);
        D.demy = D.dem + (size_t)(N - 1) * R;
        H.n = N;
        H.k = K;
        H.b = B;
        H.rmax = R;
        H.npre = D.npre;
        H.rx = D.rx;
        H.ry = D.ry;
        H.uniform = uniform;
        H.obj = obj;
        H.has_s2 = D.pre_sinks != 0 || !D.edge_xy;
    }
    if (!dry) {
        e = hipMemcpy(h->d_arena, img.data(), off, hipMemcpyHostToDevice);
        if (e != hipSuccess) return hip_fail(err, e, "hipMemcpy(tables)");
    }
    h->hdesc.assign(descs, descs + n_probs);
    h->jit_state.assign(n_probs, 0);
    h->jit.assign(n_probs, JitRows{});
    return DY_OK;
}

int check_source(const dy_plan* h, const dy_source& s, int idx, std::string* err) {
    if (s.problem < 0 || s.problem >= (int)h->hp.size())
        return fail(err, DY_EINVAL, "source %d: problem %d out of range", idx, s.problem);
    const HostProb& H = h->hp[s.problem];
    if (s.count < 1) return fail(err, DY_EINVAL, "source %d: count must be >= 1", idx);
    if (s.count > kMaxSourcePlans) return fail(err, DY_ELIMIT, "source %d: more than 2^40 plans", idx);
    if (s.kind == DY_SOURCE_RANGE) {
        if (s.begin > UINT64_MAX - s.count)
            return fail(err, DY_EINVAL, "source %d: begin + count overflows", idx);
        if (!H.plans_saturated && s.begin + s.count > H.n_plans)
            return fail(err, DY_EINVAL, "source %d: range exceeds the problem's plan count", idx);
        if (s.begin + s.count - 1 > (uint64_t)INT64_MAX)
            return fail(err, DY_ELIMIT, "source %d: plan index exceeds 2^63-1", idx);
    } else if (s.kind == DY_SOURCE_ROWS) {
        if (!s.rows) return fail(err, DY_EINVAL, "source %d: rows is NULL", idx);
        if (s.row_stride < (uint64_t)H.n) return fail(err, DY_EINVAL, "source %d: row_stride < n_nodes", idx);
        if (s.index_base > (uint64_t)INT64_MAX - (s.count - 1))
            return fail(err, DY_ELIMIT, "source %d: plan index exceeds 2^63-1", idx);
    } else {
        return fail(err, DY_EINVAL, "source %d: unknown kind", idx);
    }
    return DY_OK;
}

JobDev make_job(const dy_plan* h, const dy_source& s) {
    const HostProb& H = h->hp[s.problem];
    JobDev J;
    std::memset(&J, 0, sizeof J);
    J.prob = h->d_probs + s.problem;
    J.kind = s.kind;
    J.begin = s.begin;
    J.count = s.count;
    J.rows = s.rows;
    J.stride = s.row_stride;
    J.index_base = s.index_base;
    J.sample_stride = h->sample_stride;
    J.gblk = 1;
    if (s.kind == DY_SOURCE_RANGE) {
        const uint64_t inner = (uint64_t)H.rx * (uint64_t)H.ry;
        J.blk_first = s.begin / inner;
        const uint64_t blk_last = (s.begin + s.count - 1) / inner;
        J.nblk = blk_last - J.blk_first + 1;
        J.big = (blk_last > 0xffffffffull || s.begin + s.count - 1 > 0xffffffffull) ? 1 : 0;
    }
    return J;
}

}  // namespace

extern "C" {

int32_t dy_abi_version(void) { return DY_ABI_VERSION; }

const char* dy_status_str(int status) {
    switch (status) {
        case DY_OK: return "ok";
        case DY_EINVAL: return "invalid argument";
        case DY_ENOTDAG: return "edges are not in topological order";
        case DY_ELIMIT: return "limit exceeded";
        case DY_ENOMEM: return "out of memory";
        case DY_EDEVICE: return "device error";
        default: return "unknown status";
    }
}

const char* dy_plan_last_error(const dy_plan* h) { return h ? h->err.c_str() : g_create_error.c_str(); }

int dy_plan_create(const dy_problem* probs, int32_t n_probs, int32_t device, dy_plan** out) {
    if (!out) {
        g_create_error = "out is NULL";
        return DY_EINVAL;
    }
    *out = nullptr;
    if (!probs || n_probs < 1) {
        g_create_error = "probs is NULL or n_probs < 1";
        return DY_EINVAL;
    }
    for (int j = 0; j < n_probs; ++j) {
        int st = validate_problem(probs[j], j, &g_create_error);
        if (st != DY_OK) return st;
    }
    int ndev = 0;
    hipError_t e = hipGetDeviceCount(&ndev);
    if (e != hipSuccess || ndev < 1) {
        g_create_error = std::string("no HIP device: ") + hipGetErrorString(e);
        return DY_EDEVICE;
    }
    if (device < 0 || device >= ndev) {
        g_create_error = "device index out of range";
        return DY_EDEVICE;
    }
    DeviceGuard g(device);
    if (!g.ok) {
        g_create_error = "hipSetDevice failed";
        return DY_EDEVICE;
    }
    dy_plan* h = new (std::nothrow) dy_plan();
    if (!h) {
        g_create_error = "host allocation failed";
        return DY_ENOMEM;
    }
    h->device = device;
    if (hipDeviceGetAttribute(&h->cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess || h->cus < 1)
        h->cus = 256;
    int st = stage_problems(h, probs, n_probs, &g_create_error);
    if (st == DY_OK) {
        // host copies of dy_plan_select_static's jobs and results, sized once
        Scratch tmp;
        layout_scratch(tmp, nullptr, kStaticSources, 0, h->kmax);
        h->st_host.assign(2 * (size_t)kStaticSources * sizeof(JobDev) + tmp.res_bytes, 0);
        for (int i = 0; i < 4 && st == DY_OK; ++i)
            if ((e = hipEventCreate(&h->ev[i])) != hipSuccess) st = hip_fail(&g_create_error, e, "hipEventCreate");
        if (st == DY_OK && (e = hipStreamCreateWithFlags(&h->cap_stream, hipStreamNonBlocking)) != hipSuccess)
            st = hip_fail(&g_create_error, e, "hipStreamCreate");
    }
    if (st != DY_OK) {
        dy_plan_destroy(h);
        return st;
    }
    g_create_error.clear();
    *out = h;
    return DY_OK;
}

int dy_kernel_source(const dy_problem* prob, char* buf, uint64_t cap, uint64_t* len) {
    if (!prob || !len || (cap > 0 && !buf)) {
        g_create_error = "prob/len is NULL, or buf is NULL with cap > 0";
        return DY_EINVAL;
    }
    int st = validate_problem(*prob, 0, &g_create_error);
    if (st != DY_OK) return st;
    dy_plan h;
    st = stage_problems(&h, prob, 1, &g_create_error, true);
    if (st != DY_OK) return st;
    const std::string src = jit_rows_source(h.hdesc[0]);
    *len = src.size();
    if (cap > 0) {
        const size_t n = std::min<size_t>(src.size(), (size_t)cap - 1);
        std::memcpy(buf, src.data(), n);
        buf[n] = '\0';
    }
    return DY_OK;
}

void dy_plan_destroy(dy_plan* h) {
    if (!h) return;
    DeviceGuard g(h->device);
    free_scratch(h->sc);
    if (h->d_arena) (void)hipFree(h->d_arena);
    for (int i = 0; i < 4; ++i)
        if (h->ev[i]) (void)hipEventDestroy(h->ev[i]);
    if (h->graph) (void)hipGraphExecDestroy(h->graph);
    if (h->cap_stream) (void)hipStreamDestroy(h->cap_stream);
    delete h;
}

int32_t dy_plan_max_levels(const dy_plan* h) { return h ? h->kmax : 0; }
int32_t dy_plan_num_problems(const dy_plan* h) { return h ? (int32_t)h->hp.size() : 0; }

void drop_graph(dy_plan* h) {
    if (h->graph) (void)hipGraphExecDestroy(h->graph);
    h->graph = nullptr;
}

// Capture what `issue` launches on the plan's capture stream into an
// executable graph; nullptr (and the error state cleared) when that fails.
hipGraphExec_t capture_graph(dy_plan* h,
                             const std::function<void(hipStream_t, const std::function<void(hipError_t, const char*)>&)>&
                                 issue) {
    if (hipStreamBeginCapture(h->cap_stream, hipStreamCaptureModeThreadLocal) != hipSuccess) {
        (void)hipGetLastError();
        return nullptr;
    }
    hipError_t cap_err = hipSuccess;
    issue(h->cap_stream, [&](hipError_t x, const char*) {
        if (x != hipSuccess && cap_err == hipSuccess) cap_err = x;
    });
    hipGraph_t graph = nullptr;
    bool ok = hipStreamEndCapture(h->cap_stream, &graph) == hipSuccess && cap_err == hipSuccess && graph;
    hipGraphExec_t exec = nullptr;
    if (ok) ok = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0) == hipSuccess;
    if (graph) (void)hipGraphDestroy(graph);
    if (!ok) {
        exec = nullptr;
        (void)hipGetLastError();
    }
    return exec;
}

int dy_plan_set_option(dy_plan* h, int32_t option, int64_t value) {
    if (!h) return DY_EINVAL;
    drop_graph(h);
    switch (option) {
        case DY_OPT_GRAPH: h->use_graph = value ? 1 : 0; return DY_OK;
        case DY_OPT_TIMING: h->timing = value ? 1 : 0; return DY_OK;
        case DY_OPT_SAMPLE_STRIDE:
            if (value < 1 || value > (1 << 30)) break;
            h->sample_stride = (uint32_t)value;
            h->stride_fixed = true;
            return DY_OK;
        case DY_OPT_CAND_CAPACITY:
            if (value < 16 || value > (1 << 26)) break;
            h->cand_cap = (uint32_t)value;
            return DY_OK;
        case DY_OPT_FORCE_FP64: h->force_fp64 = value ? 1 : 0; return DY_OK;
        case DY_OPT_CLIMB:
            if (value < 0 || value > 2) {
                h->err = "DY_OPT_CLIMB takes 0, 1 or 2";
                return DY_EINVAL;
            }
            h->use_climb = (int)value;
            return DY_OK;
        case DY_OPT_JIT:
            if (value < 0 || value > 2) {
                h->err = "DY_OPT_JIT takes 0, 1 or 2";
                return DY_EINVAL;
            }
            h->use_jit = (int)value;
            return DY_OK;
        default:
            h->err = "unknown option";
            return DY_EINVAL;
    }
    h->err = "option value out of range";
    return DY_EINVAL;
}

int dy_plan_get_stats(const dy_plan* h, dy_stats* out) {
    if (!h || !out) return DY_EINVAL;
    *out = h->stats;
    return DY_OK;
}

}  // extern "C"

namespace {


// Rows sources run the problem's generated
// kernels (one launch per source; the host copies of the job carry the args).
// Rows [r0, min(r1, count)) of the source for the scan (the sampler takes
// the whole source).
hipError_t launch_jit(const dy_plan* h, const JobDev& J, int problem, bool sample, hipStream_t s, uint64_t r0 = 0,
                      uint64_t r1 = ~0ull) {
    const ProbDev& D = h->hdesc[problem];
    const JitRows& jr = h->jit[problem];
    const ProbDev* dp = h->d_probs + problem;
    unsigned long long rows_stride = J.stride, count = J.count, index_base = J.index_base;
    const unsigned char* rows = J.rows;
    if (!sample) {
        r1 = std::min<uint64_t>(r1, J.count);
        if (r0 >= r1) return hipSuccess;
        rows += r0 * J.stride;
        count = r1 - r0;
        index_base += r0;
    }
    const float2* at = D.at;
    int rmax = D.rmax, bin_shift = D.bin_shift;
    int aligned = ((J.stride | (uint64_t)(uintptr_t)J.rows | (uint64_t)D.n) & 3u) == 0 ? 1 : 0;
    const float* hi = (const float*)((const char*)dp + offsetof(ProbDev, hi));
    const float* lo = (const float*)((const char*)dp + offsetof(ProbDev, lo));
    if (sample) {
        unsigned* scert = J.scert;
        unsigned long long S = J.sample_stride;
        const float* lat = D.lat;
        void* args[] = {&rows, &rows_stride, &count, &at, &rmax, &lo, &lat, &scert, &S, &aligned};
        const unsigned long long nsamp = (count + S - 1) / S;
        // four workgroups per CU: each adds one atomic per level at its end, and
        // those serialise across the device (8 per CU ran 1.6x longer on 2^21 samples)
        const unsigned gx = (unsigned)std::max<unsigned long long>(
            1, std::min<unsigned long long>((nsamp + 255) / 256, 4ull * (unsigned)h->cus));
        return hipModuleLaunchKernel(jr.sample, gx, 1, 1, 256, 1, 1, 0, s, args, nullptr);
    }
    const unsigned* table = J.table;
    const float* thr = J.thr;
    Cand* cand = J.cand;
    unsigned cap = J.cap;
    unsigned* ncand = J.ncand;
    int* flags = J.flags;
    const float* lat = D.lat;
    void* args[] = {&rows, &rows_stride, &count, &index_base, &at, &rmax, &table, &bin_shift, &hi, &thr, &lat,
                    &cand, &cap, &ncand, &flags};
    hipFunction_t fn = aligned ? jr.scan : jr.scan_u;
    int per_cu = 0;
    if (hipModuleOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, 256, 0) != hipSuccess || per_cu < 1)
        per_cu = 4;
    // About 32 rows per thread, between one resident wave of blocks and 16 of
    // them: blocks that start later take the place of those that end, so the
    // last rows of a long source are not left to a few slow waves (a single
    // persistent wave of blocks ran 9% longer on 2^28 rows); below ~32 rows
    // per thread the per-block table staging costs more than it saves.
    const unsigned long long want = (count + 255) / 256;
    const unsigned long long resident = (unsigned long long)per_cu * h->cus;
    const unsigned long long by_rows = (count + 256ull * 32 - 1) / (256ull * 32);
    const unsigned gx = (unsigned)std::min(want, std::max(resident, std::min(by_rows, 16 * resident)));
    return hipModuleLaunchKernel(fn, gx, 1, 1, 256, 1, 1, 0, s, args, nullptr);
}

// The generated seeding pass of job J (problem p), one sample per thread.
hipError_t launch_jit_seed(const dy_plan* h, const JobDev& J, int p, hipStream_t s) {
    const ProbDev& D = h->hdesc[p];
    unsigned long long S = J.sample_stride, units = J.nblk * (unsigned long long)D.rx;
    unsigned long long nsamp = (units + S - 1) / S, blk_first = J.blk_first, begin = J.begin, count = J.count;
    const float2* at = D.at;
    const float2* atx = D.atx;
    const float2* aty = D.aty;
    int rmax = D.rmax;
    const unsigned* jtab = (const unsigned*)((const char*)(h->d_probs + p) + offsetof(ProbDev, jtab));
    unsigned* scert = J.scert;
    void* args[] = {&nsamp, &S, &units, &blk_first, &begin, &count, &at, &atx, &aty, &rmax, &jtab, &scert};
    const unsigned gx = (unsigned)((nsamp + 255) / 256);
    return hipModuleLaunchKernel(h->jit[p].seed, gx, 1, 1, 256, 1, 1, 0, s, args, nullptr);
}

// Seeding pre-pass of the sweep and generic groups (jobs stored in group order at d; host copies at
// hjobs).  Jobs of the generated sweep whose problem has a generated seeding pass take it.
void launch_seed(const dy_plan* h, const JobDev* d, const JobDev* hjobs, const PassPlan& pp, hipStream_t s,
                 const std::function<void(hipError_t, const char*)>& chk) {
    auto chunks = [&](const JobDev* base, int n, auto&& fn) {
        for (int c = 0; c < n; c += 65535) fn(base + c, std::min(65535, n - c));
    };
    for (int g = 0; g < kSweepGroups; ++g) {
        const int lib = pp.n[g] - pp.njit[g];
        auto lib_launch = [&](const JobDev* b, int n) {
            chk(launch_sample_sweep(b, n, (g & 1) != 0, g >= G_OSWEEP, pp.samples[g], pp.npre[g], pp.npre_c[g],
                                    pp.kmax, s),
                "sample");
        };
        if (pp.sample_lib[g] > 0) chunks(d + pp.before(g), lib, lib_launch);
        for (int q = pp.before(g) + lib; q < pp.before(g) + pp.n[g]; ++q) {
            const int p = (int)(hjobs[q].prob - h->d_probs);
            if (h->jit[p].seed)
                chk(launch_jit_seed(h, hjobs[q], p, s), "generated seeding");
            else
                lib_launch(d + q, 1);
        }
    }
    chunks(d + pp.before(G_GENERIC), pp.n[G_GENERIC],
           [&](const JobDev* b, int n) {
               chk(launch_sample_generic(b, n, pp.samples[G_GENERIC], pp.ncol, s), "sample");
           });
}

void launch_table_all(const JobDev* d, int ntot, hipStream_t s,
                      const std::function<void(hipError_t, const char*)>& chk) {
    for (int c = 0; c < ntot; c += 65535)
        chk(launch_table(const_cast<JobDev*>(d + c), std::min(65535, ntot - c), s), "table");
}

// Scoring pass of the sweep and generic groups.
// The generated sweep of one RANGE source (host copy J of its job).
hipError_t launch_jit_sweep(const dy_plan* h, const JobDev& J, int p, hipStream_t s) {
    const ProbDev& D = h->hdesc[p];
    unsigned long long blk_first = J.blk_first, nblk = J.nblk, begin = J.begin, count = J.count;
    const float2* at = D.at;
    const float2* atx = D.atx;
    const float2* aty = D.aty;
    const float* dem = D.dem;
    const float* demx = D.demx;
    const float* demy = D.demy;
    const float* lat = D.lat;
    int rmax = D.rmax;
    const unsigned* table = D.jsh ? J.table2 : J.table;
    const float* thr = J.thr;
    Cand* cand = J.cand;
    unsigned cap = J.cap;
    unsigned* ncand = J.ncand;
    int* flags = J.flags;
    // runs of G blocks per thread that share every prefix digit but the
    // last: G divides the last prefix node's radix, the first block and the
    // block count (every block of a run then lies in the source)
    unsigned G = 1;
    const int last = D.radix[D.npre - 1];
    for (unsigned c : {3u, 2u})
        if (D.obj && last % (int)c == 0 && blk_first % c == 0 && nblk % c == 0) {
            G = c;
            break;
        }
    const unsigned long long units = nblk / G;
    constexpr unsigned long long kMaxBlocks = 1ull << 22;
    for (unsigned long long off = 0; off < units; off += kMaxBlocks * 256ull) {
        unsigned long long unit_off = off;
        const unsigned gx = (unsigned)std::min<unsigned long long>((units - off + 255) / 256, kMaxBlocks);
        void* args[] = {&unit_off, &blk_first, &nblk, &begin, &count, &at, &atx, &aty, &dem, &demx, &demy, &lat,
                        &rmax, &table, &thr, &cand, &cap, &ncand, &flags, &G};
        const hipError_t e = hipModuleLaunchKernel(h->jit[p].sweep, gx, 1, 1, 256, 1, 1, 0, s, args, nullptr);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// Main scoring pass.  hjobs: host copies of the jobs at d (for the sources of
// the sweep groups that run their generated sweep, the last pp.njit[g] of the
// group); null when pp.njit is all zero.
void launch_main(const dy_plan* h, const JobDev* d, const JobDev* hjobs, const PassPlan& pp, hipStream_t s,
                 const std::function<void(hipError_t, const char*)>& chk) {
    auto chunks = [&](const JobDev* base, int n, auto&& fn) {
        for (int c = 0; c < n; c += 65535) fn(base + c, std::min(65535, n - c));
    };
    for (int g = 0; g < kSweepGroups; ++g) {
        chunks(d + pp.before(g), pp.n[g] - pp.njit[g], [&](const JobDev* b, int n) {
            chk(launch_sweep(b, n, (g & 1) != 0, g >= G_OSWEEP, pp.units[g], pp.npre[g], pp.npre_c[g], pp.ry[g],
                             pp.b256[g], pp.rad12[g], pp.pat[g], s),
                "sweep");
        });
        for (int q = pp.before(g) + pp.n[g] - pp.njit[g]; q < pp.before(g) + pp.n[g]; ++q)
            chk(launch_jit_sweep(h, hjobs[q], (int)(hjobs[q].prob - h->d_probs), s), "generated sweep");
    }
    chunks(d + pp.before(G_GENERIC), pp.n[G_GENERIC],
           [&](const JobDev* b, int n) { chk(launch_scan(b, n, pp.units[G_GENERIC], pp.ncol, s), "scan"); });
}

void launch_certify_all(const JobDev* d, int ntot, int cert_waves, const dy_plan* h, hipStream_t s,
                        const std::function<void(hipError_t, const char*)>& chk) {
    for (int c = 0; c < ntot; c += 65535)
        chk(launch_certify(d + c, std::min(65535, ntot - c), cert_waves, h->kmax, h->nmax, h->nrmax, s), "certify");
}

// Per-plan scores of a ROWS source through problem p's generated kernel
// (about eight rows per thread, grid-stride).
hipError_t launch_jit_score(const dy_plan* h, int p, const dy_source& src, float* corr, float* cp, float* dem,
                            uint32_t* feas, hipStream_t s) {
    const ProbDev& D = h->hdesc[p];
    unsigned long long count = src.count, stride = src.row_stride;
    const unsigned char* rows = src.rows;
    int aligned = ((src.row_stride | (uint64_t)(uintptr_t)src.rows | (uint64_t)D.n) & 3u) == 0 ? 1 : 0;
    const float2* at = D.at;
    const float* dm = D.dem;
    int rmax = D.rmax;
    const double* lat64 = D.lat64;
    int vec = (cp && (D.k & 3) == 0 && ((uintptr_t)cp & 15) == 0) ? 1 : 0;
    const unsigned long long want = (count + 256ull * 8 - 1) / (256ull * 8);
    const unsigned gx = (unsigned)std::max<unsigned long long>(1, std::min<unsigned long long>(want, 1ull << 30));
    void* args[] = {&rows, &stride, &count, &aligned, &at, &dm, &rmax, &lat64, &corr, &cp, &dem, &feas, &vec};
    return hipModuleLaunchKernel(h->jit[p].score_rows, gx, 1, 1, 256, 1, 1, 0, s, args, nullptr);
}

// Generated rows kernels for problem p: compiled at first use.
bool jit_ready(dy_plan* h, int p) {
    if (!h->use_jit) return false;
    if (h->jit_state[p] == 0) {
        std::string why;
        h->jit_state[p] = jit_rows_get(h->device, h->hdesc[p], &h->jit[p], &why) ? 1 : -1;
    }
    return h->jit_state[p] == 1;
}

}  // namespace

// First share of a ROWS job scored in two shares (0: one pass).
static uint64_t split_rows(const JobDev& J, const ProbDev& D) {
    if (J.kind != DY_SOURCE_ROWS || D.obj || D.uniform || J.count < kSplitRows) return 0;
    return J.count / kSplitShare;
}

// stat: dy_plan_select_static (per-call device memory in the fixed array, no
// kernel compilation, direct launches, results copied back into the caller's
// array); otherwise dy_plan_select.
static int select_impl(dy_plan* h, const dy_source* src, int32_t n_src, dy_choice* out, void* stream, bool stat) {
    if (!h) return DY_EINVAL;
    if (!src || !out || n_src < 1) {
        h->err = "src/out is NULL or n_src < 1";
        return DY_EINVAL;
    }
    // sources identical to the previous call's passed these checks then
    const bool same_src = !stat && h->call.valid && h->call.src.size() == (size_t)n_src &&
                          std::memcmp(h->call.src.data(), src, (size_t)n_src * sizeof(dy_source)) == 0;
    for (int j = 0; j < n_src && !same_src; ++j) {
        int st = check_source(h, src[j], j, &h->err);
        if (st != DY_OK) return st;
    }
    DeviceGuard guard(h->device);
    if (!guard.ok) {
        h->err = "hipSetDevice failed";
        return DY_EDEVICE;
    }
    hipStream_t s = (hipStream_t)stream;
    // candidate slots per source: the option, bounded by a shared pool
    uint64_t cap = h->cand_cap;
    const uint64_t pool_cap = kCandPoolBytes / sizeof(Cand) / (uint64_t)n_src;
    if (cap > pool_cap) cap = std::max<uint64_t>(pool_cap, 1024);
    Scratch view;
    int st = stat ? static_view(h, (size_t)n_src, (uint32_t)cap, &view) : ensure_scratch(h, (size_t)n_src, (uint32_t)cap);
    if (st != DY_OK) return st;
    Scratch& S = stat ? view : h->sc;
    if (stat) cap = S.cap;
    // generated kernels: compiled at first use, except in calls that may not
    // allocate (loading a module does), which take them only when loaded
    auto jit_use = [&](int p) { return stat ? (h->use_jit && h->jit_state[p] == 1) : jit_ready(h, p); };
    const int km = h->kmax;
    const int cert_waves = n_src <= 64 ? CERT_WAVES : 1;

    // the sources' groups, launch order, jobs and launch plan: derived anew,
    // or the previous call's when this call repeats it (same sources, slots,
    // scratch, options and generated-kernel states)
    CallPlan fresh;
    CallPlan& C = stat ? fresh : h->call;
    const int64_t opts[6] = {h->use_jit, h->use_climb, (int64_t)h->sample_stride, h->stride_fixed ? 1 : 0,
                             h->force_fp64, cert_waves};
    const bool reuse = same_src && C.cap == cap && C.scratch == (const void*)S.scert &&
                       std::memcmp(C.opts, opts, sizeof opts) == 0 && C.jit_state == h->jit_state;
    std::vector<int>& grp = C.grp;
    std::vector<int>& order = C.order;
    std::vector<JobDev>& jobs = C.jobs;
    PassPlan& pp = C.pp;
    // first share of a JIT rows job scored in two shares (0: one pass)
    auto split_at = [&](const JobDev& J) { return split_rows(J, h->hdesc[(int)(J.prob - h->d_probs)]); };
    if (!reuse) {
        C.valid = false;
        grp.assign((size_t)n_src, 0);
        for (int j = 0; j < n_src; ++j) {
            const int p = src[j].problem;
            const HostProb& H = h->hp[p];
            if (src[j].kind == DY_SOURCE_RANGE)
                grp[j] = H.obj ? (H.has_s2 ? G_OSWEEP_S2 : G_OSWEEP) : (H.has_s2 ? G_SWEEP_S2 : G_SWEEP);
            else if (src[j].kind == DY_SOURCE_ROWS && !h->force_fp64 && jit_use(p))
                grp[j] = G_JIT;
            else
                grp[j] = G_GENERIC;
        }
        // RANGE sources of 32-bit plan indices run the sweep generated for their DAG, when the plan has few
        // problems (one compilation each), the source is large enough to repay
        // it (2^24 plans; every source with DY_OPT_JIT 2) and it compiles; they
        // go last in their group, whose library sweep launch covers the others
        std::vector<char> jsw(n_src, 0);
        const uint64_t jit_min = h->use_jit >= 2 ? 1 : (1ull << 24);
        if (h->use_jit && !h->force_fp64 && h->hp.size() <= 8)
            for (int j = 0; j < n_src; ++j) {
                const int p = src[j].problem;
                if (src[j].kind == DY_SOURCE_RANGE && src[j].count >= jit_min &&
                    src[j].begin + src[j].count - 1 <= 0xffffffffull && jit_use(p) && h->jit[p].sweep)
                    jsw[j] = 1;
            }
        // local-search seeds (whole-space RANGE sources of problems of at most
        // kClimbNodes nodes, either objective): in calls of many such sources, where they replace
        // most of the sampling and of the certification work; a call of a few
        // sources waits for the searches' latency instead (tens of microseconds)
        auto climb_ok = [&](int j) {
            const HostProb& H = h->hp[src[j].problem];
            return !h->force_fp64 && H.n <= kClimbNodes && src[j].kind == DY_SOURCE_RANGE &&
                   src[j].begin == 0 && !H.plans_saturated && src[j].count == H.n_plans;
        };
        int n_climb = 0;
        for (int j = 0; j < n_src; ++j) n_climb += climb_ok(j) ? 1 : 0;
        const bool climb = h->use_climb == 2 || (h->use_climb == 1 && n_climb >= kClimbMinSources);
        order.clear();
        order.reserve(n_src);
        for (int g = 0; g < kGroups; ++g)
            for (int pass = 0; pass < 2; ++pass)
                for (int j = 0; j < n_src; ++j)
                    if (grp[j] == g && jsw[j] == pass) order.push_back(j);
        C.plans = 0;
        C.all_units = 0;
        pp = PassPlan();
        jobs.resize((size_t)n_src);
        for (int q = 0; q < n_src; ++q) {
            const int j = order[q];
            const int g = grp[j];
            const HostProb& H = h->hp[src[j].problem];
            JobDev J = make_job(h, src[j]);
            J.cap = (uint32_t)cap;
            J.scert = S.scert + (size_t)q * KMAX * NSLOT;
            J.thr = S.thr + (size_t)q * KMAX;
            J.table = S.table + (size_t)q * NBINS;
            J.table2 = S.table2 + (size_t)q * NBINS2;
            J.cand = S.cand + (size_t)q * cap;
            J.ncand = S.ncand + q;
            J.flags = S.flags + q;
            J.out = S.out + (size_t)j * km;
            if (n_src <= kDirectResults && !stat) {  // few sources: certification writes the host copy directly
                J.hout = (dy_choice*)S.d_hres + (size_t)j * km;
                J.hncand = (uint32_t*)(S.d_hres + S.res_ncand_off) + q;
                J.hflags = (int32_t*)(S.d_hres + S.res_flags_off) + q;
                J.hdone = S.d_done + q;
            }
            J.fb_corr = S.fb_corr + (size_t)q * KMAX;
            J.fb_index = S.fb_index + (size_t)q * KMAX;
            J.cert_waves = cert_waves;
            J.cert_c = S.cert_c + (size_t)q * KMAX * CERT_WAVES;
            J.cert_i = S.cert_i + (size_t)q * KMAX * CERT_WAVES;
            J.cert_cp = S.cert_cp + (size_t)q * KMAX * CERT_WAVES;
            J.cert_d = S.cert_d + (size_t)q * KMAX * CERT_WAVES;
            J.sync = S.sync + q;
            J.fb_levels = h->force_fp64 ? (H.k == 32 ? 0xffffffffu : ((1u << H.k) - 1u)) : 0u;
            J.climb = climb && climb_ok(j) ? 1 : 0;
            int climb_entries = 0;  // the search's table entries (it runs when they fit CLIMB_ENTRIES)
            if (J.climb) {
                for (int n = 0; n < H.n; ++n) climb_entries += h->hdesc[src[j].problem].radix[n];
                pp.climb_e = std::max(pp.climb_e, climb_entries);
                pp.climb_n = std::max(pp.climb_n, H.n);
            }
            // seeding work units: rows of the inner sweep, or plans
            const bool sweep = g < kSweepGroups;
            const uint64_t sunits = sweep ? J.nblk * (uint64_t)H.rx : J.count;
            uint64_t stride = h->sample_stride;
            if (!h->stride_fixed) stride = std::max<uint64_t>(1, std::min<uint64_t>(stride, sunits / kMinSamples));
            // the local search gives each level a seed near its optimum; the
            // sample then only backs it up (about 256 samples per source)
            if (!h->stride_fixed && J.climb) stride = std::max<uint64_t>(stride, std::min<uint64_t>(2048, sunits / 256));
            if (!h->stride_fixed && g == G_JIT && split_rows(J, h->hdesc[src[j].problem]))
                stride = std::max<uint64_t>(stride, std::min<uint64_t>(kSplitStride, sunits / kMinSamples));
            J.sample_stride = (uint32_t)stride;
            J.units = sweep ? J.nblk : J.count;
            ++pp.n[g];
            if (g < kSweepGroups && jsw[j]) ++pp.njit[g];
            if (g < kSweepGroups && jsw[j] && h->hdesc[src[j].problem].jsh != 0 && H.ry >= 1 && H.ry <= 64)
                ++pp.ydiv_jit[g];
            if (g < G_JIT) {
                pp.units[g] = std::max(pp.units[g], J.units);
                pp.samples[g] = std::max(pp.samples[g], (sunits + stride - 1) / stride);
            }
            // a source of more than 2^21 plans whose levels are seeded by the
            // local search needs no sample in corr / SLO mode under uniform
            // pressure (the search starts from the plan of least CP, so a
            // level it cannot seed has no certainly feasible plan at all) and
            // in objective mode (every plan is admissible, so every level's
            // search seeds it); on so large a space a sample of about 256 rows
            // rarely beats the search's seed (on smaller spaces, and under
            // per-backend pressure, it does now and then)
            const bool climb_only = J.climb && (H.obj || H.uniform) && climb_entries <= CLIMB_ENTRIES &&
                                    J.count > (1ull << 21);
            if (g < kSweepGroups && !jsw[j] && !climb_only) ++pp.sample_lib[g];
            pp.kmax = std::max(pp.kmax, H.k);
            if (g == G_GENERIC) pp.ncol = std::max(pp.ncol, H.n);
            if (sweep) {
                if (!jsw[j] && h->hdesc[src[j].problem].jsh != 18) pp.b256[g] = false;
                if (!jsw[j]) {
                    const ProbDev& Dp = h->hdesc[src[j].problem];
                    bool r12 = J.big == 0;
                    for (int n = 0; n < Dp.npre; ++n) r12 = r12 && Dp.radix[n] == 12;
                    if (!r12) pp.rad12[g] = false;
                }
                pp.npre[g] = std::max(pp.npre[g], H.npre);
                pp.pat[g] = std::max(pp.pat[g], H.npre * H.rmax);
                pp.ry[g] = pp.n[g] == 1 ? H.ry : (pp.ry[g] == H.ry ? pp.ry[g] : -1);
                pp.npre_c[g] = pp.n[g] == 1 ? H.npre : (pp.npre_c[g] == H.npre ? pp.npre_c[g] : -1);
            }
            C.all_units = std::max(C.all_units, J.count);
            C.plans += J.count;
            jobs[q] = J;
        }
        C.n3 = pp.before(G_JIT);  // jobs of the other groups; JIT jobs follow
        const int n3 = C.n3;
        // library sweep (both objectives) with a compile-time prefix length: a
        // source whose blocks are aligned runs of G (G dividing the last prefix
        // node's radix, up to 12) gives each thread G blocks that share the
        // prefix but its last node; only in groups of many blocks, so that the
        // fewer threads still fill the device (batch6's 85 M blocks: sweep 1.61
        // -> 1.53 ms with runs of 12, 1.59 with runs of 4)
        for (int g = 0; g < kSweepGroups; ++g) {
            const int npc = pp.npre_c[g];
            if (npc != 2 && npc != 4 && npc != 6 && npc != 8) continue;
            const int q0 = pp.before(g), q1 = pp.before(g) + pp.n[g] - pp.njit[g];
            uint64_t total = 0;
            for (int q = q0; q < q1; ++q) total += jobs[q].nblk;
            if (total < kSweepRunMin) continue;
            uint64_t units = 0;
            for (int q = q0; q < q1; ++q) {
                JobDev& J = jobs[q];
                const int last = h->hdesc[(int)(J.prob - h->d_probs)].radix[npc - 1];
                for (int G : {12, 6, 4, 3, 2})
                    if (last % G == 0 && J.blk_first % (uint64_t)G == 0 && J.nblk % (uint64_t)G == 0) {
                        J.gblk = G;
                        J.units = J.nblk / (uint64_t)G;
                        break;
                    }
                units = std::max(units, J.units);
            }
            pp.units[g] = units;
        }
        // whether any source is scored in two shares, or climbs
        C.any_split = false;
        for (int q = n3; q < n3 + pp.n[G_JIT]; ++q) C.any_split = C.any_split || split_at(jobs[q]) != 0;
        C.any_climb = false;
        // bit 0: a corr / SLO source climbs, bit 1: an objective one; bit 2:
        // every corr / SLO source that climbs is under uniform pressure (its
        // levels can share one search)
        C.climb_modes = 4;
        for (int q = 0; q < n3; ++q)
            if (jobs[q].climb) {
                const ProbDev& Dq = h->hdesc[(int)(jobs[q].prob - h->d_probs)];
                C.any_climb = true;
                C.climb_modes |= Dq.obj ? 2 : 1;
                if (!Dq.obj && !Dq.uniform) C.climb_modes &= ~4;
            }
        C.src.assign(src, src + n_src);
        C.cap = cap;
        C.scratch = (const void*)S.scert;
        std::memcpy(C.opts, opts, sizeof opts);
        C.jit_state = h->jit_state;
        C.valid = !stat;
    }
    const int n3 = C.n3;
    const uint64_t plans = C.plans, all_units = C.all_units;
    const bool any_split = C.any_split, any_climb = C.any_climb;
    const int climb_modes = C.climb_modes;
    // the job array is uploaded only when it changed (a reused plan's jobs are
    // the ones the previous call uploaded)
    const bool changed = stat || S.uploaded != (size_t)n_src ||
                         (!reuse && std::memcmp(S.h_jobs, jobs.data(), (size_t)n_src * sizeof(JobDev)) != 0);
    if (changed) {
        if (!stat) drop_graph(h);
        hipError_t e = hipStreamSynchronize(s);  // a previous upload may still read the pinned buffer
        if (e == hipSuccess) {
            std::memcpy(S.h_jobs, jobs.data(), (size_t)n_src * sizeof(JobDev));
            e = hipMemcpyAsync(S.d_jobs, S.h_jobs, (size_t)n_src * sizeof(JobDev), hipMemcpyHostToDevice, s);
        }
        if (e != hipSuccess) {
            S.uploaded = 0;
            return hip_fail(&h->err, e, "hipMemcpyAsync(jobs)");
        }
        S.uploaded = (size_t)n_src;
    }
    std::function<void(hipError_t, const char*)> chk = [&](hipError_t x, const char* what) {
        if (x != hipSuccess && st == DY_OK) st = hip_fail(&h->err, x, what);
    };
    // share 0: every row; 1: the first share of split sources, every row of
    // the others; 2: the rest of split sources
    auto jit_pass = [&](const JobDev* hjobs, int first, int n, bool sample, hipStream_t st,
                        const std::function<void(hipError_t, const char*)>& ck, int share = 0) {
        for (int q = first; q < first + n; ++q) {
            const int p = (int)(hjobs[q].prob - h->d_probs);
            const uint64_t cut = share ? split_at(hjobs[q]) : 0;
            if (share == 2 && cut == 0) continue;
            const uint64_t r0 = share == 2 ? cut : 0, r1 = share == 1 && cut ? cut : ~0ull;
            ck(launch_jit(h, hjobs[q], p, sample, st, r0, r1), sample ? "rows sample" : "rows scan");
        }
    };
    using Check = std::function<void(hipError_t, const char*)>;
    // seeding and tables; the scoring pass (between timing events); certification and copy-out
    auto issue_pre = [&](hipStream_t st, const Check& ck) {
        launch_seed(h, S.d_jobs, jobs.data(), pp, st, ck);
        if (any_climb)
            for (int c = 0; c < n3; c += 65535)
                ck(launch_climb(S.d_jobs + c, std::min(65535, n3 - c), pp.kmax, climb_modes, pp.climb_e, pp.climb_n,
                                st),
                   "climb");
        jit_pass(jobs.data(), n3, pp.n[G_JIT], true, st, ck);
        launch_table_all(S.d_jobs, n_src, st, ck);
    };
    auto issue_mid = [&](hipStream_t st, const Check& ck) {
        if (h->timing) ck(hipEventRecord(h->ev[1], st), "hipEventRecord");
        launch_main(h, S.d_jobs, jobs.data(), pp, st, ck);
        if (any_split) {
            jit_pass(jobs.data(), n3, pp.n[G_JIT], false, st, ck, 1);
            for (int c = 0; c < pp.n[G_JIT]; c += 65535) {
                const int m = std::min(65535, pp.n[G_JIT] - c);
                ck(launch_seed_cands(S.d_jobs + n3 + c, m, pp.kmax, h->nmax, st), "seed from candidates");
            }
            jit_pass(jobs.data(), n3, pp.n[G_JIT], false, st, ck, 2);
        } else {
            jit_pass(jobs.data(), n3, pp.n[G_JIT], false, st, ck);
        }
        if (h->timing) ck(hipEventRecord(h->ev[2], st), "hipEventRecord");
    };
    auto issue_post = [&](hipStream_t st, const Check& ck) {
        launch_certify_all(S.d_jobs, n_src, cert_waves, h, st, ck);
        if (h->timing) ck(hipEventRecord(h->ev[3], st), "hipEventRecord");
        if (n_src > kDirectResults || stat)
            ck(hipMemcpyAsync(S.h_res, S.out, S.res_bytes, hipMemcpyDeviceToHost, st), "copy out");
    };
    // With the results written straight to host memory, the call waits for the
    // certification's completion words (set after the results, behind a
    // system-scope fence) instead of the stream: they land several
    // microseconds before the stream reports the graph complete.
    const bool poll = !stat && n_src <= kDirectResults && !h->timing && !h->force_fp64;
    if (poll)
        for (int q = 0; q < n_src; ++q) __atomic_store_n(S.h_done + q, 0u, __ATOMIC_RELAXED);
    bool exhausted = h->force_fp64 != 0;
    bool launched = false;
    if (!stat && h->use_graph && !h->timing && !h->force_fp64 && S.clean && !changed) {
        if (!h->graph) {  // capture once; a failure falls back to direct launches for this plan
            h->graph = capture_graph(h, [&](hipStream_t st, const Check& ck) {
                issue_pre(st, ck);
                issue_mid(st, ck);
                issue_post(st, ck);
            });
            if (!h->graph) h->use_graph = 0;
        }
        if (h->graph) {
            S.clean = false;
            chk(hipGraphLaunch(h->graph, s), "hipGraphLaunch");
            launched = true;
        }
    }
    if (!launched) {
        if (h->timing) chk(hipEventRecord(h->ev[0], s), "hipEventRecord");
        // A call that ends with every source certified and no flag raised leaves
        // the scratch clear (the certification's last blocks re-zero the seeds);
        // anything else, or a fresh allocation, clears it here.
        if (!S.clean || h->force_fp64)
            for (int c = 0; c < n_src; c += 65535)
                chk(launch_init(S.d_jobs + c, std::min(65535, n_src - c), s), "init");
        S.clean = false;
        if (!h->force_fp64) {
            issue_pre(s, chk);
            issue_mid(s, chk);
            issue_post(s, chk);
        } else {
            if (h->timing) chk(hipEventRecord(h->ev[1], s), "hipEventRecord");
            for (int c = 0; c < n_src; c += 65535)
                chk(launch_exhaust(S.d_jobs + c, std::min(65535, n_src - c), all_units, s), "exhaust");
            if (h->timing) chk(hipEventRecord(h->ev[2], s), "hipEventRecord");
            if (h->timing) chk(hipEventRecord(h->ev[3], s), "hipEventRecord");
            chk(hipMemcpyAsync(S.h_res, S.out, S.res_bytes, hipMemcpyDeviceToHost, s), "copy out");
        }
    }
    if (poll && st == DY_OK) {
        // the stream is queried every 256 reads, so a failed launch or a
        // fault ends the wait as well
        for (uint32_t it = 1;; ++it) {
            int q = 0;
            while (q < n_src && __atomic_load_n(S.h_done + q, __ATOMIC_ACQUIRE) != 0u) ++q;
            if (q == n_src) break;
            if ((it & 255u) == 0u) {
                const hipError_t qe = hipStreamQuery(s);
                if (qe != hipErrorNotReady) {  // complete (every result visible) or failed
                    chk(qe, "hipStreamQuery");
                    break;
                }
            }
        }
    } else if (st == DY_OK) {
        // poll the stream rather than block on it: a blocking wait returns
        // about 15 microseconds after the work ends here (batch6 step 1.189
        // -> 1.174 ms); hipStreamQuery reports completion or the error
        hipError_t qe;
        while ((qe = hipStreamQuery(s)) == hipErrorNotReady) {
        }
        chk(qe, "hipStreamQuery");
    } else {
        (void)hipStreamSynchronize(s);  // a failed launch: let the work already queued end
    }
    if (st != DY_OK) return st;

    dy_stats stats{};
    stats.plans = plans;
    stats.n_jobs = n_src;
    stats.generated_jobs = pp.n[G_JIT];
    for (int g = 0; g < kSweepGroups; ++g) stats.generated_jobs += pp.njit[g];
    // the library sweep takes the thresholds divided (corr) or lowered
    // (objective) ahead by y's terms for groups on 256 bins with R_y = 12
    for (int g : {(int)G_SWEEP, (int)G_SWEEP_S2, (int)G_OSWEEP, (int)G_OSWEEP_S2})
        stats.ydiv_jobs += pp.ydiv_jit[g] + (pp.b256[g] && pp.ry[g] == 12 ? pp.n[g] - pp.njit[g] : 0);
    if (h->timing) {
        float ms = 0.0f;
        if (hipEventElapsedTime(&ms, h->ev[1], h->ev[2]) == hipSuccess) stats.main_ms = ms;
        if (hipEventElapsedTime(&ms, h->ev[0], h->ev[3]) == hipSuccess) stats.total_ms = ms;
    }
    if (h->force_fp64)
        for (int j = 0; j < n_src; ++j) stats.fallbacks += h->hp[src[j].problem].k;
    int32_t any_flag = 0;  // the union of the sources' flags
    for (int q = 0; q < n_src; ++q) {
        stats.candidates += std::min<uint64_t>(S.h_ncand[q], cap);
        any_flag |= S.h_flags[q];
    }
    if (any_flag & JF_BAD_ROW) {
        h->err = "a row holds an implementation id >= radix of its node";
        return DY_EINVAL;
    }
    // candidate-list overflow: reseed from the gathered candidates and score
    // those sources again (each round raises the thresholds); whatever still
    // overflows after kReseedRounds is decided exhaustively
    constexpr int kReseedRounds = 3;
    for (int round = 0; round <= kReseedRounds && !h->force_fp64 && (any_flag & JF_OVERFLOW); ++round) {
        PassPlan rp;
        std::vector<JobDev> re, ex;
        uint64_t fb_units = 0;
        for (int g = 0; g < kGroups; ++g)
            for (int q = 0; q < n_src; ++q) {
                if (!(S.h_flags[q] & JF_OVERFLOW)) continue;
                const int j = order[q];
                if (grp[j] != g) continue;
                const HostProb& H = h->hp[src[j].problem];
                JobDev J = jobs[q];
                if (g < kSweepGroups) {  // the rescoring sweep takes one block per thread
                    J.gblk = 1;
                    J.units = J.nblk;
                }
                if (round < kReseedRounds) {
                    ++rp.n[g];
                    if (g < G_JIT) rp.units[g] = std::max(rp.units[g], J.units);
                    if (g < kSweepGroups) rp.npre[g] = std::max(rp.npre[g], H.npre);
                    if (g < kSweepGroups) rp.pat[g] = std::max(rp.pat[g], H.npre * H.rmax);
                    if (g < kSweepGroups && h->hdesc[src[j].problem].jsh != 18) rp.b256[g] = false;
                    rp.rad12[g] = false;  // reseeded sources take the general kernel
                    if (g == G_GENERIC) rp.ncol = std::max(rp.ncol, H.n);
                    re.push_back(J);
                } else {
                    J.fb_levels = H.k == 32 ? 0xffffffffu : ((1u << H.k) - 1u);
                    stats.fallbacks += H.k;
                    fb_units = std::max(fb_units, J.count);
                    ex.push_back(J);
                }
            }
        const int n_re = (int)re.size(), n_ex = (int)ex.size();
        if (n_re + n_ex == 0) break;
        std::memcpy(S.h_fb, re.data(), (size_t)n_re * sizeof(JobDev));
        std::memcpy(S.h_fb + n_re, ex.data(), (size_t)n_ex * sizeof(JobDev));
        chk(hipMemcpyAsync(S.d_fb, S.h_fb, (size_t)(n_re + n_ex) * sizeof(JobDev), hipMemcpyHostToDevice, s),
            "copy fb");
        if (n_re > 0) {  // every overflowing source is rescored
            for (int c = 0; c < n_re; c += 65535)
                chk(launch_reseed(S.d_fb + c, std::min(65535, n_re - c), s), "reseed");
            launch_table_all(S.d_fb, n_re, s, chk);
            launch_main(h, S.d_fb, nullptr, rp, s, chk);
            jit_pass(re.data(), rp.before(G_JIT), rp.n[G_JIT], false, s, chk);
            launch_certify_all(S.d_fb, n_re, cert_waves, h, s, chk);
        }
        if (n_ex > 0) {
            exhausted = true;
            const JobDev* b = S.d_fb + n_re;
            for (int c = 0; c < n_ex; c += 65535)
                chk(launch_exhaust(b + c, std::min(65535, n_ex - c), fb_units, s), "exhaust");
        }
        chk(hipMemcpyAsync(S.h_res, S.out, S.res_bytes, hipMemcpyDeviceToHost, s), "copy out");
        chk(hipStreamSynchronize(s), "hipStreamSynchronize");
        if (st != DY_OK) return st;
        if (n_re == 0) break;
        stats.candidates = 0;
        for (int q = 0; q < n_src; ++q) stats.candidates += std::min<uint64_t>(S.h_ncand[q], cap);
    }
    bool all_km = true;
    for (int j = 0; j < n_src && all_km; ++j) all_km = h->hp[src[j].problem].k == km;
    if (all_km) {  // one copy; else columns past a problem's levels stay untouched
        std::memcpy(out, S.h_out, (size_t)n_src * km * sizeof(dy_choice));
    } else {
        for (int j = 0; j < n_src; ++j) {
            const int K = h->hp[src[j].problem].k;
            std::memcpy(out + (size_t)j * km, S.h_out + (size_t)j * km, (size_t)K * sizeof(dy_choice));
        }
    }
    bool flagged = any_flag != 0;  // rescan only when a flag was raised (reseeding may clear it)
    if (flagged) {
        flagged = false;
        for (int q = 0; q < n_src; ++q) flagged = flagged || S.h_flags[q] != 0;
    }
    S.clean = !exhausted && !flagged;
    h->stats = stats;
    return DY_OK;
}

extern "C" {

int dy_plan_select(dy_plan* h, const dy_source* src, int32_t n_src, dy_choice* out, void* stream) {
    return select_impl(h, src, n_src, out, stream, false);
}

int dy_plan_select_static(dy_plan* h, const dy_source* src, int32_t n_src, dy_choice* out, void* stream) {
    return select_impl(h, src, n_src, out, stream, true);
}

int dy_plan_score(dy_plan* h, const dy_source* src, float* corr, float* cp, float* demand, uint32_t* feas_bits,
                  void* stream) {
    if (!h) return DY_EINVAL;
    if (!src) {
        h->err = "src is NULL";
        return DY_EINVAL;
    }
    int st = check_source(h, *src, 0, &h->err);
    if (st != DY_OK) return st;
    DeviceGuard g(h->device);
    if (!g.ok) {
        h->err = "hipSetDevice failed";
        return DY_EDEVICE;
    }
    JobDev J = make_job(h, *src);
    const HostProb& H = h->hp[src->problem];
    const ProbDev& D = h->hdesc[src->problem];
    const bool simple = D.uniform != 0 || D.obj != 0;
    hipError_t e;
    // RANGE sources of 32-bit indices (uniform pressure or the objective) take
    // the library's row kernel (the prefix once per row of y's plans); rows,
    // the problem's generated kernel when it compiles; everything else the
    // generic per-plan kernel
    if (src->kind == DY_SOURCE_ROWS && simple && jit_ready(h, src->problem) && h->jit[src->problem].score_rows)
        e = launch_jit_score(h, src->problem, *src, corr, cp, demand, feas_bits, (hipStream_t)stream);
    else
        e = launch_score(J, src->count, corr, cp, demand, feas_bits, H.n, H.n * H.rmax, H.ry, simple, D.obj != 0,
                         (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(&h->err, e, "score launch");
    return DY_OK;
}

// Host-only self checks of internal helpers (no device call).  Returns the
// number of failures.
int dy_selftest(void) {
    int bad = 0;
    const uint32_t ds[] = {1, 2, 3, 5, 7, 10, 12, 36, 100, 255, 1296, 20736, 46656, 2985984, 60466176,
                           2176782336u, 4294967295u};
    const uint32_t xs[] = {0, 1, 2, 11, 12, 13, 143, 144, 1295, 1296, 20735, 65535, 65536, 2985983,
                           429981695u, 2147483647u, 2147483648u, 4294967294u, 4294967295u};
    for (uint32_t d : ds) {
        Magic g = make_magic(d);
        for (uint32_t x : xs)
            if (magic_div(x, g) != x / d) ++bad;
        uint64_t st = 0x9E3779B97F4A7C15ull;
        for (int i = 0; i < 4096; ++i) {
            st += 0x9E3779B97F4A7C15ull;
            uint32_t x = (uint32_t)(st >> 17);
            if (magic_div(x, g) != x / d) ++bad;
        }
    }
    // directed roundings of the certification bands: the nearest fp32 at or
    // below (above) x, exact values kept
    uint64_t st = 0x243F6A8885A308D3ull;
    for (int i = 0; i < 4096; ++i) {
        st += 0x9E3779B97F4A7C15ull;
        const double x = std::ldexp((double)(st >> 11), -53 + (int)(st % 64) - 20);
        const float dn = round_down(x), up = round_up(x);
        if (!((double)dn <= x && (double)std::nextafter(dn, INFINITY) > x)) ++bad;
        if (!((double)up >= x && (double)std::nextafter(up, -INFINITY) < x)) ++bad;
        const float e = (float)x;
        if (round_down((double)e) != e || round_up((double)e) != e) ++bad;
    }
    return bad;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// suffix recompilation: the residual problem on G[U_t] and the merge
// ---------------------------------------------------------------------------

struct dy_suffix {
    std::vector<int32_t> map;          // residual node -> full node
    std::vector<int32_t> full_radix;
    std::vector<int32_t> edges, radix, backend, is_tool;
    std::vector<float> p, tau, size, w, rho, cost, levels;
    dy_objective obj{};
    dy_problem prob{};
};

extern "C" {

int dy_suffix_create(const dy_problem* full, const uint8_t* committed, dy_suffix** out) {
    if (!out) {
        g_create_error = "out is NULL";
        return DY_EINVAL;
    }
    *out = nullptr;
    if (!full || !committed) {
        g_create_error = "full or committed is NULL";
        return DY_EINVAL;
    }
    std::string err;
    const int st = validate_problem(*full, 0, &err);
    if (st != DY_OK) {
        g_create_error = err;
        return st;
    }
    dy_suffix* S = new (std::nothrow) dy_suffix;
    if (!S) {
        g_create_error = "out of host memory";
        return DY_ENOMEM;
    }
    try {
        const int N = full->n_nodes, R = full->max_radix;
        const bool obj = full->objective != nullptr;
        std::vector<int> rid(N, -1);
        for (int n = 0; n < N; ++n) {
            S->full_radix.push_back(full->radix[n]);
            if (!committed[n]) {
                rid[n] = (int)S->map.size();
                S->map.push_back(n);
            }
        }
        const int M = (int)S->map.size();
        if (M == 0) {
            delete S;
            g_create_error = "every node is committed: nothing to recompile";
            return DY_EINVAL;
        }
        // edges between undispatched nodes; the renumbering keeps u < v
        for (int e = 0; e < full->n_edges; ++e) {
            const int u = rid[full->edges[2 * e]], v = rid[full->edges[2 * e + 1]];
            if (u >= 0 && v >= 0) {
                S->edges.push_back(u);
                S->edges.push_back(v);
            }
        }
        auto rows = [&](const float* t, std::vector<float>& dst) {
            for (int r = 0; r < M; ++r) dst.insert(dst.end(), t + (size_t)S->map[r] * R, t + (size_t)(S->map[r] + 1) * R);
        };
        for (int r = 0; r < M; ++r) {
            S->radix.push_back(full->radix[S->map[r]]);
            S->w.push_back(full->w[S->map[r]]);
        }
        rows(full->p, S->p);
        rows(full->tau, S->tau);
        dy_problem& P = S->prob;
        P.n_nodes = M;
        P.n_edges = (int32_t)(S->edges.size() / 2);
        P.radix = S->radix.data();
        P.max_radix = R;
        P.w = S->w.data();
        if (!obj) {
            rows(full->size, S->size);
            for (int r = 0; r < M; ++r)
                S->backend.insert(S->backend.end(), full->backend + (size_t)S->map[r] * R,
                                  full->backend + (size_t)(S->map[r] + 1) * R);
            S->rho.assign(full->rho, full->rho + (size_t)full->n_levels * full->n_backends);
            P.size = S->size.data();
            P.backend = S->backend.data();
            P.n_levels = full->n_levels;
            P.n_backends = full->n_backends;
            P.rho = S->rho.data();
            P.slo = full->slo;
        } else {
            const dy_objective& o = *full->objective;
            rows(o.cost, S->cost);
            if (o.is_tool)
                for (int r = 0; r < M; ++r) S->is_tool.push_back(o.is_tool[S->map[r]]);
            S->levels.assign(o.levels, o.levels + o.n_levels);
            S->obj = o;
            S->obj.cost = S->cost.data();
            S->obj.is_tool = o.is_tool ? S->is_tool.data() : nullptr;
            S->obj.levels = S->levels.data();
            P.objective = &S->obj;
            P.slo = full->slo;
        }
        P.edges = S->edges.empty() ? nullptr : S->edges.data();
        P.p = S->p.data();
        P.tau = S->tau.data();
    } catch (const std::bad_alloc&) {
        delete S;
        g_create_error = "out of host memory";
        return DY_ENOMEM;
    }
    *out = S;
    return DY_OK;
}

const dy_problem* dy_suffix_problem(const dy_suffix* s) { return s ? &s->prob : nullptr; }

int32_t dy_suffix_nodes(const dy_suffix* s, int32_t* node_map) {
    if (!s) return 0;
    if (node_map)
        for (size_t r = 0; r < s->map.size(); ++r) node_map[r] = s->map[r];
    return (int32_t)s->map.size();
}

int dy_suffix_merge(const dy_suffix* s, const int32_t* committed_impl, int64_t residual_index, int32_t* impl_out,
                    int64_t* full_index) {
    if (!s || !impl_out || residual_index < 0) return DY_EINVAL;
    const int N = (int)s->full_radix.size(), M = (int)s->map.size();
    std::vector<char> free_node(N, 0);
    for (int r = 0; r < M; ++r) free_node[s->map[r]] = 1;
    for (int n = 0; n < N; ++n) {
        if (free_node[n]) continue;
        if (!committed_impl || committed_impl[n] < 0 || committed_impl[n] >= s->full_radix[n]) return DY_EINVAL;
    }
    // decode the residual index (last residual node least significant)
    uint64_t x = (uint64_t)residual_index;
    std::vector<int32_t> suffix(M);
    for (int r = M - 1; r >= 0; --r) {
        const uint64_t rad = (uint64_t)s->radix[r];
        suffix[r] = (int32_t)(x % rad);
        x /= rad;
    }
    if (x != 0) return DY_EINVAL;
    for (int n = 0; n < N; ++n)
        if (!free_node[n]) impl_out[n] = committed_impl[n];
    for (int r = 0; r < M; ++r) impl_out[s->map[r]] = suffix[r];
    if (full_index) {
        unsigned __int128 idx = 0;
        bool over = false;
        for (int n = 0; n < N && !over; ++n) {
            idx = idx * (unsigned)s->full_radix[n] + (unsigned)impl_out[n];
            over = idx > (unsigned __int128)INT64_MAX;
        }
        *full_index = over ? -1 : (int64_t)idx;
    }
    return DY_OK;
}

void dy_suffix_destroy(dy_suffix* s) { delete s; }

}  // extern "C"
