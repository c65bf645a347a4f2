// HIP kernels for gfx950 (CDNA4): scoring workflow physical plans and selecting
// the best SLO-feasible plan per pressure level.
//
// Definitions (per plan, i_n = implementation of node n):
//   corr   = prod_n a_{n,i_n},  a = 1 - w_n (1 - p)    (Sec. 4.1 / 4.3: residual
//            error weighted by vulnerability, kept as a product over nodes)
//   CP_k   = longest path with node durations tau / (1 - rho_{k,b})
//            (Sec. 4.3 "Accounting for parallel branches"; completion time of
//            eq. admission-constraints for fixed assignments)
//   demand = sum_n tau * size  (Sec. 4.4, D_tau annotation)
// Selection per level k: max corr s.t. CP_k <= SLO, ties to the lowest index
// (one selection per level, Algorithm gen).
//
// Objective mode (the paper's additive objective, Sec. 4.3 eq.
// admission-objective with the level weight of Sec. 4.4 eq. variant-objective):
//   J_k = U - lambda_l T - lambda_ld L_k D,  U = sum of LLM utilities u,
//   T = nominal longest path, D = sum of LLM durations;
// max J_k per level, ties to the lowest index.  The same pipeline runs with
// additive per-node terms: a plan is scored by G = U - lambda_l T and D in
// fp32, and the prefilter bins index D (a level's test J_k >= T_k reads
// G >= T_k + m_k D with m_k = lambda_ld L_k >= 0, so a bin's threshold is the
// smallest T_k + m_k D_low over the levels).
//
// Pipeline of one selection call (all on the caller's stream):
//   k_init        zero the per-source scratch
//   k_sample_*    seeding pre-pass: 1 in S work units, per level the best fp32
//                 corr among plans whose fp32 CP is certainly feasible
//   k_table       per level candidate threshold T_k (fp64 error bound on the
//                 seed) and a 64-bin prefilter table indexed by the fp32 CP
//   k_sweep / k_scan   the scoring pass: every plan is scored in fp32; a plan
//                 goes to the candidate list when it could be a level's winner
//   k_certify     fp64 re-evaluation of the candidates; exact winner per level
//                 (the last block of a source merges its waves)
//   k_exhaust*    fallback: exhaustive fp64 decision (candidate overflow)
#include <hip/hip_runtime.h>

#include <math.h>

#include <mutex>

#include "dyplan_internal.h"

namespace dyp {

// Descriptors and tables never change while a kernel runs: reading them
// through the constant address space lets wave-uniform reads become scalar
// loads (and the inner-sweep trip counts stay uniform).
#if defined(__HIP_DEVICE_COMPILE__)
#define CS __attribute__((address_space(4)))
#else
#define CS
#endif
typedef const CS ProbDev* PD;
typedef const CS JobDev* JD;

template <class T>
__device__ __forceinline__ const CS T* cs(const T* p) {
    return (const CS T*)p;
}

// ---------------------------------------------------------------------------
// helpers
// ---------------------------------------------------------------------------

__device__ __forceinline__ uint32_t mdiv(uint32_t x, const CS Magic& g) {
    uint32_t t = __umulhi(g.m, x);
    return (t + ((x - t) >> g.sh1)) >> g.sh2;
}

// Wave-wide max of an unsigned key with DPP row shifts and row broadcasts
// (lane 63 ends with the maximum); the result is read back uniformly.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, false));  // row_shr:1
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, false));  // row_shr:2
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x113, 0xf, 0xf, false));  // row_shr:3
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xe, false));  // row_shr:4
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xc, false));  // row_shr:8
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false));  // row_bcast:15
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false));  // row_bcast:31
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// Candidate threshold from the fp32 corr `s` of a certainly-feasible plan.
// With |corr32 - corr64| <= g corr64 + eta for every plan (g = (2N+1) 2^-24,
// eta = N 2^-148), the exact winner W satisfies corr32_W >= returned value.
__device__ __forceinline__ float cand_threshold(float s, int n) {
    if (!(s >= 0.0f)) return -INFINITY;
    const double g = (2.0 * n + 1.0) * 0x1p-24;
    const double eta = (double)n * 0x1p-148;
    double t = ((double)s - eta) * (1.0 - g) / (1.0 + g) - eta;
    t = t - fabs(t) * 0x1p-48;
    return __double2float_rd(t);
}

// ---- objective mode: keys and thresholds ----------------------------------------

// Order-preserving unsigned key of a float (a greater number has a greater
// key; no number maps to 0, which marks "none").
__device__ __forceinline__ uint32_t fkey(float x) {
    const uint32_t b = __float_as_uint(x);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ float fkey_value(uint32_t k) {
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

__device__ __forceinline__ uint64_t dkey(double x) {
    const uint64_t b = (uint64_t)__double_as_longlong(x);
    return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

// An fp32 value <= a - b (exact real difference): the fp64 difference, lowered
// by more than its rounding error, rounded down.
__device__ __forceinline__ float sub_rd(double a, double b) {
    double x = a - b;
    x = x - (fabs(a) + fabs(b)) * 0x1p-50;
    return __double2float_rd(x);
}

// Candidate threshold of level k from the best estimate s of any plan's J_k:
// every estimate is within err2/2 of the plan's fp64 J_k, so the winner's
// estimate is >= s - err2.
__device__ __forceinline__ float obj_threshold(float s, double err2) {
    return sub_rd((double)s, err2);
}

// Prefilter bin threshold: an fp32 value <= thr + m D_low (exact), m >= 0.
__device__ __forceinline__ float obj_bin_threshold(float thr, double m, float dlow) {
    if (thr == -INFINITY) return -INFINITY;
    const double md = m * (double)dlow;
    double x = (double)thr + md;
    x = x - (fabs((double)thr) + md) * 0x1p-50;
    return __double2float_rd(x);
}

// exact test of the scoring passes: some level's J_k estimate G - m_k D (one
// rounding) reaches its threshold
__device__ __forceinline__ bool is_candidate_obj(PD P, JD J, float G, float D) {
    for (int k = 0; k < P->k; ++k)
        if (fma(-P->m64[k], (double)D, (double)G) >= (double)J->thr[k]) return true;
    return false;
}

// J_k = U - lambda_l T - m_k D in fp64, operation by operation as the definition
// writes it (no contraction into fused multiply-adds).
__device__ __forceinline__ double obj_j(double lam_l, double m, double U, double T, double D) {
#pragma clang fp contract(off)
    double j = lam_l * T;
    j = U - j;
    const double q = m * D;
    return j - q;
}

// ---- fp64 re-evaluation ------------------------------------------------------
// The per-node terms (1 - w(1-p), tau/(1-rho), tau*size) are precomputed on the
// host in fp64 with the same operations as the definition, so the products,
// sums and maxima below reproduce an fp64 evaluation of the definition in
// node order bit for bit.  ids / f are strided per-thread columns.

__device__ double ex_corr(PD P, const uint8_t* ids, int is) {
    const CS double* a = cs(P->a64);
    double c = 1.0;
    for (int n = 0; n < P->n; ++n) c = c * a[n * P->rmax + ids[n * is]];
    return c;
}

__device__ double ex_cp(PD P, const uint8_t* ids, int is, int k, double* f, int fs) {
    const CS double* lat = cs(P->lat64) + (size_t)k * P->n * P->rmax;
    double cp = 0.0;
    for (int n = 0; n < P->n; ++n) {
        double m = 0.0;
        uint32_t pm = P->pred[n];
        while (pm) {
            const int u = __builtin_ctz(pm);
            pm &= pm - 1;
            const double fu = f[u * fs];
            if (fu > m) m = fu;
        }
        const double fn = lat[n * P->rmax + ids[n * is]] + m;
        f[n * fs] = fn;
        if ((P->sinks >> n & 1u) && fn > cp) cp = fn;
    }
    return cp;
}

// Objective mode: U (returned), T and D in fp64, node order (the definition's).
__device__ double ex_obj(PD P, const uint8_t* ids, int is, double* f, int fs, double& T, double& D) {
    const CS double* u64 = cs(P->a64);
    const CS double* d64 = cs(P->dem64);
    const CS double* t64 = cs(P->lat64);
    double U = 0.0, d = 0.0, t = 0.0;
    for (int n = 0; n < P->n; ++n) {
        const int e = n * P->rmax + ids[n * is];
        if (P->llm >> n & 1u) {
            U = U + u64[e];
            d = d + d64[e];
        }
        double m = 0.0;
        uint32_t pm = P->pred[n];
        while (pm) {
            const int u = __builtin_ctz(pm);
            pm &= pm - 1;
            const double fu = f[u * fs];
            if (fu > m) m = fu;
        }
        const double fn = t64[e] + m;
        f[n * fs] = fn;
        if ((P->sinks >> n & 1u) && fn > t) t = fn;
    }
    T = t;
    D = d;
    return U;
}

__device__ double ex_demand(PD P, const uint8_t* ids, int is) {
    const CS double* d64 = cs(P->dem64);
    double d = 0.0;
    for (int n = 0; n < P->n; ++n) d = d + d64[n * P->rmax + ids[n * is]];
    return d;
}

// Implementation ids of plan `index` of the problem (node N-1 least significant).
__device__ void decode64(PD P, uint64_t index, uint8_t* ids, int is) {
    if (index <= 0xffffffffull) {
        uint32_t x = (uint32_t)index;
        for (int n = P->n - 1; n >= 0; --n) {
            const uint32_t q = mdiv(x, P->rmag[n]);
            ids[n * is] = (uint8_t)(x - q * (uint32_t)P->radix[n]);
            x = q;
        }
        return;
    }
    for (int n = P->n - 1; n >= 0; --n) {
        const uint64_t r = (uint64_t)P->radix[n];
        ids[n * is] = (uint8_t)(index % r);
        index /= r;
    }
}

// ids of a candidate or of a fallback unit; returns false for a bad row id
__device__ bool job_ids(JD J, PD P, uint64_t index, uint8_t* ids, int is) {
    if (J->kind == DY_SOURCE_RANGE) {
        decode64(P, index, ids, is);
        return true;
    }
    const uint8_t* row = J->rows + (index - J->index_base) * J->stride;
    const int N = P->n;
    bool ok = true;
    // eight byte loads in flight at a time (a lane otherwise waits on each)
    for (int n0 = 0; n0 < N; n0 += 8) {
        uint8_t v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = n0 + j < N ? row[n0 + j] : (uint8_t)0;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int n = n0 + j;
            if (n < N) {
                uint8_t x = v[j];
                if (x >= (uint32_t)P->radix[n]) {
                    ok = false;
                    x = 0;
                }
                ids[n * is] = x;
            }
        }
    }
    return ok;
}

__device__ __forceinline__ void append_cand(JD J, uint64_t index, float c, float cp) {
    uint32_t slot = atomicAdd(J->ncand, 1u);
    if (slot < J->cap) {
        Cand* d = J->cand + slot;
        d->index = index;
        d->corr = c;
        d->cp = cp;
    } else {
        atomicOr(J->flags, (int32_t)JF_OVERFLOW);
    }
}

// exact per-level candidate test of the scoring pass (levels in P->k)
__device__ __forceinline__ bool is_candidate(PD P, JD J,
                                             float cp, float c) {
    for (int k = 0; k < P->k; ++k)
        if (cp <= P->hi[k] && c >= J->thr[k]) return true;
    return false;
}

// ---------------------------------------------------------------------------
// scratch initialisation
// ---------------------------------------------------------------------------

__global__ void k_init(JobDev* __restrict__ jobs, int njobs) {
    int j = blockIdx.x;
    if (j >= njobs) return;
    JD J = cs(jobs + j);
    int t = threadIdx.x;
    for (int i = t; i < KMAX * NSLOT; i += 64) J->scert[i] = 0u;
    if (t < KMAX) {
        J->thr[t] = -INFINITY;
        J->fb_corr[t] = 0ull;
        J->fb_index[t] = ~0ull;
    }
    if (t < cs(J->prob)->k) {
        dy_choice* o = J->out + t;
        o->index = -1;
        o->feasible = 0;
        o->corr = NAN;
        o->cp = NAN;
        o->demand = NAN;
    }
    if (t < NBINS) J->table[t] = 0u;
    if (t == 0) {
        *J->ncand = 0u;
        *J->flags = 0;
        *J->sync = 0u;
    }
}

// True in the block of a job that finishes a launch last (once every block of
// the job that reaches this point has done so), with the other blocks' global
// writes visible; that block also re-arms the counter.  Called by every thread.
// Every block adds to one device-scope counter, and such atomics serialize
// across the XCDs (tens of ns each): only for launches of few blocks.
__device__ bool last_block(uint32_t* counter, uint32_t expected) {
    __shared__ uint32_t s_last;
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t prev = atomicAdd(counter, 1u);
        s_last = prev + 1u == expected ? 1u : 0u;
        if (s_last) atomicExch(counter, 0u);
    }
    __syncthreads();
    const bool last = s_last != 0u;
    if (last) __threadfence();
    return last;
}

// Per level candidate threshold T_k from the seed slots, and the 64-bin
// prefilter table (and, for problems with a generated sweep, its 256-bin
// table); resets the job's candidate count and flags for the scoring pass.  Called by every thread of one block (>= 64 threads).
// reset: also empty the candidate list and clear the flags (before a scoring
// pass; a rebuild between the shares of a source keeps what the first share
// gathered)
__device__ void build_table(JD J, PD P, bool reset = true) {
    __shared__ float s_thr[KMAX];
    const int lane = threadIdx.x;
    const bool obj = P->obj != 0;
    if (lane < P->k) {
        uint32_t e = 0;
        for (int q = 0; q < NSLOT; ++q) e = max(e, J->scert[lane * NSLOT + q]);
        float t = -INFINITY;
        if (e) t = obj ? obj_threshold(fkey_value(e), P->err2[lane]) : cand_threshold(__uint_as_float(e - 1u), P->n);
        s_thr[lane] = t;
        J->thr[lane] = t;
    }
    __syncthreads();
    if (lane < NBINS) {
        // bin `lane` covers fp32 patterns [B << s, (B+1) << s) with B = lane (mod 64),
        // B in [cp_lo >> s, (cp_lo >> s) + 63]; its threshold is the lowest T_k of
        // every level some CP in the bin may meet.
        const uint32_t s = (uint32_t)P->bin_shift;
        const uint32_t blo = P->cp_lo_bits >> s;
        const uint32_t B = blo + (((uint32_t)lane - blo) & 63u);
        uint32_t lowbits = B << s;
        if (lowbits < P->cp_lo_bits) lowbits = P->cp_lo_bits;
        const float low = __uint_as_float(lowbits);
        float g = INFINITY;
        if (obj) {  // bins of D: a level's bound T_k + m_k D is smallest at the bin's low end
            for (int k = 0; k < P->k; ++k) g = fminf(g, obj_bin_threshold(s_thr[k], P->m64[k], low));
        } else {
            for (int k = 0; k < P->k; ++k)
                if (P->hi[k] >= low) g = fminf(g, s_thr[k]);
        }
        J->table[lane] = __float_as_uint(g);
    }
    if (P->jsh != 0) {
        // the generated sweep's table: bin i of NBINS2 covers fp32 patterns
        // [B << jsh, (B+1) << jsh), B = i (mod NBINS2), B >= cp_lo >> jsh
        // (objective mode: patterns of D, as above)
        const uint32_t s = (uint32_t)P->jsh;
        const uint32_t blo = P->cp_lo_bits >> s;
        for (int i = lane; i < NBINS2; i += blockDim.x) {
            const uint32_t B = blo + (((uint32_t)i - blo) & (uint32_t)(NBINS2 - 1));
            uint32_t lowbits = B << s;
            if (lowbits < P->cp_lo_bits) lowbits = P->cp_lo_bits;
            const float low = __uint_as_float(lowbits);
            float g = INFINITY;
            if (obj) {
                for (int k = 0; k < P->k; ++k) g = fminf(g, obj_bin_threshold(s_thr[k], P->m64[k], low));
            } else {
                for (int k = 0; k < P->k; ++k)
                    if (P->hi[k] >= low) g = fminf(g, s_thr[k]);
            }
            J->table2[i] = __float_as_uint(g);
        }
    }
    if (reset && lane == 0) {
        *J->ncand = 0u;
        *J->flags = 0;
    }
}

// ---------------------------------------------------------------------------
// RANGE sources, uniform pressure: prefix-shared sweep
//
// Work unit = one "block": a fixed assignment of the prefix nodes 0..N-3; the
// inner pair (x = N-2, y = N-1) is swept in lockstep by every lane of a wave,
// so the tables of x and y are wave-uniform (scalar loads) and each plan costs
// a multiply (corr), an add (CP) and a prefilter compare.
// ---------------------------------------------------------------------------

// pc: product of the prefix factors (objective mode: sum of the prefix
// utilities); px, py: longest prefix path into x and into y; s: longest prefix
// path ending at a prefix sink; pd: objective mode, sum of the prefix d terms.
struct Prefix {
    float pc, px, py, s, pd;
};

// The (a, tau) rows of the prefix nodes (objective mode: (u, tau) and d),
// staged in LDS by the workgroup when they fit (a random LDS read instead of
// a global load in the decode chain).
constexpr int PAT_MAX = 1024;  // entries

template <bool OBJ>
__device__ __forceinline__ const float2* stage_prefix_rows(PD P, float2* s_pat, float* s_pd, int cap = PAT_MAX) {
    const int n = P->npre * P->rmax;
    const bool fit = n <= cap;
    if (fit)
        for (int i = threadIdx.x; i < n; i += WG) {
            s_pat[i] = cs(P->at)[i];
            if (OBJ) s_pd[i] = cs(P->dem)[i];
        }
    __syncthreads();
    return fit ? s_pat : nullptr;
}

// Digit of prefix node n in block index b (node 0 most significant).
__device__ __forceinline__ uint32_t prefix_digit(PD P, int n, uint64_t b, int big) {
    if (!big) {
        const uint32_t q = P->pv_big[n] ? 0u : mdiv((uint32_t)b, P->pvmag[n]);
        return q - mdiv(q, P->rmag[n]) * (uint32_t)P->radix[n];
    }
    return (uint32_t)((b / P->pv64[n]) % (uint64_t)P->radix[n]);
}

// Prefix recurrence of block b.  NPRE > 0: the prefix has exactly NPRE nodes
// (checked by the host); the loops unroll, every descriptor load is issued up
// front and the f_n live in registers (predecessor bits are wave-uniform, so
// each test is a scalar branch).  NPRE == 0: any length, f_n in an LDS column.
// RAD > 0: every prefix node has RAD implementations and block indices fit
// 32 bits (checked by the host), so the digits come from successive divisions
// by the constant RAD.
template <int NPRE, bool OBJ, int RAD = 0>
__device__ __forceinline__ Prefix prefix_eval(PD P, uint64_t b, int big, float* __restrict__ s_f,
                                              const float2* s_pat, const float* s_pd) {
    if constexpr (NPRE > 0) {
        const int rmax = P->rmax;
        float f[NPRE];
        float pc = OBJ ? 0.0f : 1.0f, pd = 0.0f;
        uint32_t dg[NPRE];
        if constexpr (RAD > 0) {
            uint32_t x = (uint32_t)b;
#pragma unroll
            for (int n = NPRE - 1; n >= 0; --n) {
                dg[n] = x % (uint32_t)RAD;
                x /= (uint32_t)RAD;
            }
        }
#pragma unroll
        for (int n = 0; n < NPRE; ++n) {
            const uint32_t d = RAD > 0 ? dg[n] : prefix_digit(P, n, b, big);
            const float2 v = s_pat ? s_pat[n * rmax + d] : cs(P->at)[n * rmax + d];
            if (OBJ) {
                pc = pc + v.x;
                pd = pd + (s_pat ? s_pd[n * rmax + d] : cs(P->dem)[n * rmax + d]);
            } else {
                pc = pc * v.x;
            }
            float m = 0.0f;
            const uint32_t pm = P->pred[n];
#pragma unroll
            for (int u = 0; u < n; ++u)
                if (pm >> u & 1u) m = fmaxf(m, f[u]);
            f[n] = v.y + m;
        }
        float px = 0.0f, py = 0.0f, s = 0.0f;
        const int xn = P->xnode;
        const uint32_t pmx = xn >= 0 ? P->pred[xn] : 0u;
        const uint32_t pmy = P->pred[P->ynode] & (xn >= 0 ? ~(1u << xn) : ~0u);
        const uint32_t pms = P->pre_sinks;
#pragma unroll
        for (int u = 0; u < NPRE; ++u) {
            if (pmx >> u & 1u) px = fmaxf(px, f[u]);
            if (pmy >> u & 1u) py = fmaxf(py, f[u]);
            if (pms >> u & 1u) s = fmaxf(s, f[u]);
        }
        return Prefix{pc, px, py, s, pd};
    }
    const int tid = threadIdx.x;
    const int npre = P->npre;
    float pc = OBJ ? 0.0f : 1.0f, pd = 0.0f;
    for (int n = 0; n < npre; ++n) {
        const uint32_t d = prefix_digit(P, n, b, big);
        const float2 v = s_pat ? s_pat[n * P->rmax + d] : cs(P->at)[n * P->rmax + d];
        if (OBJ) {
            pc = pc + v.x;
            pd = pd + (s_pat ? s_pd[n * P->rmax + d] : cs(P->dem)[n * P->rmax + d]);
        } else {
            pc = pc * v.x;
        }
        float m = 0.0f;
        uint32_t pm = P->pred[n];
        while (pm) {
            int u = __builtin_ctz(pm);
            pm &= pm - 1;
            m = fmaxf(m, s_f[u * WG + tid]);
        }
        s_f[n * WG + tid] = v.y + m;
    }
    float px = 0.0f, py = 0.0f, s = 0.0f;
    if (P->xnode >= 0) {
        uint32_t pm = P->pred[P->xnode];
        while (pm) {
            int u = __builtin_ctz(pm);
            pm &= pm - 1;
            px = fmaxf(px, s_f[u * WG + tid]);
        }
    }
    {
        uint32_t pm = P->pred[P->ynode];
        if (P->xnode >= 0) pm &= ~(1u << P->xnode);
        while (pm) {
            int u = __builtin_ctz(pm);
            pm &= pm - 1;
            py = fmaxf(py, s_f[u * WG + tid]);
        }
    }
    {
        uint32_t pm = P->pre_sinks;
        while (pm) {
            int u = __builtin_ctz(pm);
            pm &= pm - 1;
            s = fmaxf(s, s_f[u * WG + tid]);
        }
    }
    return Prefix{pc, px, py, s, pd};
}

// Prefix of a run of blocks b0 .. b0 + G - 1 that differ only in the last
// prefix node's digit (b0 a multiple of G, G dividing that node's radix, so
// the digits never carry): the nodes before the last are evaluated once by
// prefix_head, the last one per block by prefix_tail.  Same operations in
// the same order as prefix_eval, so the same values: the product takes the
// last node's factor last, and the maxima are exact.
struct PrefixHead {
    float pc;      // product of the factors of nodes 0 .. NPRE-2 (objective mode: sum of u)
    float pd;      // objective mode: sum of d over nodes 0 .. NPRE-2
    float m;       // the last node's predecessor maximum
    float px, py, s;  // the maxima into x, into y and over the prefix sinks, nodes 0 .. NPRE-2
    uint32_t d;    // the last node's digit in b0
};

template <int NPRE, bool OBJ, int RAD>
__device__ __forceinline__ PrefixHead prefix_head(PD P, uint64_t b0, int big, const float2* s_pat, const float* s_pd) {
    static_assert(NPRE > 1, "a head and a last node");
    const int rmax = P->rmax;
    float f[NPRE - 1];
    float pc = OBJ ? 0.0f : 1.0f, pd = 0.0f;
    uint32_t dg[NPRE];
    if constexpr (RAD > 0) {
        uint32_t x = (uint32_t)b0;
#pragma unroll
        for (int n = NPRE - 1; n >= 0; --n) {
            dg[n] = x % (uint32_t)RAD;
            x /= (uint32_t)RAD;
        }
    } else {
#pragma unroll
        for (int n = 0; n < NPRE; ++n) dg[n] = prefix_digit(P, n, b0, big);
    }
#pragma unroll
    for (int n = 0; n < NPRE - 1; ++n) {
        const float2 v = s_pat ? s_pat[n * rmax + dg[n]] : cs(P->at)[n * rmax + dg[n]];
        if (OBJ) {
            pc = pc + v.x;
            pd = pd + (s_pat ? s_pd[n * rmax + dg[n]] : cs(P->dem)[n * rmax + dg[n]]);
        } else {
            pc = pc * v.x;
        }
        float m = 0.0f;
        const uint32_t pm = P->pred[n];
#pragma unroll
        for (int u = 0; u < n; ++u)
            if (pm >> u & 1u) m = fmaxf(m, f[u]);
        f[n] = v.y + m;
    }
    float m = 0.0f, px = 0.0f, py = 0.0f, s = 0.0f;
    const uint32_t pml = P->pred[NPRE - 1];
    const int xn = P->xnode;
    const uint32_t pmx = xn >= 0 ? P->pred[xn] : 0u;
    const uint32_t pmy = P->pred[P->ynode] & (xn >= 0 ? ~(1u << xn) : ~0u);
    const uint32_t pms = P->pre_sinks;
#pragma unroll
    for (int u = 0; u < NPRE - 1; ++u) {
        if (pml >> u & 1u) m = fmaxf(m, f[u]);
        if (pmx >> u & 1u) px = fmaxf(px, f[u]);
        if (pmy >> u & 1u) py = fmaxf(py, f[u]);
        if (pms >> u & 1u) s = fmaxf(s, f[u]);
    }
    return PrefixHead{pc, pd, m, px, py, s, dg[NPRE - 1]};
}

template <int NPRE, bool OBJ>
__device__ __forceinline__ Prefix prefix_tail(PD P, const PrefixHead& h, int g, const float2* s_pat,
                                              const float* s_pd) {
    constexpr int n = NPRE - 1;
    const int e = n * P->rmax + (int)(h.d + (uint32_t)g);
    const float2 v = s_pat ? s_pat[e] : cs(P->at)[e];
    const float fl = v.y + h.m;
    const int xn = P->xnode;
    const bool inx = xn >= 0 && (P->pred[xn] >> n & 1u);
    const bool iny = (P->pred[P->ynode] >> n & 1u) && n != xn;
    const bool ins = P->pre_sinks >> n & 1u;
    const float pc = OBJ ? h.pc + v.x : h.pc * v.x;
    const float pd = OBJ ? h.pd + (s_pat ? s_pd[e] : cs(P->dem)[e]) : 0.0f;
    return Prefix{pc, inx ? fmaxf(h.px, fl) : h.px, iny ? fmaxf(h.py, fl) : h.py, ins ? fmaxf(h.s, fl) : h.s, pd};
}

// One plan of the inner sweep: corr = cx * a_y, CP = max(tau_y + M, S2); the
// prefilter threshold of CP's bin is read from the 64-entry LDS table (a
// random LDS read issues in about half the time of a lane permute on gfx950):
// byte offset = ((bits(CP) >> bin_shift) & 63) * 4, two shift/and operations.
// B256: the 256-bin table on shift 18 instead, whose byte offset
// (bits(CP) >> 16) & 0x3fc is one AND of the pattern's upper half-word.
template <bool HAS_S2, bool B256 = false>
__device__ __forceinline__ uint64_t sweep_test(const float2 vy, float M, float S2, float cx, uint32_t sh,
                                               const float* s_bins) {
    float cp = vy.y + M;
    if (HAS_S2) cp = fmaxf(cp, S2);
    const float cc = cx * vy.x;
    const uint32_t off = B256 ? (__float_as_uint(cp) >> 16) & 0x3fcu : (__float_as_uint(cp) >> sh) & 0xfcu;
    const float thr = *(const float*)((const char*)s_bins + off);
    return __ballot(cc >= thr);
}

// Threshold on the rest of the product for implementation j of y (r_j =
// P->yinv[j]): whenever fp32(c a_j) >= T, c >= the value returned.  For T >
// 2^-60, fp32(c a_j) >= T gives c a_j >= T / (1 + 2^-24) (both normal), and
// fp32(T r_j) <= T r_j (1 + 2^-24) <= T / (a_j (1 + 2^-24)) since r_j <= 1 /
// (a_j (1 + 2^-22)); smaller T, and r_j = 0 (a_j < 2^-20), give 0, which
// every c >= 0 meets; T = +inf (no level in the bin) stays +inf.
__device__ __forceinline__ float ydiv_threshold(float T, float r) {
    if (T == INFINITY) return T;
    return T > 0x1p-60f ? T * r : 0.0f;
}

// One plan of the inner sweep with the thresholds of y's implementation
// pre-divided (s_t: its 256 bins): CP = max(tau_y + M, S2) picks the bin, whose
// threshold on cx (the rest of the product) is returned as its fp32 pattern.
// Every such threshold is +0, positive or +inf, so the patterns order as the
// values do: the row's test is cx >= the least of its plans' thresholds (no
// per-plan product or compare).  A plan that the product test admits is
// admitted here; the rare path scores the admitted rows exactly.
template <bool HAS_S2>
__device__ __forceinline__ uint32_t sweep_thr_ydiv(float ty, float M, float S2, const float* s_t) {
    float cp = ty + M;
    if (HAS_S2) cp = fmaxf(cp, S2);
    const uint32_t off = (__float_as_uint(cp) >> 16) & 0x3fcu;
    return *(const uint32_t*)((const char*)s_t + off);
}

// Per-backend pressure (not uniform): the level-k state of a row of the
// sweep, for the exact per-level tests of the seeding pass and of the rare
// path.  `dg` holds the prefix digits of the block.  NPRE > 0: the prefix has
// exactly NPRE nodes, the recurrence is unrolled with every f_n in a register;
// NPRE == 0: any length, f_n in the thread's LDS column s_f.  Returns M (the
// path into y other than through y's own duration) and S2 (the longest path
// ending at another sink), as the sweep forms them at level 0.
template <int NPRE>
__device__ void level_row(PD P, const CS float* lat, const uint32_t* dg, uint64_t b, int big, int ix,
                          float* __restrict__ s_f, float& M, float& S2) {
    const int R = P->rmax, xn = P->xnode;
    const uint32_t pmx = xn >= 0 ? P->pred[xn] : 0u;
    const uint32_t pmy = P->pred[P->ynode] & (xn >= 0 ? ~(1u << xn) : ~0u);
    float px = 0.0f, py = 0.0f, s = 0.0f;
    if constexpr (NPRE > 0) {
        float f[NPRE];
#pragma unroll
        for (int n = 0; n < NPRE; ++n) {
            float m = 0.0f;
            const uint32_t pm = P->pred[n];
#pragma unroll
            for (int u = 0; u < n; ++u)
                if (pm >> u & 1u) m = fmaxf(m, f[u]);
            f[n] = lat[n * R + dg[n]] + m;
        }
#pragma unroll
        for (int u = 0; u < NPRE; ++u) {
            if (pmx >> u & 1u) px = fmaxf(px, f[u]);
            if (pmy >> u & 1u) py = fmaxf(py, f[u]);
            if (P->pre_sinks >> u & 1u) s = fmaxf(s, f[u]);
        }
    } else {
        const int tid = threadIdx.x;
        for (int n = 0; n < P->npre; ++n) {
            const uint32_t d = prefix_digit(P, n, b, big);
            float m = 0.0f;
            uint32_t pm = P->pred[n];
            while (pm) {
                const int u = __builtin_ctz(pm);
                pm &= pm - 1;
                m = fmaxf(m, s_f[u * WG + tid]);
            }
            s_f[n * WG + tid] = lat[n * R + d] + m;
        }
        auto pmax = [&](uint32_t pm) {
            float v = 0.0f;
            while (pm) {
                const int u = __builtin_ctz(pm);
                pm &= pm - 1;
                v = fmaxf(v, s_f[u * WG + tid]);
            }
            return v;
        };
        px = pmax(pmx);
        py = pmax(pmy);
        s = pmax(P->pre_sinks);
    }
    const float fx = (xn >= 0 ? lat[xn * R + ix] : 0.0f) + px;
    const bool exy = P->edge_xy != 0;
    M = exy ? fmaxf(py, fx) : py;
    S2 = exy ? s : fmaxf(s, fx);
}

template <int NPRE>
__device__ __forceinline__ void prefix_digits(PD P, uint64_t b, int big, uint32_t* dg) {
    if constexpr (NPRE > 0) {
#pragma unroll
        for (int n = 0; n < NPRE; ++n) dg[n] = prefix_digit(P, n, b, big);
    }
}

// Rare path of the sweep under per-backend pressure: every plan of this
// lane's row that some level admits exactly in fp32 (CP_k <= ghi and corr >=
// T_k) goes to the candidate list once (with its unpressured CP, the value the
// bands of the list refer to).  A level is skipped when no plan of the row
// can reach its threshold (cx times the largest factor of y) or its band on
// the unpressured CP (the row's smallest unpressured CP).  R_y > 64 may list
// a plan once per level.
template <bool HAS_S2, int NPRE>
__device__ void general_row(PD P, JD J, uint64_t b, int big, int ix, float cx, float M0, float S20,
                            float* __restrict__ s_f) {
    const int N = P->n, R = P->rmax, ry = P->ry;
    const uint64_t base = (b * (uint64_t)P->rx + (uint64_t)ix) * (uint64_t)ry;
    const CS float2* aty = cs(P->aty);
    uint32_t dg[NPRE > 0 ? NPRE : 1];
    prefix_digits<NPRE>(P, b, big, dg);
    const float cmax = cx * P->ay_max;
    float cp0_lb = P->ty_min + M0;
    if (HAS_S2) cp0_lb = fmaxf(cp0_lb, S20);
    uint64_t done = 0;
    for (int k = 0; k < P->k; ++k) {
        const float thr = J->thr[k];
        if (!(cmax >= thr && cp0_lb <= P->hi[k])) continue;
        const CS float* lat = cs(P->lat) + (size_t)k * N * R;
        float M, S2;
        level_row<NPRE>(P, lat, dg, b, big, ix, s_f, M, S2);
        const CS float* laty = lat + P->ynode * R;
        if (P->lymin[k] + M > P->ghi || (HAS_S2 && S2 > P->ghi)) continue;  // every CP_k of the row above
        if (ry <= 64) {
            // y by decreasing factor: corr falls along the loop, which stops
            // at the first plan below the level's threshold
            for (int jj = 0; jj < ry; ++jj) {
                const int iy = P->yord[jj];
                const float2 vy = aty[iy];
                const float cc = cx * vy.x;
                if (!(cc >= thr)) break;
                if (done >> iy & 1ull) continue;
                float cp = laty[iy] + M;
                if (HAS_S2) cp = fmaxf(cp, S2);
                const uint64_t idx = base + (uint64_t)iy;
                if (cp <= P->ghi && idx - J->begin < J->count) {
                    float cp0 = vy.y + M0;
                    if (HAS_S2) cp0 = fmaxf(cp0, S20);
                    append_cand(J, idx, cc, cp0);
                    done |= 1ull << iy;
                }
            }
            continue;
        }
        for (int iy = 0; iy < ry; ++iy) {
            if (ry <= 64 && (done >> iy & 1ull)) continue;
            float cp = laty[iy] + M;
            if (HAS_S2) cp = fmaxf(cp, S2);
            const float2 vy = aty[iy];
            const float cc = cx * vy.x;
            const uint64_t idx = base + (uint64_t)iy;
            if (cp <= P->ghi && cc >= thr && idx - J->begin < J->count) {
                float cp0 = vy.y + M0;
                if (HAS_S2) cp0 = fmaxf(cp0, S20);
                append_cand(J, idx, cc, cp0);
                if (ry <= 64) done |= 1ull << iy;
            }
        }
    }
}

// RY > 0: every source of the launch has R_y = RY; the y table is loaded once
// per workgroup into scalar registers and the y loop is fully unrolled, so the
// inner sweep issues no memory load and no wait other than its LDS bin reads.
// B256: every source of the launch has the 256-bin table (P->jsh = 18); with
// RY > 0 the table is held per implementation of y, pre-divided by its factor
// (s_bins[j][256], sweep_test_ydiv).
// RAD > 0: every prefix node of every source has RAD implementations and the
// block indices fit 32 bits (constant-divisor digits).
// The inner sweep of block b (the prefix pf evaluated): every (x, y) pair,
// the prefilter per plan, the exact test in the rare path.
// Rare path of the sweep: a lane whose row (x = ix) of block b passed the
// prefilter (mine) re-scores it with the exact test.
template <bool HAS_S2, int NPRE>
__device__ __forceinline__ void sweep_rare(PD P, JD J, uint64_t b, bool live, int ix, float cx, float M, float S2,
                                           bool mine, float* s_f) {
    if (!(live && mine)) return;
    if (!P->uniform) {
        general_row<HAS_S2, NPRE>(P, J, b, J->big, ix, cx, M, S2, s_f);
        return;
    }
    const CS float2* aty = cs(P->aty);
    const int ry = P->ry;
    const uint64_t base = (b * (uint64_t)P->rx + (uint64_t)ix) * (uint64_t)ry;
    for (int iy = 0; iy < ry; ++iy) {
        const float2 vy = aty[iy];
        float cp = vy.y + M;
        if (HAS_S2) cp = fmaxf(cp, S2);
        const float cc = cx * vy.x;
        const uint64_t idx = base + (uint64_t)iy;
        if (idx - J->begin < J->count && is_candidate(P, J, cp, cc)) append_cand(J, idx, cc, cp);
    }
}

// A row of the sweep that passed the prefilter, parked in its wave's LDS
// queue until the queue fills (or the wave's work ends), when every lane of
// the wave re-scores one parked row: the exact test then runs on the whole
// wave at once instead of stalling it for a single lane.
struct RareRow {
    uint64_t b;      // block
    uint32_t ix;     // implementation of x
    float cx, M, S2;
};
constexpr int RQ = 64;  // parked rows per wave

template <bool HAS_S2, int NPRE>
__device__ __forceinline__ void flush_rare(PD P, JD J, const RareRow* q, uint32_t n, float* s_f) {
    const uint32_t lane = threadIdx.x & 63;
    if (lane < n) {
        const RareRow e = q[lane];
        sweep_rare<HAS_S2, NPRE>(P, J, e.b, true, (int)e.ix, e.cx, e.M, e.S2, true, s_f);
    }
}

// The row's least pre-divided threshold (see sweep_thr_ydiv).
template <bool HAS_S2, int RY>
__device__ __forceinline__ uint32_t sweep_row_ydiv(const float2 (&vyr)[RY], float M, float S2, const float* s_bins) {
    uint32_t m = sweep_thr_ydiv<HAS_S2>(vyr[0].y, M, S2, s_bins);
#pragma unroll
    for (int j = 1; j < RY; ++j) m = min(m, sweep_thr_ydiv<HAS_S2>(vyr[j].y, M, S2, s_bins + j * NBINS2));
    return m;
}

// q, qn, live_mask: the wave's queue of parked rows (B256 with RY > 0 only;
// qn is wave-uniform) and the ballot of its live lanes.
template <bool HAS_S2, int RY, int NPRE, bool B256>
__device__ __forceinline__ void sweep_block(PD P, JD J, uint64_t b, bool live, const Prefix& pf,
                                            const float2 (&vyr)[RY > 0 ? RY : 1], const float* s_bins,
                                            float* s_f, RareRow* q, uint32_t& qn, uint64_t live_mask) {
    const uint32_t sh = (uint32_t)P->bin_shift - 2u;
    const CS float2* atx = cs(P->atx);
    const CS float2* aty = cs(P->aty);
    const int rx = P->rx, ry = P->ry;
    // without a second sink x is no sink, so it feeds y
    const bool exy = !HAS_S2 || P->edge_xy != 0;
    if constexpr (B256 && RY > 0) {
        for (int ix = 0; ix < rx; ++ix) {
            const float2 vx = atx[ix];
            const float fx = vx.y + pf.px;
            const float cx = pf.pc * vx.x;
            const float M = exy ? fmaxf(pf.py, fx) : pf.py;
            const float S2 = exy ? pf.s : fmaxf(pf.s, fx);
            const uint64_t hit =
                __ballot(cx >= __uint_as_float(sweep_row_ydiv<HAS_S2, RY>(vyr, M, S2, s_bins))) & live_mask;
            if (hit) {
                const uint32_t nh = (uint32_t)__popcll(hit);
                if (qn + nh > (uint32_t)RQ) {
                    flush_rare<HAS_S2, NPRE>(P, J, q, qn, s_f);
                    qn = 0;
                }
                const uint32_t lane = threadIdx.x & 63;
                if (hit >> lane & 1ull) {
                    const uint32_t o = qn + __builtin_amdgcn_mbcnt_hi((uint32_t)(hit >> 32),
                                                                      __builtin_amdgcn_mbcnt_lo((uint32_t)hit, 0u));
                    q[o] = RareRow{b, (uint32_t)ix, cx, M, S2};
                }
                qn += nh;
            }
        }
        return;
    }
    for (int ix = 0; ix < rx; ++ix) {
        const float2 vx = atx[ix];
        const float fx = vx.y + pf.px;
        const float cx = pf.pc * vx.x;
        const float M = exy ? fmaxf(pf.py, fx) : pf.py;
        const float S2 = exy ? pf.s : fmaxf(pf.s, fx);
        uint64_t hit = 0;
        int iy = 0;
        if (RY > 0) {
#pragma unroll
            for (int j = 0; j < (RY > 0 ? RY : 1); ++j) hit |= sweep_test<HAS_S2, B256>(vyr[j], M, S2, cx, sh, s_bins);
            iy = ry;
        }
        for (; iy + 4 <= ry; iy += 4) {
            const float2 v0 = aty[iy], v1 = aty[iy + 1], v2 = aty[iy + 2], v3 = aty[iy + 3];
            hit |= sweep_test<HAS_S2, B256>(v0, M, S2, cx, sh, s_bins);
            hit |= sweep_test<HAS_S2, B256>(v1, M, S2, cx, sh, s_bins);
            hit |= sweep_test<HAS_S2, B256>(v2, M, S2, cx, sh, s_bins);
            hit |= sweep_test<HAS_S2, B256>(v3, M, S2, cx, sh, s_bins);
        }
        for (; iy < ry; ++iy) hit |= sweep_test<HAS_S2, B256>(aty[iy], M, S2, cx, sh, s_bins);
        if (hit) sweep_rare<HAS_S2, NPRE>(P, J, b, live, ix, cx, M, S2, (hit >> (threadIdx.x & 63)) & 1ull, s_f);
    }
}

// Work unit = J->gblk consecutive blocks per thread (J->units of them per
// source): with a compile-time prefix length (NPRE > 0) the host may give a
// source whose blocks are aligned runs of G (G dividing the last prefix
// node's radix) G blocks per thread, which share the prefix but its last node
// (prefix_head once, prefix_tail per block); NPRE == 0 takes one block per
// thread.
template <bool HAS_S2, int RY, int NPRE, bool B256, int RAD>
__global__ void __launch_bounds__(WG) k_sweep(const JobDev* __restrict__ jobs, uint64_t unit_off, int pat_cap) {
    extern __shared__ float s_f[];
    JD J = cs(jobs + blockIdx.y);
    PD P = cs(J->prob);
    const uint64_t units = J->units;
    const int G = NPRE > 0 ? J->gblk : 1;
    const uint64_t t0 = unit_off + (uint64_t)blockIdx.x * WG;
    if (t0 >= units) return;
    const uint64_t t = t0 + threadIdx.x;
    const bool live = t < units;
    const uint64_t b0 = J->blk_first + (live ? t : units - 1) * (uint64_t)G;
    constexpr bool YDIV = B256 && RY > 0;
    __shared__ float s_bins[YDIV ? (RY > 0 ? RY : 1) * NBINS2 : (B256 ? NBINS2 : NBINS)];
    if (B256) {
        static_assert(!B256 || NBINS2 == WG, "one bin per thread");
        const float thr = __uint_as_float(J->table2[threadIdx.x]);
        if constexpr (YDIV) {
#pragma unroll
            for (int j = 0; j < (RY > 0 ? RY : 1); ++j)
                s_bins[j * NBINS2 + threadIdx.x] = ydiv_threshold(thr, P->yinv[j]);
        } else {
            s_bins[threadIdx.x] = thr;
        }
    } else if (threadIdx.x < NBINS) {
        s_bins[threadIdx.x] = __uint_as_float(J->table[threadIdx.x]);
    }
    // dynamic LDS: one f_n column per prefix node and thread (NPRE == 0
    // only), then the prefix nodes' rows (pat_cap entries)
    float2* s_pat = (float2*)(s_f + (NPRE > 0 ? (size_t)0 : (size_t)max(P->npre, 1) * WG));
    const float2* pat = stage_prefix_rows<false>(P, s_pat, nullptr, pat_cap);
    // a wave whose lanes all lie past the last unit has nothing to score (no
    // barrier follows)
    if (t0 + (threadIdx.x & ~63u) >= units) return;
    float2 vyr[RY > 0 ? RY : 1];
    if (RY > 0) {
        const CS float2* aty = cs(P->aty);
#pragma unroll
        for (int iy = 0; iy < RY; ++iy) {
            vyr[iy] = aty[iy];
            if constexpr (YDIV) {
                // only the durations are read in the loop; keep them in
                // scalar registers (a reload per row would wait on the LDS
                // reads too, both counting on lgkmcnt)
                uint32_t v = __float_as_uint(vyr[iy].y);
                asm volatile("" : "+s"(v));
                vyr[iy].y = __uint_as_float(v);
            }
        }
    }
    __shared__ RareRow s_q[YDIV ? WG / 64 : 1][RQ];
    RareRow* q = s_q[YDIV ? threadIdx.x >> 6 : 0];
    uint32_t qn = 0;
    const uint64_t live_mask = __ballot(live);
    if constexpr (NPRE > 0) {
        const PrefixHead ph = prefix_head<NPRE, false, RAD>(P, b0, J->big, pat, nullptr);
        for (int g = 0; g < G; ++g)
            sweep_block<HAS_S2, RY, NPRE, B256>(P, J, b0 + (uint64_t)g, live, prefix_tail<NPRE, false>(P, ph, g, pat, nullptr),
                                                vyr, s_bins, s_f, q, qn, live_mask);
    } else {
        const Prefix pf = prefix_eval<NPRE, false, RAD>(P, b0, J->big, s_f, pat, nullptr);
        sweep_block<HAS_S2, RY, NPRE, B256>(P, J, b0, live, pf, vyr, s_bins, s_f, q, qn, live_mask);
    }
    if (YDIV && qn) flush_rare<HAS_S2, NPRE>(P, J, q, qn, s_f);
}

// Work unit of sample j: one unit of the window [j S, min((j+1) S, n)), at a
// hashed offset.  A fixed offset would alias with the mixed-radix digits (a
// stride sharing factors with the radices visits only some implementation ids
// of the low-order prefix nodes).
__device__ __forceinline__ uint64_t sample_unit(uint64_t j, uint64_t S, uint64_t n) {
    const uint64_t start = j * S;
    const uint32_t width = (uint32_t)min(S, n - start);
    const uint32_t h = (uint32_t)(j * 0x9E3779B1ull) >> 16;
    return start + (uint64_t)(h % width);
}

// Seeding pre-pass of the sweep: work unit = one row (block, x-implementation)
// of R_y plans; one hashed row per window of S rows.  Per level, the best fp32
// corr among sampled plans whose fp32 CP is certainly feasible.  A plan's CP
// bin gives (jtab, staged in LDS) how many levels, in
// order of decreasing band, it certainly meets; the plan updates one bucket,
// and a suffix maximum over buckets gives every level's value.  Reduction:
// DPP within the wave, LDS across the workgroup, then an atomic max on the
// ordered bit pattern into one of NSLOT slots per level.
template <bool HAS_S2, int NPRE>
__global__ void __launch_bounds__(WG) k_sample_sweep(const JobDev* __restrict__ jobs) {
    extern __shared__ float s_dyn[];
    __shared__ uint32_t s_red[KMAX][WG / 64];
    JD J = cs(jobs + blockIdx.y);
    PD P = cs(J->prob);
    const int K = P->k;
    float* s_f = s_dyn;                                  // prefix recurrence, [npre][WG]
    float* s_b = s_dyn + (size_t)max(P->npre, 1) * WG;   // buckets, [K][WG]
    float2* s_pat = (float2*)(s_b + (size_t)K * WG);     // prefix rows, PAT_MAX entries
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint64_t S = J->sample_stride;
    const int rx = P->rx, ry = P->ry;
    const uint64_t units = J->nblk * (uint64_t)rx;
    const uint64_t nsamp = (units + S - 1) / S;
    const uint64_t t0 = (uint64_t)blockIdx.x * WG;
    if (t0 >= nsamp) return;
    const uint64_t t = t0 + tid;
    const bool live = t < nsamp;
    const uint64_t u = sample_unit(live ? t : nsamp - 1, S, units);
    uint64_t b;
    int ix;
    if (units <= 0xffffffffull && P->xnode >= 0) {  // 32-bit split by the invariant divisor
        const uint32_t q = mdiv((uint32_t)u, P->rmag[P->xnode]);
        b = J->blk_first + q;
        ix = (int)((uint32_t)u - q * (uint32_t)rx);
    } else {
        b = J->blk_first + u / (uint64_t)rx;
        ix = (int)(u % (uint64_t)rx);
    }
    const float2* pat = stage_prefix_rows<false>(P, s_pat, nullptr);
    const Prefix pf = prefix_eval<NPRE, false>(P, b, J->big, s_f, pat, nullptr);
    for (int j = 0; j < K; ++j) s_b[j * WG + tid] = -1.0f;
    const float2 vx = cs(P->atx)[ix];
    const float fx = vx.y + pf.px;
    const float cx = pf.pc * vx.x;
    const bool exy = P->edge_xy != 0;
    const float M = exy ? fmaxf(pf.py, fx) : pf.py;
    const float S2 = exy ? pf.s : fmaxf(pf.s, fx);
    const uint64_t base = (b * (uint64_t)rx + (uint64_t)ix) * (uint64_t)ry;
    __shared__ int s_jt[NBINS];
    if (tid < NBINS) s_jt[tid] = (int)P->jtab[tid];
    __syncthreads();
    const uint32_t sh = (uint32_t)P->bin_shift - 2u;
    const CS float2* aty = cs(P->aty);
    if (!P->uniform) {
        // per-backend pressure: each level's exact fp32 CP_k; certainly
        // feasible when CP_k <= glo (level k writes bucket k, no suffix maximum)
        uint32_t dg[NPRE > 0 ? NPRE : 1];
        prefix_digits<NPRE>(P, b, J->big, dg);
        for (int k = 0; k < K; ++k) {
            const CS float* lat = cs(P->lat) + (size_t)k * P->n * P->rmax;
            float Mk, S2k;
            level_row<NPRE>(P, lat, dg, b, J->big, ix, s_f, Mk, S2k);
            const CS float* laty = lat + P->ynode * P->rmax;
            float best = -1.0f;
            // no plan of the row is certainly feasible when y's fastest
            // implementation (or the other sinks) already misses the band
            if (P->lymin[k] + Mk > P->glo || (HAS_S2 && S2k > P->glo)) {
            } else if (ry <= 64) {
                // y by decreasing factor: the first plan certainly feasible
                // (and in the range) has the row's best corr at this level
                for (int jj = 0; jj < ry; ++jj) {
                    const int iy = P->yord[jj];
                    float cp = laty[iy] + Mk;
                    if (HAS_S2) cp = fmaxf(cp, S2k);
                    if (cp <= P->glo && live && (base + (uint64_t)iy - J->begin < J->count)) {
                        best = cx * aty[iy].x;
                        break;
                    }
                }
            } else {
                for (int iy = 0; iy < ry; ++iy) {
                    float cp = laty[iy] + Mk;
                    if (HAS_S2) cp = fmaxf(cp, S2k);
                    if (cp <= P->glo && live && (base + (uint64_t)iy - J->begin < J->count))
                        best = fmaxf(best, cx * aty[iy].x);
                }
            }
            const uint32_t e = wave_max_u32(best >= 0.0f ? __float_as_uint(best) + 1u : 0u);
            if (lane == 0) s_red[k][wave] = e;
        }
        __syncthreads();
        if (tid < K) {
            uint32_t e = 0;
            for (int w = 0; w < WG / 64; ++w) e = max(e, s_red[tid][w]);
            if (e) atomicMax(J->scert + tid * NSLOT + (blockIdx.x % NSLOT), e);
        }
        return;
    }
    for (int iy = 0; iy < ry; ++iy) {
        const float2 vy = aty[iy];
        float cp = vy.y + M;
        if (HAS_S2) cp = fmaxf(cp, S2);
        const float cc = cx * vy.x;
        const int j = *(const int*)((const char*)s_jt + ((__float_as_uint(cp) >> sh) & 0xfcu));
        if (j > 0 && live && (base + (uint64_t)iy - J->begin < J->count)) {
            float* q = s_b + (j - 1) * WG + tid;
            *q = fmaxf(*q, cc);
        }
    }
    float run = -1.0f;
    for (int i = K - 1; i >= 0; --i) {
        run = fmaxf(run, s_b[i * WG + tid]);
        const uint32_t e = wave_max_u32(run >= 0.0f ? __float_as_uint(run) + 1u : 0u);
        if (lane == 0) s_red[i][wave] = e;
    }
    __syncthreads();
    if (tid < K) {
        uint32_t e = 0;
        for (int w = 0; w < WG / 64; ++w) e = max(e, s_red[tid][w]);
        if (e) atomicMax(J->scert + P->lvl_order[tid] * NSLOT + (blockIdx.x % NSLOT), e);
    }
}

// ---------------------------------------------------------------------------
// Local-search seeds (RANGE sources that cover their problem's whole plan
// space)
//
// Any certainly-feasible plan gives a valid candidate threshold through its
// fp32 corr, exactly as a sampled plan does, and the nearer that corr is to
// the level's optimum, the fewer plans pass the prefilter and reach fp64
// certification.  Under the additive objective every plan is admissible and
// any plan's fp32 estimate of J_k (computed as the sweep computes it) gives a
// valid threshold; the search then climbs that estimate from the plan that
// gives every node its best entry by u - lambda_l tau - lambda_ld L_k d.  One wave per (source, level) climbs: it starts at the plan
// that gives every node its fastest implementation at the level (the least
// CP of all plans: the longest path is monotone in every duration, in fp32
// too) and, while some plan that differs from the current one in one node --
// or, once no such plan helps, in two nodes -- is certainly feasible and has
// a greater fp32 corr, moves to the best of them (greatest corr, then first in
// move order).  Every move raises corr, so the walk ends; a step limit bounds
// it anyway.  The result only raises a seed slot: the selection is unchanged,
// only the work that reaches it shrinks.
// ---------------------------------------------------------------------------
constexpr int CLIMB_STEPS = 64;          // moves per (source, level) at most
constexpr uint32_t CLIMB_PAIRS = 16384;  // two-node moves per pass at most (else single moves only)
constexpr int CLIMB_NODES = 8;           // problems of at most this many nodes climb (the plan sits in registers)

// Wave-wide maximum of a 64-bit key, every lane active: the greatest high
// word, then the greatest low word among the lanes holding it, each through
// the DPP reduction (lane permutes through the LDS crossbar took several
// times as long per round).
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
    const uint32_t hi = wave_max_u32((uint32_t)(v >> 32));
    const uint32_t lo = wave_max_u32((uint32_t)(v >> 32) == hi ? (uint32_t)v : 0u);
    return (uint64_t)hi << 32 | lo;
}

// fp32 corr (node-order product) and CP of the plan whose node n has factor
// a[n] and duration t[n], except node n1 (a1, t1) and node n2 (a2, t2).  NN
// >= N is a compile-time bound, so every array stays in registers; the
// predecessor masks are wave-uniform.
template <int NN>
__device__ __forceinline__ void climb_eval(PD P, int N, const float (&a)[NN], const float (&t)[NN], int n1, float a1,
                                           float t1, int n2, float a2, float t2, float& c, float& cp) {
    float f[NN];
    c = 1.0f;
    cp = 0.0f;
#pragma unroll
    for (int n = 0; n < NN; ++n) {
        f[n] = 0.0f;
        if (n < N) {
            const float an = n == n1 ? a1 : (n == n2 ? a2 : a[n]);
            const float tn = n == n1 ? t1 : (n == n2 ? t2 : t[n]);
            c = c * an;
            float m = 0.0f;
            const uint32_t pm = P->pred[n];
#pragma unroll
            for (int u = 0; u < n; ++u)
                if (pm >> u & 1u) m = fmaxf(m, f[u]);
            f[n] = tn + m;
            if (P->sinks >> n & 1u) cp = fmaxf(cp, f[n]);
        }
    }
}

// Objective mode: the fp32 estimate of J_k of the same plan, in the sweep's
// operations and order: U and D summed in node order, T the longest path,
// G = fma(-lambda_l, T, U), estimate = fma(-m_k, D, G).
template <int NN>
__device__ __forceinline__ float climb_est(PD P, int N, const float (&u)[NN], const float (&t)[NN],
                                           const float (&d)[NN], int n1, float u1, float t1, float d1, int n2,
                                           float u2, float t2, float d2, float m) {
    float f[NN];
    float U = 0.0f, D = 0.0f, T = 0.0f;
#pragma unroll
    for (int n = 0; n < NN; ++n) {
        f[n] = 0.0f;
        if (n < N) {
            const float un = n == n1 ? u1 : (n == n2 ? u2 : u[n]);
            const float tn = n == n1 ? t1 : (n == n2 ? t2 : t[n]);
            const float dn = n == n1 ? d1 : (n == n2 ? d2 : d[n]);
            U = U + un;
            D = D + dn;
            float mx = 0.0f;
            const uint32_t pm = P->pred[n];
#pragma unroll
            for (int v = 0; v < n; ++v)
                if (pm >> v & 1u) mx = fmaxf(mx, f[v]);
            f[n] = tn + mx;
            if (P->sinks >> n & 1u) T = fmaxf(T, f[n]);
        }
    }
    return fmaf(-m, D, fmaf(-P->lam_l, T, U));
}

// One wave per (source, level): grid (levels, sources), 64 threads.  The
// current plan is held by every lane in registers; each lane evaluates a
// share of the moves, a wave reduction picks the best.  Moves only use each
// node's Pareto-optimal implementations at the level (no other has both a
// factor at least as high and a duration at least as short): an optimal
// plan needs no other, since trading a dominated one for its dominator keeps
// the plan feasible and its corr as high.
// The block has blockDim.x = 64 W threads (W waves): few (source, level)
// pairs take W = 16, so that each move pass is one short round (the pass is
// latency-bound), many take W = 1.
// Bytes of one search's LDS tables for E entries: a, tau (and d in objective
// mode) as fp32, the kept entries as int16, node and kept flag as bytes.
__host__ __device__ constexpr size_t climb_slot_bytes(int E, bool obj) {
    return ((size_t)E * (4 + 4 + (obj ? 4 : 0) + 2 + 1 + 1) + 7) & ~(size_t)7;
}

// Wave-level sync of a packed search (its wave is alone in its tables), or
// the block's barrier when the block's waves share one search.
__device__ __forceinline__ void climb_sync(bool pack) {
    if (pack) {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    } else {
        __syncthreads();
    }
}

// Launch shapes: blockDim.x = 256 packs four searches per block, one per
// wave, search blockIdx.x * 4 + wave = (source, level) in source-major order
// (nsearch searches in all); blockDim.x = 1024 gives one search, source
// blockIdx.y and level blockIdx.x, to all 16 waves.  E: entries of the
// largest table set (the sum of a problem's radices) of the launch, at most
// CLIMB_ENTRIES; dynamic LDS holds climb_slot_bytes(E) per search.
template <int NN, bool OBJ, bool CHAIN = false>
__global__ void __launch_bounds__(1024) k_climb(const JobDev* __restrict__ jobs, int nsearch, int kmax, int E) {
    extern __shared__ uint64_t s_climb_dyn[];
    __shared__ int32_t s_pn[4][NN * (NN - 1) / 2 + 1];  // pair p = (n1, n2): n1 * NMAX + n2
    __shared__ int32_t s_po[4][NN * (NN - 1) / 2 + 1];  // first move of pair p (flat pair-move order)
    __shared__ uint64_t s_red[16];
    const bool pack = blockDim.x == 256;
    // the wave's slot, wave-uniform (scalar), so that its tables' addresses are too
    const int slot = pack ? __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)) : 0;
    int ji = blockIdx.y, k = blockIdx.x;
    if (pack) {
        const int q = (int)blockIdx.x * 4 + slot;
        if (q >= nsearch) return;
        ji = CHAIN ? q : q / kmax;
        k = CHAIN ? 0 : q % kmax;
    }
    // this search's tables: node tables (entry off[n] + i), node of entry e,
    // entry e is Pareto-optimal at the level, the kept entries node by node
    char* tb = (char*)s_climb_dyn + (size_t)slot * climb_slot_bytes(E, OBJ);
    float* s_a = (float*)tb;
    float* s_t = s_a + E;
    float* s_d = s_t + (OBJ ? E : 0);  // objective mode: d
    int16_t* s_fe = (int16_t*)(s_t + E + (OBJ ? E : 0));
    uint8_t* s_node = (uint8_t*)(s_fe + E);
    uint8_t* s_keep = s_node + E;
    int32_t* s_pnv = s_pn[slot];
    int32_t* s_pov = s_po[slot];
    JD J = cs(jobs + ji);
    if (!J->climb) return;
    PD P = cs(J->prob);
    const int N = P->n, R = P->rmax, lane = threadIdx.x & 63;
    const int tid = pack ? lane : (int)threadIdx.x, nt = pack ? 64 : (int)blockDim.x;
    if ((P->obj != 0) != OBJ || N > NN) return;
    const bool uni = OBJ || P->uniform != 0;
    const CS float2* at = cs(P->at);
    int off[NN + 1];
    int tot = 0;
#pragma unroll
    for (int n = 0; n < NN; ++n) {
        off[n] = tot;
        if (n < N) tot += P->radix[n];
    }
    off[NN] = tot;
    if (tot > E) return;
    // CHAIN: the wave climbs every level of its source in turn.  Under
    // uniform pressure the levels share the tables, their Pareto sets and the
    // start, and are taken from the tightest band to the loosest, each from
    // the plan the previous one reached (feasible at any looser band too); in
    // objective mode the tables and Pareto sets do not depend on the level
    // either and every plan is admissible, so each level starts from the
    // plan the previous one reached; otherwise each level is set up and
    // started afresh.
    const bool chain = CHAIN && (OBJ || P->uniform != 0);
    const int nlev = CHAIN ? P->k : 1;
    const int ksel = k;
    int foff[NN + 1];
    int ftot = 0;
    int cur[NN];
    float ca[NN], ct[NN], cd[NN];
    bool pairs_ok = false;
    const int npairs = N * (N - 1) / 2;
    // move keys order by the value: corr bits (non-negative), or the
    // order-preserving key of the estimate
    auto vkey = [&](float v) -> uint32_t { return OBJ ? fkey(v) : __float_as_uint(v); };
    auto block_max = [&](uint64_t v) {
        v = wave_max_u64(v);
        if (nt == 64) return v;
        if (lane == 0) s_red[tid >> 6] = v;
        climb_sync(pack);
        uint64_t b = 0;
        for (int w = 0; w < (nt >> 6); ++w) b = s_red[w] > b ? s_red[w] : b;
        climb_sync(pack);
        return b;
    };
    for (int li = 0; li < nlev; ++li) {
    const int k = CHAIN ? (chain ? P->lvl_order[P->k - 1 - li] : li) : ksel;
    if (k >= P->k) continue;
    // objective mode: a greater u and a smaller tau and d never lower J_k
    // only when lambda_l and lambda_ld L_k are not negative
    const float mk = OBJ ? P->m32[k] : 0.0f;
    if (OBJ && (!(P->lam_l >= 0.0f) || !(mk >= 0.0f))) continue;
    // durations the band is tested on: the unpressured ones against lo_k
    // (uniform pressure), else the level's own against the exact band
    const CS float* lt = uni ? nullptr : cs(P->lat) + (size_t)k * N * R;
    const float band = uni ? P->lo[k] : P->glo;
    if (li == 0 || !chain) {
    for (int n = 0; n < N; ++n)
        for (int i = tid; i < P->radix[n]; i += nt) {
            const float2 v = at[n * R + i];
            s_a[off[n] + i] = v.x;
            s_t[off[n] + i] = uni ? v.y : lt[n * R + i];
            if (OBJ) s_d[off[n] + i] = cs(P->dem)[n * R + i];
            s_node[off[n] + i] = (uint8_t)n;
        }
    climb_sync(pack);
    for (int e = tid; e < tot; e += nt) {
        const int n = s_node[e];
        int lo = 0, hi = 0;
#pragma unroll
        for (int m = 0; m < NN; ++m)
            if (m == n) {
                lo = off[m];
                hi = off[m + 1];
            }
        const float a = s_a[e], t = s_t[e], d = OBJ ? s_d[e] : 0.0f;
        bool keep = true;
        for (int q = lo; q < hi && keep; ++q) {
            const float a2 = s_a[q], t2 = s_t[q], d2 = OBJ ? s_d[q] : 0.0f;
            if (q != e && a2 >= a && t2 <= t && d2 <= d && (a2 > a || t2 < t || d2 < d || q < e)) keep = false;
        }
        s_keep[e] = keep ? 1 : 0;
    }
    climb_sync(pack);
    // compact the kept entries per node (ballot and prefix count)
    ftot = 0;
#pragma unroll
    for (int n = 0; n < NN; ++n) {
        foff[n] = ftot;
        if (n < N)
            for (int c0 = off[n]; c0 < off[n + 1]; c0 += 64) {
                const int e = c0 + lane;
                const bool kp = e < off[n + 1] && s_keep[e];
                const uint64_t m = __ballot(kp);
                const int pos = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
                if (kp && tid < 64) s_fe[ftot + pos] = (int16_t)e;
                ftot += __popcll(m);
            }
    }
    foff[NN] = ftot;
    climb_sync(pack);
    // start: every node's fastest kept implementation (the fastest of all);
    // objective mode: every node's best kept entry by u - lambda_l tau - m_k d
#pragma unroll
    for (int n = 0; n < NN; ++n) {
        cur[n] = 0;
        ca[n] = OBJ ? 0.0f : 1.0f;
        ct[n] = 0.0f;
        cd[n] = 0.0f;
        if (n < N) {
            float best = OBJ ? -INFINITY : INFINITY;
            for (int f = foff[n]; f < foff[n + 1]; ++f) {
                const int e = s_fe[f];
                const float sc = OBJ ? s_a[e] - P->lam_l * s_t[e] - mk * s_d[e] : s_t[e];
                if (OBJ ? sc > best : sc < best) {
                    best = sc;
                    cur[n] = e - off[n];
                }
            }
            ca[n] = s_a[off[n] + cur[n]];
            ct[n] = s_t[off[n] + cur[n]];
            if (OBJ) cd[n] = s_d[off[n] + cur[n]];
        }
    }
    uint32_t pairs = 0;
#pragma unroll
    for (int n = 0; n < NN; ++n)
        if (n < N) pairs += (uint32_t)(foff[n + 1] - foff[n]) * (uint32_t)(ftot - foff[n + 1]);
    pairs_ok = pairs <= CLIMB_PAIRS;
    if (tid == 0) {  // pairs in (n1, n2) order and where their moves start
        int p = 0, o = 0;
        for (int n1 = 0; n1 < N; ++n1)
            for (int n2 = n1 + 1; n2 < N; ++n2) {
                int F1 = 0, F2 = 0;
#pragma unroll
                for (int m = 0; m < NN; ++m) {
                    if (m == n1) F1 = foff[m + 1] - foff[m];
                    if (m == n2) F2 = foff[m + 1] - foff[m];
                }
                s_pnv[p] = n1 * NMAX + n2;
                s_pov[p] = o;
                o += F1 * F2;
                ++p;
            }
        s_pov[p] = o;
    }
    climb_sync(pack);
    }  // set-up of the level
    float cc, ccp = 0.0f;
    if (OBJ) {
        cc = climb_est<NN>(P, N, ca, ct, cd, -1, 0.0f, 0.0f, 0.0f, -1, 0.0f, 0.0f, 0.0f, mk);
    } else {
        climb_eval<NN>(P, N, ca, ct, -1, 0.0f, 0.0f, -1, 0.0f, 0.0f, cc, ccp);
        if (!(ccp <= band)) continue;  // no plan is certainly feasible at this level
    }
    for (int step = 0; step < CLIMB_STEPS; ++step) {
        // single moves over the kept entries; key = (corr bits, reversed move order), 0 = none
        uint64_t best = 0;
        for (int f = tid; f < ftot; f += nt) {
            const int e = s_fe[f], n = s_node[e];
            int cn = 0, on = 0;
#pragma unroll
            for (int m = 0; m < NN; ++m)
                if (m == n) {
                    cn = cur[m];
                    on = off[m];
                }
            if (e - on == cn) continue;
            float c, cp = 0.0f;
            if (OBJ)
                c = climb_est<NN>(P, N, ca, ct, cd, n, s_a[e], s_t[e], s_d[e], -1, 0.0f, 0.0f, 0.0f, mk);
            else
                climb_eval<NN>(P, N, ca, ct, n, s_a[e], s_t[e], -1, 0.0f, 0.0f, c, cp);
            if (c > cc && (OBJ || cp <= band)) {
                const uint64_t key = (uint64_t)vkey(c) << 32 | (uint32_t)(0xffffffffu - (uint32_t)e);
                best = key > best ? key : best;
            }
        }
        uint64_t mv = block_max(best);
        bool pair = false;
        if (mv == 0 && pairs_ok) {
            // two-node moves (n1 < n2, kept entries e1 and e2) in one flat order
            // (n1, n2, e1, e2); t -> pair p (its moves start at s_pov[p]) -> (j1, j2)
            const int total = s_pov[npairs];
            int p = 0;
            for (int t = tid; t < total; t += nt) {
                while (s_pov[p + 1] <= t) ++p;
                const int n1 = s_pnv[p] / NMAX, n2 = s_pnv[p] % NMAX;
                int c1 = 0, o1 = 0, f1 = 0, c2 = 0, o2 = 0, f2 = 0, F2 = 1;
#pragma unroll
                for (int m = 0; m < NN; ++m) {
                    if (m == n1) {
                        c1 = cur[m];
                        o1 = off[m];
                        f1 = foff[m];
                    }
                    if (m == n2) {
                        c2 = cur[m];
                        o2 = off[m];
                        f2 = foff[m];
                        F2 = foff[m + 1] - foff[m];
                    }
                }
                // t - s_pov[p] = j1 F2 + j2; the float quotient is exact: (x + 0.5) / F2
                // stays at least 0.5 / F2 >= 2^-10 away from an integer, far above its error
                const int x = t - s_pov[p];
                const int j1 = (int)(((float)x + 0.5f) / (float)F2);
                const int j2 = x - j1 * F2;
                const int e1 = s_fe[f1 + j1], e2 = s_fe[f2 + j2];
                if (e1 - o1 == c1 || e2 - o2 == c2) continue;
                if (!OBJ && !(s_a[e1] * s_a[e2] > s_a[o1 + c1] * s_a[o2 + c2])) continue;  // cannot raise corr
                float c, cp = 0.0f;
                if (OBJ)
                    c = climb_est<NN>(P, N, ca, ct, cd, n1, s_a[e1], s_t[e1], s_d[e1], n2, s_a[e2], s_t[e2], s_d[e2],
                                      mk);
                else
                    climb_eval<NN>(P, N, ca, ct, n1, s_a[e1], s_t[e1], n2, s_a[e2], s_t[e2], c, cp);
                if (c > cc && (OBJ || cp <= band)) {
                    const uint32_t id = (uint32_t)(n1 * NMAX + n2) << 16 | (uint32_t)(e1 - o1) << 8 | (uint32_t)(e2 - o2);
                    const uint64_t key = (uint64_t)vkey(c) << 32 | (uint32_t)(0xffffffffu - id);
                    best = key > best ? key : best;
                }
            }
            mv = block_max(best);
            pair = true;
        }
        if (mv == 0) break;
        // every lane applies the move to its copy of the plan
        const uint32_t id = 0xffffffffu - (uint32_t)mv;
        cc = OBJ ? fkey_value((uint32_t)(mv >> 32)) : __uint_as_float((uint32_t)(mv >> 32));
        int mn1, mi1, mn2 = -1, mi2 = 0;
        if (pair) {
            mn1 = (int)(id >> 16) / NMAX;
            mn2 = (int)(id >> 16) % NMAX;
            mi1 = (int)(id >> 8 & 0xffu);
            mi2 = (int)(id & 0xffu);
        } else {
            mn1 = s_node[id];
            int o1 = 0;
#pragma unroll
            for (int m = 0; m < NN; ++m)
                if (m == mn1) o1 = off[m];
            mi1 = (int)id - o1;
        }
#pragma unroll
        for (int m = 0; m < NN; ++m) {
            if (m == mn1 || m == mn2) {
                cur[m] = m == mn1 ? mi1 : mi2;
                ca[m] = s_a[off[m] + cur[m]];
                ct[m] = s_t[off[m] + cur[m]];
                if (OBJ) cd[m] = s_d[off[m] + cur[m]];
            }
        }
    }
    // the seed slot's format: corr bits + 1, or the estimate's key
    if (tid == 0) atomicMax(J->scert + k * NSLOT, OBJ ? fkey(cc) : __float_as_uint(cc) + 1u);
    }  // levels
}

// ---------------------------------------------------------------------------
// RANGE sources, objective mode: the same prefix-shared sweep with additive
// terms.  Per plan: T = max(tau_y + M, S2), G = U_x + u_y - lambda_l T (one
// fused rounding), D = D_x + d_y; the bin of D gives the prefilter threshold.
// U and D are summed in node order (prefix, x, y) in fp32.
// ---------------------------------------------------------------------------

struct ObjPlan {
    float G, D;
};

template <bool HAS_S2>
__device__ __forceinline__ ObjPlan obj_plan(const float2 vy, float dy, float M, float S2, float ux, float dx,
                                            float nl) {
    float T = vy.y + M;
    if (HAS_S2) T = fmaxf(T, S2);
    return ObjPlan{fmaf(nl, T, ux + vy.x), dx + dy};
}

template <bool HAS_S2, bool B256 = false>
__device__ __forceinline__ uint64_t sweep_test_obj(const float2 vy, float dy, float M, float S2, float ux, float dx,
                                                   float nl, uint32_t sh, const float* s_bins) {
    const ObjPlan q = obj_plan<HAS_S2>(vy, dy, M, S2, ux, dx, nl);
    const uint32_t off = B256 ? (__float_as_uint(q.D) >> 16) & 0x3fcu : (__float_as_uint(q.D) >> sh) & 0xfcu;
    const float thr = *(const float*)((const char*)s_bins + off);
    return __ballot(q.G >= thr);
}

// Objective mode, bin thresholds lowered ahead by each implementation j of y.
// A row fixes ux (utility through x) and M (fp32 path into y without y's own
// duration); its plan j has G = fma(-lambda_l, T, ux + u_j) with T =
// max(fp32(tau_j + M), S2) >= fp32(tau_j + M), so, lambda_l being >= 0, G is
// at most ux - lambda_l M + u_j - lambda_l tau_j plus the rounding of its
// three operations, and R = fp32 fma(-lambda_l, M, ux) is at least ux -
// lambda_l M less one rounding.  With c_j = P->ysub[j] >= u_j - lambda_l tau_j
// + (a bound on those four roundings), a plan whose G reaches a bin threshold
// t has R >= t - c_j.  Returned: the order key (fkey) of an fp32 value <= t -
// c_j, so the row's test is skey(R) >= the least key of its plans' bins.
// skey: the signed order key of a float (the magnitude bits of a negative
// value flipped; -0 keys just below +0), three operations.
__device__ __forceinline__ int32_t skey(float x) {
    const int32_t b = __float_as_int(x);
    return b ^ ((b >> 31) & 0x7fffffff);
}

__device__ __forceinline__ int32_t yshift_key(float t, float c) {
    float x = t;
    if (t != INFINITY && t != -INFINITY) {
        x = t - c;  // nearest: within half an ulp of t - c
        if (x != -INFINITY) {
            const uint32_t b = __float_as_uint(x);
            if (x > 0.0f) x = __uint_as_float(b - 1u);       // one ulp down (+inf: the largest finite)
            else if (x < 0.0f) x = __uint_as_float(b + 1u);  // one ulp down
        }
        if (x == 0.0f) x = -0.0f;  // -0 keys below +0; a zero R (either sign) still passes
    }
    return skey(x);
}

// The rare path of the shifted sweep: the row's plans with the sweep's own
// per-plan prefilter (G against its D bin's threshold, s_thr) and the exact
// per-level test.
template <bool HAS_S2>
__device__ __forceinline__ void sweep_rare_obj(PD P, JD J, uint64_t b, int ix, float ux, float dx, float M, float S2,
                                               const float* s_thr) {
    const CS float2* aty = cs(P->aty);
    const CS float* dyt = cs(P->demy);
    const int ry = P->ry;
    const float nl = -P->lam_l;
    const uint64_t base = (b * (uint64_t)P->rx + (uint64_t)ix) * (uint64_t)ry;
    for (int iy = 0; iy < ry; ++iy) {
        const ObjPlan q = obj_plan<HAS_S2>(aty[iy], dyt[iy], M, S2, ux, dx, nl);
        const float thr = *(const float*)((const char*)s_thr + ((__float_as_uint(q.D) >> 16) & 0x3fcu));
        const uint64_t idx = base + (uint64_t)iy;
        if (q.G >= thr && idx - J->begin < J->count && is_candidate_obj(P, J, q.G, q.D)) append_cand(J, idx, q.G, q.D);
    }
}

// A row of the shifted sweep parked in its wave's queue (as RareRow).
struct ObjRareRow {
    uint64_t b;
    uint32_t ix;
    float ux, dx, M, S2;
};

template <bool HAS_S2>
__device__ __forceinline__ void flush_rare_obj(PD P, JD J, const ObjRareRow* q, uint32_t n, const float* s_thr) {
    const uint32_t lane = threadIdx.x & 63;
    if (lane < n) {
        const ObjRareRow e = q[lane];
        sweep_rare_obj<HAS_S2>(P, J, e.b, (int)e.ix, e.ux, e.dx, e.M, e.S2, s_thr);
    }
}

// The objective-mode inner sweep of block b (the prefix pf evaluated).  B256
// with RY > 0: the shifted thresholds (s_bins: the 256 bin thresholds, then
// RY x 256 keys of yshift_key), one test per row, rows that pass parked in q.
template <bool HAS_S2, int RY, bool B256>
__device__ __forceinline__ void sweep_block_obj(PD P, JD J, uint64_t b, bool live, const Prefix& pf,
                                                const float2 (&vyr)[RY > 0 ? RY : 1],
                                                const float (&dyr)[RY > 0 ? RY : 1], const float* s_bins,
                                                ObjRareRow* q, uint32_t& qn, uint64_t live_mask) {
    const uint32_t sh = (uint32_t)P->bin_shift - 2u;
    const CS float2* atx = cs(P->atx);
    const CS float2* aty = cs(P->aty);
    const CS float* dxt = cs(P->demx);
    const CS float* dyt = cs(P->demy);
    const int rx = P->rx, ry = P->ry;
    // without a second sink x is no sink, so it feeds y
    const bool exy = !HAS_S2 || P->edge_xy != 0;
    const float nl = -P->lam_l;
    if constexpr (B256 && RY > 0) {
        const int32_t* s_key = (const int32_t*)(s_bins + NBINS2);
        for (int ix = 0; ix < rx; ++ix) {
            const float2 vx = atx[ix];
            const float fx = vx.y + pf.px;
            const float ux = pf.pc + vx.x;
            const float dx = pf.pd + dxt[ix];
            const float M = exy ? fmaxf(pf.py, fx) : pf.py;
            const float S2 = exy ? pf.s : fmaxf(pf.s, fx);
            const float R = fmaf(nl, M, ux);
            int32_t m = INT32_MAX;
#pragma unroll
            for (int j = 0; j < (RY > 0 ? RY : 1); ++j) {
                const float D = dx + dyr[j];
                m = min(m, *(const int32_t*)((const char*)(s_key + j * NBINS2) + ((__float_as_uint(D) >> 16) & 0x3fcu)));
            }
            const uint64_t hit = __ballot(skey(R) >= m) & live_mask;
            if (hit) {
                const uint32_t nh = (uint32_t)__popcll(hit);
                if (qn + nh > (uint32_t)RQ) {
                    flush_rare_obj<HAS_S2>(P, J, q, qn, s_bins);
                    qn = 0;
                }
                const uint32_t lane = threadIdx.x & 63;
                if (hit >> lane & 1ull) {
                    const uint32_t o = qn + __builtin_amdgcn_mbcnt_hi((uint32_t)(hit >> 32),
                                                                      __builtin_amdgcn_mbcnt_lo((uint32_t)hit, 0u));
                    q[o] = ObjRareRow{b, (uint32_t)ix, ux, dx, M, S2};
                }
                qn += nh;
            }
        }
        return;
    }
    for (int ix = 0; ix < rx; ++ix) {
        const float2 vx = atx[ix];
        const float fx = vx.y + pf.px;
        const float ux = pf.pc + vx.x;
        const float dx = pf.pd + dxt[ix];
        const float M = exy ? fmaxf(pf.py, fx) : pf.py;
        const float S2 = exy ? pf.s : fmaxf(pf.s, fx);
        uint64_t hit = 0;
        int iy = 0;
        if (RY > 0) {
#pragma unroll
            for (int j = 0; j < (RY > 0 ? RY : 1); ++j)
                hit |= sweep_test_obj<HAS_S2, B256>(vyr[j], dyr[j], M, S2, ux, dx, nl, sh, s_bins);
            iy = ry;
        }
        for (; iy + 4 <= ry; iy += 4) {
            const float2 v0 = aty[iy], v1 = aty[iy + 1], v2 = aty[iy + 2], v3 = aty[iy + 3];
            const float d0 = dyt[iy], d1 = dyt[iy + 1], d2 = dyt[iy + 2], d3 = dyt[iy + 3];
            hit |= sweep_test_obj<HAS_S2, B256>(v0, d0, M, S2, ux, dx, nl, sh, s_bins);
            hit |= sweep_test_obj<HAS_S2, B256>(v1, d1, M, S2, ux, dx, nl, sh, s_bins);
            hit |= sweep_test_obj<HAS_S2, B256>(v2, d2, M, S2, ux, dx, nl, sh, s_bins);
            hit |= sweep_test_obj<HAS_S2, B256>(v3, d3, M, S2, ux, dx, nl, sh, s_bins);
        }
        for (; iy < ry; ++iy) hit |= sweep_test_obj<HAS_S2, B256>(aty[iy], dyt[iy], M, S2, ux, dx, nl, sh, s_bins);
        if (hit) {
            // rare: re-score this lane's row with the exact per-level test
            const uint64_t base = (b * (uint64_t)rx + (uint64_t)ix) * (uint64_t)ry;
            if (live && (hit >> (threadIdx.x & 63) & 1ull)) {
                for (int iy = 0; iy < ry; ++iy) {
                    const ObjPlan q = obj_plan<HAS_S2>(aty[iy], dyt[iy], M, S2, ux, dx, nl);
                    const uint64_t idx = base + (uint64_t)iy;
                    if (idx - J->begin < J->count && is_candidate_obj(P, J, q.G, q.D)) append_cand(J, idx, q.G, q.D);
                }
            }
        }
    }
}

// Work units as in k_sweep (runs of J->gblk blocks per thread with NPRE > 0);
// B256: the 256 bins of D's pattern on shift 18 (one AND per plan).
template <bool HAS_S2, int RY, int NPRE, bool B256 = false, int RAD = 0>
__global__ void __launch_bounds__(WG) k_sweep_obj(const JobDev* __restrict__ jobs, uint64_t unit_off, int pat_cap) {
    extern __shared__ float s_f[];
    JD J = cs(jobs + blockIdx.y);
    PD P = cs(J->prob);
    const uint64_t units = J->units;
    const int G = NPRE > 0 ? J->gblk : 1;
    const uint64_t t0 = unit_off + (uint64_t)blockIdx.x * WG;
    if (t0 >= units) return;
    const uint64_t t = t0 + threadIdx.x;
    const bool live = t < units;
    const uint64_t b0 = J->blk_first + (live ? t : units - 1) * (uint64_t)G;
    constexpr bool YSH = B256 && RY > 0;
    __shared__ float s_bins[YSH ? (1 + (RY > 0 ? RY : 1)) * NBINS2 : (B256 ? NBINS2 : NBINS)];
    if (B256) {
        static_assert(!B256 || NBINS2 == WG, "one bin per thread");
        const float thr = __uint_as_float(J->table2[threadIdx.x]);
        s_bins[threadIdx.x] = thr;
        if constexpr (YSH) {
            int32_t* s_key = (int32_t*)(s_bins + NBINS2);
#pragma unroll
            for (int j = 0; j < (RY > 0 ? RY : 1); ++j) s_key[j * NBINS2 + threadIdx.x] = yshift_key(thr, P->ysub[j]);
        }
    } else if (threadIdx.x < NBINS) {
        s_bins[threadIdx.x] = __uint_as_float(J->table[threadIdx.x]);
    }
    // dynamic LDS as in k_sweep, then the prefix nodes' d terms (pat_cap entries)
    float2* s_pat = (float2*)(s_f + (NPRE > 0 ? (size_t)0 : (size_t)max(P->npre, 1) * WG));
    float* s_pd = (float*)(s_pat + pat_cap);
    const float2* pat = stage_prefix_rows<true>(P, s_pat, s_pd, pat_cap);
    // a wave whose lanes all lie past the last unit has nothing to score (no
    // barrier follows)
    if (t0 + (threadIdx.x & ~63u) >= units) return;
    float2 vyr[RY > 0 ? RY : 1];
    float dyr[RY > 0 ? RY : 1];
    if (RY > 0) {
        const CS float2* aty = cs(P->aty);
        const CS float* dyt = cs(P->demy);
#pragma unroll
        for (int iy = 0; iy < RY; ++iy) {
            vyr[iy] = aty[iy];
            dyr[iy] = dyt[iy];
            if constexpr (YSH) {
                // the shifted sweep reads only y's d terms; keep them in
                // scalar registers
                uint32_t v = __float_as_uint(dyr[iy]);
                asm volatile("" : "+s"(v));
                dyr[iy] = __uint_as_float(v);
            }
        }
    }
    __shared__ ObjRareRow s_q[YSH ? WG / 64 : 1][RQ];
    ObjRareRow* q = s_q[YSH ? threadIdx.x >> 6 : 0];
    uint32_t qn = 0;
    const uint64_t live_mask = __ballot(live);
    if constexpr (NPRE > 0) {
        const PrefixHead ph = prefix_head<NPRE, true, RAD>(P, b0, J->big, pat, s_pd);
        for (int g = 0; g < G; ++g)
            sweep_block_obj<HAS_S2, RY, B256>(P, J, b0 + (uint64_t)g, live,
                                              prefix_tail<NPRE, true>(P, ph, g, pat, s_pd), vyr, dyr, s_bins, q, qn,
                                              live_mask);
    } else {
        const Prefix pf = prefix_eval<NPRE, true>(P, b0, J->big, s_f, pat, s_pd);
        sweep_block_obj<HAS_S2, RY, B256>(P, J, b0, live, pf, vyr, dyr, s_bins, q, qn, live_mask);
    }
    if (YSH && qn) flush_rare_obj<HAS_S2>(P, J, q, qn, s_bins);
}

// Seeding pre-pass of the objective sweep: one hashed row per window of S
// rows; per level the greatest fp32 estimate fma(-m_k, D, G) of a sampled plan
// (every plan is admissible), reduced through DPP, LDS and an atomic max on
// its ordered key.
template <bool HAS_S2, int NPRE>
__global__ void __launch_bounds__(WG) k_sample_sweep_obj(const JobDev* __restrict__ jobs) {
    extern __shared__ float s_dyn[];
    __shared__ uint32_t s_red[KMAX][WG / 64];
    JD J = cs(jobs + blockIdx.y);
    PD P = cs(J->prob);
    const int K = P->k;
    float* s_f = s_dyn;                                  // prefix recurrence, [npre][WG]
    float* s_b = s_dyn + (size_t)max(P->npre, 1) * WG;   // best estimate per level, [K][WG]
    float2* s_pat = (float2*)(s_b + (size_t)K * WG);     // prefix rows, PAT_MAX entries
    float* s_pd = (float*)(s_pat + PAT_MAX);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint64_t S = J->sample_stride;
    const int rx = P->rx, ry = P->ry;
    const uint64_t units = J->nblk * (uint64_t)rx;
    const uint64_t nsamp = (units + S - 1) / S;
    const uint64_t t0 = (uint64_t)blockIdx.x * WG;
    if (t0 >= nsamp) return;
    const uint64_t t = t0 + tid;
    const bool live = t < nsamp;
    const uint64_t u = sample_unit(live ? t : nsamp - 1, S, units);
    uint64_t b;
    int ix;
    if (units <= 0xffffffffull && P->xnode >= 0) {
        const uint32_t q = mdiv((uint32_t)u, P->rmag[P->xnode]);
        b = J->blk_first + q;
        ix = (int)((uint32_t)u - q * (uint32_t)rx);
    } else {
        b = J->blk_first + u / (uint64_t)rx;
        ix = (int)(u % (uint64_t)rx);
    }
    const float2* pat = stage_prefix_rows<true>(P, s_pat, s_pd);
    const Prefix pf = prefix_eval<NPRE, true>(P, b, J->big, s_f, pat, s_pd);
    for (int k = 0; k < K; ++k) s_b[k * WG + tid] = -INFINITY;
    const float2 vx = cs(P->atx)[ix];
    const float fx = vx.y + pf.px;
    const float ux = pf.pc + vx.x;
    const float dx = pf.pd + cs(P->demx)[ix];
    const bool exy = P->edge_xy != 0;
    const float M = exy ? fmaxf(pf.py, fx) : pf.py;
    const float S2 = exy ? pf.s : fmaxf(pf.s, fx);
    const float nl = -P->lam_l;
    const uint64_t base = (b * (uint64_t)rx + (uint64_t)ix) * (uint64_t)ry;
    const CS float2* aty = cs(P->aty);
    const CS float* dyt = cs(P->demy);
    for (int iy = 0; iy < ry; ++iy) {
        const ObjPlan q = obj_plan<HAS_S2>(aty[iy], dyt[iy], M, S2, ux, dx, nl);
        if (live && (base + (uint64_t)iy - J->begin < J->count))
            for (int k = 0; k < K; ++k) {
                float* r = s_b + k * WG + tid;
                *r = fmaxf(*r, fmaf(-P->m32[k], q.D, q.G));
            }
    }
    for (int k = 0; k < K; ++k) {
        const float v = s_b[k * WG + tid];
        const uint32_t e = wave_max_u32(v > -INFINITY ? fkey(v) : 0u);
        if (lane == 0) s_red[k][wave] = e;
    }
    __syncthreads();
    if (tid < K) {
        uint32_t e = 0;
        for (int w = 0; w < WG / 64; ++w) e = max(e, s_red[tid][w]);
        if (e) atomicMax(J->scert + tid * NSLOT + (blockIdx.x % NSLOT), e);
    }
}

// ---------------------------------------------------------------------------
// per-source threshold and prefilter table (one wave per source)
// ---------------------------------------------------------------------------

__global__ void k_table(JobDev* __restrict__ jobs, int njobs) {
    const int j = blockIdx.x;
    if (j >= njobs) return;
    JD J = cs(jobs + j);
    build_table(J, cs(J->prob));
}

// The thresholds and tables again from the seeds, the candidate list kept.
__global__ void k_retable(JobDev* __restrict__ jobs, int njobs) {
    const int j = blockIdx.x;
    if (j >= njobs) return;
    JD J = cs(jobs + j);
    build_table(J, cs(J->prob), false);
}

// ---------------------------------------------------------------------------
// generic per-plan path: ROWS sources, non-uniform pressure, per-plan scores
// ---------------------------------------------------------------------------

// ids of plan `j` of the source into the thread's LDS column; returns the plan
// index; sets *bad for an out-of-range row id (the id is then read as 0).
__device__ __forceinline__ uint64_t load_plan(JD J, PD P,
                                              uint64_t j, uint8_t* __restrict__ s_id, bool* bad) {
    const int tid = threadIdx.x;
    const int N = P->n;
    if (J->kind == DY_SOURCE_RANGE) {
        const uint64_t idx = J->begin + j;
        if (!J->big) {
            uint32_t x = (uint32_t)idx;
            for (int n = N - 1; n >= 0; --n) {
                uint32_t q = mdiv(x, P->rmag[n]);
                s_id[n * WG + tid] = (uint8_t)(x - q * (uint32_t)P->radix[n]);
                x = q;
            }
        } else {
            uint64_t x = idx;
            for (int n = N - 1; n >= 0; --n) {
                uint64_t r = (uint64_t)P->radix[n];
                s_id[n * WG + tid] = (uint8_t)(x % r);
                x /= r;
            }
        }
        return idx;
    }
    const uint8_t* row = J->rows + j * J->stride;
    bool b = false;
    // word loads only when a row is whole words, so the last row is never over-read
    if (((J->stride | (uint64_t)(uintptr_t)J->rows | (uint64_t)N) & 3u) == 0) {
        const uint32_t* w = (const uint32_t*)row;
        for (int q = 0; q < (N + 3) / 4; ++q) {
            uint32_t v = __builtin_nontemporal_load(w + q);
            for (int r = 0; r < 4 && 4 * q + r < N; ++r) {
                uint32_t id = (v >> (8 * r)) & 0xffu;
                const int n = 4 * q + r;
                if (id >= (uint32_t)P->radix[n]) {
                    b = true;
                    id = 0;
                }
                s_id[n * WG + tid] = (uint8_t)id;
            }
        }
    } else {
        for (int n = 0; n < N; ++n) {
            uint32_t id = row[n];
            if (id >= (uint32_t)P->radix[n]) {
                b = true;
                id = 0;
            }
            s_id[n * WG + tid] = (uint8_t)id;
        }
    }
    *bad = b;
    return J->index_base + j;
}

// fp32 corr and the unpressured CP (uniform mode) of the plan in the LDS column.
__device__ __forceinline__ void eval_uniform(PD P, const uint8_t* __restrict__ s_id,
                                             float* __restrict__ s_f, float& cc, float& cp) {
    const int tid = threadIdx.x;
    float c = 1.0f, best = 0.0f;
    for (int n = 0; n < P->n; ++n) {
        const float2 v = P->at[n * P->rmax + s_id[n * WG + tid]];
        c = c * v.x;
        float m = 0.0f;
        uint32_t pm = P->pred[n];
        while (pm) {
            int u = __builtin_ctz(pm);
            pm &= pm - 1;
            m = fmaxf(m, s_f[u * WG + tid]);
        }
        const float f = v.y + m;
        s_f[n * WG + tid] = f;
        if (P->sinks >> n & 1u) best = fmaxf(best, f);
    }
    cc = c;
    cp = best;
}

// Objective mode: fp32 U, nominal T and D of the plan in the LDS column, node
// order (tool nodes hold u = d = 0 in the tables).
__device__ __forceinline__ void eval_obj(PD P, const uint8_t* __restrict__ s_id, float* __restrict__ s_f, float& U,
                                         float& T, float& D) {
    const int tid = threadIdx.x;
    float u = 0.0f, d = 0.0f, best = 0.0f;
    for (int n = 0; n < P->n; ++n) {
        const int e = n * P->rmax + s_id[n * WG + tid];
        const float2 v = P->at[e];
        u = u + v.x;
        d = d + P->dem[e];
        float m = 0.0f;
        uint32_t pm = P->pred[n];
        while (pm) {
            int q = __builtin_ctz(pm);
            pm &= pm - 1;
            m = fmaxf(m, s_f[q * WG + tid]);
        }
        const float f = v.y + m;
        s_f[n * WG + tid] = f;
        if (P->sinks >> n & 1u) best = fmaxf(best, f);
    }
    U = u;
    T = best;
    D = d;
}

__device__ __forceinline__ float eval_corr(PD P, const uint8_t* __restrict__ s_id) {
    float c = 1.0f;
    for (int n = 0; n < P->n; ++n) c = c * P->at[n * P->rmax + s_id[n * WG + threadIdx.x]].x;
    return c;
}

// fp32 CP at level k from the general-mode latency table.
__device__ __forceinline__ float eval_cp_level(PD P, const uint8_t* __restrict__ s_id,
                                               float* __restrict__ s_f, int k) {
    const int tid = threadIdx.x;
    const float* lat = P->lat + (size_t)k * P->n * P->rmax;
    float best = 0.0f;
    for (int n = 0; n < P->n; ++n) {
        float m = 0.0f;
        uint32_t pm = P->pred[n];
        while (pm) {
            int u = __builtin_ctz(pm);
            pm &= pm - 1;
            m = fmaxf(m, s_f[u * WG + tid]);
        }
        const float f = lat[n * P->rmax + s_id[n * WG + tid]] + m;
        s_f[n * WG + tid] = f;
        if (P->sinks >> n & 1u) best = fmaxf(best, f);
    }
    return best;
}

// Seeding pre-pass of the generic path: one hashed plan per window of S plans.
// ncol: node columns of the per-thread LDS arrays (the launch's largest N).
__global__ void __launch_bounds__(WG) k_sample_generic(const JobDev* __restrict__ jobs, int ncol) {
    extern __shared__ float s_dyn[];
    JD J = cs(jobs + blockIdx.y);
    PD P = cs(J->prob);
    float* s_f = s_dyn;
    uint8_t* s_id = (uint8_t*)(s_dyn + (size_t)ncol * WG);
    const uint64_t S = J->sample_stride;
    const uint64_t nsamp = (J->count + S - 1) / S;
    const uint64_t t0 = (uint64_t)blockIdx.x * WG;
    if (t0 >= nsamp) return;
    const uint64_t t = t0 + threadIdx.x;
    const bool live = t < nsamp;
    bool bad = false;
    load_plan(J, P, sample_unit(live ? t : nsamp - 1, S, J->count), s_id, &bad);
    const int K = P->k;
    if (P->obj) {
        float U, T, D;
        eval_obj(P, s_id, s_f, U, T, D);
        const float G = fmaf(-P->lam_l, T, U);
        const bool ok = live && !bad;
#pragma unroll 1
        for (int k = 0; k < K; ++k) {
            uint32_t e = ok ? fkey(fmaf(-P->m32[k], D, G)) : 0u;
            e = wave_max_u32(e);
            if ((threadIdx.x & 63) == 0 && e)
                atomicMax(J->scert + k * NSLOT + ((blockIdx.x * (WG / 64) + (threadIdx.x >> 6)) % NSLOT), e);
        }
        return;
    }
    float cc, cp0 = 0.0f;
    if (P->uniform) {
        eval_uniform(P, s_id, s_f, cc, cp0);
    } else {
        cc = eval_corr(P, s_id);
    }
    const bool ok = live && !bad;
#pragma unroll 1
    for (int k = 0; k < K; ++k) {
        const float cp = P->uniform ? cp0 : eval_cp_level(P, s_id, s_f, k);
        uint32_t e = (ok && cp <= (P->uniform ? P->lo[k] : P->glo)) ? __float_as_uint(cc) + 1u : 0u;
        e = wave_max_u32(e);
        if ((threadIdx.x & 63) == 0 && e)
            atomicMax(J->scert + k * NSLOT + ((blockIdx.x * (WG / 64) + (threadIdx.x >> 6)) % NSLOT), e);
    }
}

// Scoring pass of the generic path: one plan per thread.
__global__ void __launch_bounds__(WG) k_scan(const JobDev* __restrict__ jobs, uint64_t unit_off, int ncol) {
    extern __shared__ float s_dyn[];
    JD J = cs(jobs + blockIdx.y);
    PD P = cs(J->prob);
    float* s_f = s_dyn;
    uint8_t* s_id = (uint8_t*)(s_dyn + (size_t)ncol * WG);
    const uint64_t n_units = J->count;
    const uint64_t t0 = unit_off + (uint64_t)blockIdx.x * WG;
    if (t0 >= n_units) return;
    const uint64_t t = t0 + threadIdx.x;
    const bool live = t < n_units;
    bool bad = false;
    const uint64_t idx = load_plan(J, P, live ? t : n_units - 1, s_id, &bad);
    if (live && bad) atomicOr(J->flags, (int32_t)JF_BAD_ROW);
    if (P->obj) {
        float U, T, D;
        eval_obj(P, s_id, s_f, U, T, D);
        const float G = fmaf(-P->lam_l, T, U);
        const float thr = __uint_as_float(J->table[(__float_as_uint(D) >> (uint32_t)P->bin_shift) & 63u]);
        if (live && !bad && G >= thr && is_candidate_obj(P, J, G, D)) append_cand(J, idx, G, D);
    } else if (P->uniform) {
        float cc, cp;
        eval_uniform(P, s_id, s_f, cc, cp);
        const float thr = __uint_as_float(J->table[(__float_as_uint(cp) >> (uint32_t)P->bin_shift) & 63u]);
        if (live && !bad && cc >= thr && is_candidate(P, J, cp, cc)) append_cand(J, idx, cc, cp);
    } else {
        // per-backend pressure: the unpressured CP's bands first (a conservative
        // prefilter), then each level's exact fp32 CP_k; the candidate keeps the
        // unpressured CP, which the list's bands refer to
        float cc, cp0;
        eval_uniform(P, s_id, s_f, cc, cp0);
        const float thr = __uint_as_float(J->table[(__float_as_uint(cp0) >> (uint32_t)P->bin_shift) & 63u]);
        bool want = false;
        if (live && !bad && cc >= thr && is_candidate(P, J, cp0, cc))
            for (int k = 0; k < P->k && !want; ++k)
                if (cc >= J->thr[k]) want = eval_cp_level(P, s_id, s_f, k) <= P->ghi;
        if (want) append_cand(J, idx, cc, cp0);
    }
}

// ---------------------------------------------------------------------------
// certification: exact fp64 winner among the candidates (one WG per level)
// ---------------------------------------------------------------------------

__device__ __forceinline__ bool better(double c1, uint64_t i1, double c2, uint64_t i2) {
    return c1 > c2 || (c1 == c2 && i1 < i2);
}

// Wave-wide best (corr desc, index asc) through lane exchanges.
__device__ __forceinline__ void wave_best(double& c, uint64_t& i) {
    for (int o = 32; o > 0; o >>= 1) {
        const double c2 = __shfl_xor(c, o);
        const uint64_t i2 = __shfl_xor(i, o);
        if (better(c2, i2, c, i)) {
            c = c2;
            i = i2;
        }
    }
}

// Wave-wide best (corr desc, index asc) carrying the winner's CP and demand.
__device__ __forceinline__ void wave_best4(double& c, uint64_t& i, double& cp, double& d) {
    for (int o = 32; o > 0; o >>= 1) {
        const double c2 = __shfl_xor(c, o);
        const uint64_t i2 = __shfl_xor(i, o);
        const double p2 = __shfl_xor(cp, o);
        const double d2 = __shfl_xor(d, o);
        if (better(c2, i2, c, i)) {
            c = c2;
            i = i2;
            cp = p2;
            d = d2;
        }
    }
}

constexpr int CERT_LDS_TABLES = 32 * 1024;  // fp64 tables staged in LDS when they fit
constexpr int CERT_CACHE = 512;             // candidates cached in LDS by each certification wave
constexpr int CERT_PACK_CACHE = 64;         // ... when four waves share a block

// Merge of a source's certification waves into its K choices, by the block
// that finishes certification last (64 threads).  When no list overflowed and
// no row was bad, the seed slots and the fallback state are cleared for the
// next call (a call that leaves anything else behind makes the host re-run
// k_init first).
__device__ void merge_cert(JD J, PD P) {
    __shared__ dy_choice s_out[KMAX];
    const int K = P->k;
    // lane = (level, wave) pair; levels in groups of 64 / CERT_WAVES
    constexpr int LPG = 64 / CERT_WAVES;
    const int lane = threadIdx.x, w = lane % CERT_WAVES, kk = lane / CERT_WAVES;
    for (int k0 = 0; k0 < K; k0 += LPG) {
        const int k = k0 + kk;
        double bc = -INFINITY, bcp = 0.0, bd = 0.0;
        uint64_t bi = ~0ull;
        if (k < K && w < J->cert_waves) {
            bc = J->cert_c[k * CERT_WAVES + w];
            bi = J->cert_i[k * CERT_WAVES + w];
            bcp = J->cert_cp[k * CERT_WAVES + w];
            bd = J->cert_d[k * CERT_WAVES + w];
        }
        for (int o = CERT_WAVES / 2; o > 0; o >>= 1) {
            const double c2 = __shfl_xor(bc, o);
            const uint64_t i2 = __shfl_xor(bi, o);
            const double p2 = __shfl_xor(bcp, o);
            const double d2 = __shfl_xor(bd, o);
            if (better(c2, i2, bc, bi)) {
                bc = c2;
                bi = i2;
                bcp = p2;
                bd = d2;
            }
        }
        if (w == 0 && k < K) {
            dy_choice c;
            if (bi != ~0ull) {
                c.index = (int64_t)bi;
                c.feasible = 1;
                c.corr = (float)bc;
                c.cp = (float)bcp;
                c.demand = (float)bd;
            } else {
                c.index = -1;
                c.feasible = 0;
                c.corr = NAN;
                c.cp = NAN;
                c.demand = NAN;
            }
            J->out[k] = c;
            s_out[k] = c;
        }
    }
    // scratch for the next call first: a caller that returns on the completion
    // word below may start its next call (on any stream) right away, and that
    // call skips k_init when this one raised no flag
    const int32_t flags = *J->flags;
    if (flags == 0) {
        for (int i = threadIdx.x; i < KMAX * NSLOT; i += 64) J->scert[i] = 0u;
        if (threadIdx.x < KMAX) {
            J->fb_corr[threadIdx.x] = 0ull;
            J->fb_index[threadIdx.x] = ~0ull;
        }
    }
    // the host-mapped copy: the K choices as consecutive dwords, then the counters
    __syncthreads();
    if (J->hout) {
        static_assert(sizeof(dy_choice) == 24, "6 dwords per choice");
        const uint32_t* src = (const uint32_t*)s_out;
        uint32_t* dst = (uint32_t*)J->hout;
        for (int i = threadIdx.x; i < K * 6; i += 64) dst[i] = src[i];
        if (threadIdx.x == 0) {
            *J->hncand = *J->ncand;
            *J->hflags = flags;
        }
        if (J->hdone) {  // completion word last, behind the results and the cleared scratch
            __threadfence_system();
            __syncthreads();
            if (threadIdx.x == 0) __hip_atomic_store(J->hdone, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
        }
    }
}

// fp64 scores of the plan whose ids sit at ids[n * 64], in node order as the
// definitions take them: x = corr (objective: U, the LLM nodes' sum of u), cp
// = the CP at the level's durations, d = demand (objective: D, the LLM nodes'
// sum of tau).  The three table loads of eight nodes are issued together, so a
// lane waits on memory about N / 8 times instead of 3 N.
template <bool OBJ>
__device__ __forceinline__ void cert_eval(PD P, int N, int R, const uint8_t* ids, double* f, const double* a64,
                                          const double* d64, const double* lat, double& x, double& cp,
                                          double& d) {
    x = OBJ ? 0.0 : 1.0;
    cp = 0.0;
    d = 0.0;
    for (int n0 = 0; n0 < N; n0 += 8) {
        double va[8], vl[8], vd[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int n = n0 + j;
            const int e = n < N ? n * R + ids[n * 64] : 0;
            va[j] = a64[e];
            vl[j] = lat[e];
            vd[j] = d64[e];
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int n = n0 + j;
            if (n < N) {
                if (!OBJ) {
                    x = x * va[j];
                    d = d + vd[j];
                } else if (P->llm >> n & 1u) {
                    x = x + va[j];
                    d = d + vd[j];
                }
                double m = 0.0;
                uint32_t pm = P->pred[n];
                while (pm) {
                    const int u = __builtin_ctz(pm);
                    pm &= pm - 1;
                    const double fu = f[u * 64];
                    if (fu > m) m = fu;
                }
                const double fn = vl[j] + m;
                f[n * 64] = fn;
                if ((P->sinks >> n & 1u) && fn > cp) cp = fn;
            }
        }
    }
}

// Certification: grid (cert_waves, source, level), one wave per block.  Pass
// A tightens the level's threshold with the candidates whose fp32 CP is
// certainly feasible.  Pass B re-evaluates in fp64 every candidate of this
// wave's share that could still win the level and keeps the feasible one
// with the greatest corr, then the lowest index.  The source's block that finishes
// last merges the waves (merge_cert).  Levels run in separate blocks: each
// lane walks its candidates once per block instead of once per level.
// Dynamic LDS: tab_d doubles for the fp64 tables (0: read from global memory),
// then the recurrence column f [nf][64] (fp64) and the ids [nf][64], nf >= N.
// Dynamic LDS of one certification wave, in doubles: the fp64 tables (tab_d),
// nf node values and nf id bytes per lane, `cache` candidates.
__host__ __device__ constexpr size_t cert_slot_doubles(int tab_d, int nf, int cache) {
    return (size_t)tab_d + (size_t)nf * 64 + ((size_t)nf * 64 + 7) / 8 + (size_t)cache * (sizeof(Cand) / 8);
}

// PACK = false: grid (waves, sources, levels), 64 threads, the source's
// cert_waves waves per level, `cache` = CERT_CACHE candidates in LDS.
// PACK = true (every source has one wave per level and no host-mapped copy):
// blockDim 256, four (source, level) searches per block, one per wave,
// search blockIdx.x * 4 + wave in source-major order (nsearch in all), each
// with its own LDS slot (a CU holds few one-wave blocks).
template <bool PACK>
__global__ void __launch_bounds__(256) k_certify(const JobDev* __restrict__ jobs, int tab_d, int nf, int cache,
                                                 int nsearch, int kmax) {
    extern __shared__ double s_dyn64[];
    const int slot = PACK ? __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)) : 0;
    double* s_tab = s_dyn64 + (size_t)slot * cert_slot_doubles(tab_d, nf, cache);
    double* s_f = s_tab + tab_d;
    uint8_t* s_id = (uint8_t*)(s_f + (size_t)nf * 64);
    Cand* s_cand = (Cand*)(s_f + (size_t)nf * 64 + ((size_t)nf * 64 + 7) / 8);
    int ji = blockIdx.y, g = blockIdx.x, k = blockIdx.z;
    if (PACK) {
        const int q = (int)blockIdx.x * 4 + slot;
        if (q >= nsearch) return;
        ji = q / kmax;
        k = q % kmax;
        g = 0;
    }
    JD J = cs(jobs + ji);
    PD P = cs(J->prob);
    if (g >= J->cert_waves || k >= P->k) return;
    const int N = P->n, R = P->rmax, lane = threadIdx.x & 63;
    const uint32_t nc = min(*J->ncand, J->cap);
    uint8_t* ids = s_id + lane;
    double* f = s_f + lane;
    const size_t NR = (size_t)N * R;
    const double* a64 = P->a64;
    const double* d64 = P->dem64;
    const double* lat = P->lat64 + (P->obj ? (size_t)0 : (size_t)k * NR);
    if (3 * NR <= (size_t)tab_d) {
        // unrolled so that many loads are in flight before the first LDS store
#pragma unroll 8
        for (size_t q = lane; q < NR; q += 64) {
            s_tab[q] = a64[q];
            s_tab[NR + q] = d64[q];
            s_tab[2 * NR + q] = lat[q];
        }
        a64 = s_tab;
        d64 = s_tab + NR;
        lat = s_tab + 2 * NR;
    }
    static_assert(NSLOT == 64, "one seed slot per lane");
    const uint32_t sl = J->scert[k * NSLOT + lane];
    const uint32_t ncache = min(nc, (uint32_t)cache);
#pragma unroll 8
    for (uint32_t i = lane; i < ncache; i += 64) s_cand[i] = J->cand[i];
    if (PACK) {  // the wave is alone in its slot
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    } else {
        __syncthreads();
    }
    const uint32_t step = 64u * (uint32_t)J->cert_waves;
    double bc = -INFINITY, bcp = 0.0, bd = 0.0;
    uint64_t bi = ~0ull;
    if (P->obj) {
        // Pass A: the best estimate of J_k among the seed and the candidates
        // (fma(-m, D, G), one rounding); Pass B: every candidate whose estimate
        // reaches that minus 2 E_k, re-evaluated exactly.
        const double m = P->m64[k], e2 = P->err2[k];
        double sb = sl ? (double)fkey_value(sl) : -INFINITY;
        for (uint32_t i = lane; i < nc; i += 64) {
            const Cand c = i < ncache ? s_cand[i] : J->cand[i];
            sb = fmax(sb, fma(-m, (double)c.cp, (double)c.corr));
        }
        for (int o = 32; o > 0; o >>= 1) sb = fmax(sb, __shfl_xor(sb, o));
        double T = -INFINITY;
        if (sb > -INFINITY) {
            T = sb - e2;
            T = T - (fabs(sb) + e2) * 0x1p-50;
        }
        for (uint32_t i = (uint32_t)g * 64u + lane; i < nc; i += step) {
            const Cand c = i < ncache ? s_cand[i] : J->cand[i];
            if (!(fma(-m, (double)c.cp, (double)c.corr) >= T)) continue;
            if (!job_ids(J, P, c.index, ids, 64)) continue;
            double U, D, t;
            cert_eval<true>(P, N, R, ids, f, a64, d64, lat, U, t, D);
            const double j = obj_j(P->lam_l64, m, U, t, D);
            if (better(j, c.index, bc, bi)) {
                bc = j;
                bi = c.index;
                bcp = t;
                bd = D;
            }
        }
    } else {
        const float lo = P->lo[k], hi = P->hi[k];
        float sb = sl ? __uint_as_float(sl - 1u) : -1.0f;
        for (uint32_t i = lane; i < nc; i += 64) {
            const Cand c = i < ncache ? s_cand[i] : J->cand[i];
            if (c.cp <= lo) sb = fmaxf(sb, c.corr);
        }
        const uint32_t e = wave_max_u32(sb >= 0.0f ? __float_as_uint(sb) + 1u : 0u);
        const float T = cand_threshold(e ? __uint_as_float(e - 1u) : -1.0f, N);
        for (uint32_t i = (uint32_t)g * 64u + lane; i < nc; i += step) {
            const Cand c = i < ncache ? s_cand[i] : J->cand[i];
            if (!(c.corr >= T && c.cp <= hi)) continue;
            if (!job_ids(J, P, c.index, ids, 64)) continue;
            double corr, cp, d;
            cert_eval<false>(P, N, R, ids, f, a64, d64, lat, corr, cp, d);
            if (!better(corr, c.index, bc, bi)) continue;
            if (!(cp <= P->slo)) continue;
            bc = corr;
            bi = c.index;
            bcp = cp;
            bd = d;
        }
    }
    wave_best4(bc, bi, bcp, bd);
    if (J->cert_waves == 1 && !J->hout) {
        // one wave per level and no host-mapped copy: this block alone decides
        // level k, so it writes the choice and clears the level's seed slots
        // for the next call itself (no cross-block merge, whose device-scope
        // fences would make every one of thousands of blocks wait for the L2)
        if (lane == 0) {
            dy_choice c;
            if (bi != ~0ull) {
                c.index = (int64_t)bi;
                c.feasible = 1;
                c.corr = (float)bc;
                c.cp = (float)bcp;
                c.demand = (float)bd;
            } else {
                c.index = -1;
                c.feasible = 0;
                c.corr = NAN;
                c.cp = NAN;
                c.demand = NAN;
            }
            J->out[k] = c;
        }
        if (*J->flags == 0) {
            J->scert[k * NSLOT + lane] = 0u;
            if (lane == 0) {
                J->fb_corr[k] = 0ull;
                J->fb_index[k] = ~0ull;
            }
        }
        return;
    }
    if (PACK) return;  // not reached: PACK launches have one wave per level and no host copy
    if (lane == 0) {
        J->cert_c[k * CERT_WAVES + g] = bc;
        J->cert_i[k * CERT_WAVES + g] = bi;
        J->cert_cp[k * CERT_WAVES + g] = bcp;
        J->cert_d[k * CERT_WAVES + g] = bd;
    }
    if (last_block(J->sync, (uint32_t)(J->cert_waves * P->k))) merge_cert(J, P);
}

// Seeds from the first share of a long ROWS source (corr / SLO mode): every
// candidate gathered so far whose fp32 corr would raise level k's seed and
// whose CP is inside the level's band is re-evaluated exactly in fp64; a
// certainly-feasible one (the definition's CP_k <= SLO) becomes the level's
// seed, with its fp32 corr.  Any certainly-feasible plan gives a valid
// threshold, so the rest of the source is then scored against thresholds
// near the best plan of that share instead of the best of a sparse sample.
// One wave per (source, level); the seed slots are written by this block
// only.  Dynamic LDS: N doubles and N id bytes per lane.
__global__ void __launch_bounds__(64) k_seed_cands(const JobDev* __restrict__ jobs) {
    extern __shared__ double s_dyn64[];
    JD J = cs(jobs + blockIdx.x);
    PD P = cs(J->prob);
    const int k = blockIdx.y, lane = threadIdx.x;
    if (k >= P->k || P->obj) return;
    const int N = P->n, R = P->rmax;
    double* f = s_dyn64 + lane;
    uint8_t* ids = (uint8_t*)(s_dyn64 + (size_t)N * 64) + lane;
    const uint32_t nc = min(*J->ncand, J->cap);
    uint32_t* slot = J->scert + k * NSLOT;
    static_assert(NSLOT == 64, "one seed slot per lane");
    const uint32_t e0 = wave_max_u32(slot[lane]);
    const float sb0 = e0 ? __uint_as_float(e0 - 1u) : -1.0f;
    float sb = sb0;
    const double* lat = P->lat64 + (size_t)k * N * R;
    const float hi = P->hi[k];
    for (uint32_t i = lane; i < nc; i += 64) {
        const Cand c = J->cand[i];
        if (!(c.corr > sb && c.cp <= hi)) continue;
        if (!job_ids(J, P, c.index, ids, 64)) continue;
        double corr, cp, d;
        cert_eval<false>(P, N, R, ids, f, P->a64, P->dem64, lat, corr, cp, d);
        if (cp <= P->slo) sb = c.corr;
    }
    const uint32_t e = wave_max_u32(sb > sb0 ? __float_as_uint(sb) + 1u : 0u);
    if (lane == 0 && e > e0) slot[0] = e;
}

// Overflow recovery: the candidates gathered before the list overflowed
// include certainly-feasible plans; fold their fp32 corr into the seeds (a
// valid threshold comes from any certainly-feasible plan) and reset the list
// for another scoring pass.  One wave per source; uniform pressure only.
__global__ void __launch_bounds__(64) k_reseed(const JobDev* __restrict__ jobs) {
    JD J = cs(jobs + blockIdx.x);
    PD P = cs(J->prob);
    const int lane = threadIdx.x;
    const uint32_t nc = min(*J->ncand, J->cap);
    for (int k = 0; k < P->k; ++k) {
        uint32_t e;
        if (P->obj) {  // every candidate is admissible: its fp32 estimate of J_k
            float sb = -INFINITY;
            for (uint32_t i = lane; i < nc; i += 64) {
                const Cand c = J->cand[i];
                sb = fmaxf(sb, fmaf(-P->m32[k], c.cp, c.corr));
            }
            e = wave_max_u32(sb > -INFINITY ? fkey(sb) : 0u);
        } else {
            float sb = -1.0f;
            for (uint32_t i = lane; i < nc; i += 64) {
                const Cand c = J->cand[i];
                if (c.cp <= P->lo[k]) sb = fmaxf(sb, c.corr);
            }
            e = wave_max_u32(sb >= 0.0f ? __float_as_uint(sb) + 1u : 0u);
        }
        if (lane == 0 && e) atomicMax(J->scert + k * NSLOT, e);
    }
    __syncthreads();
    if (lane == 0) {
        *J->ncand = 0u;
        *J->flags = 0;
    }
}

// ---------------------------------------------------------------------------
// exhaustive fp64 path (candidate overflow, or forced): pass 0 finds the best
// feasible corr of each level, pass 1 the lowest index reaching it
// ---------------------------------------------------------------------------

__global__ void __launch_bounds__(WG) k_exhaust(const JobDev* __restrict__ jobs, int pass) {
    JD J = cs(jobs + blockIdx.y);
    PD P = cs(J->prob);
    if (!J->fb_levels) return;
    const uint64_t units = J->count;
    const uint64_t stride = (uint64_t)gridDim.x * WG;
    uint8_t ids[NMAX];
    double f[NMAX];
    for (int k = 0; k < P->k; ++k) {
        if (!(J->fb_levels >> k & 1u)) continue;
        const uint64_t target = pass ? J->fb_corr[k] : 0ull;
        uint64_t acc = pass ? ~0ull : 0ull;
        for (uint64_t j = (uint64_t)blockIdx.x * WG + threadIdx.x; j < units; j += stride) {
            const uint64_t idx = J->kind == DY_SOURCE_RANGE ? J->begin + j : J->index_base + j;
            if (!job_ids(J, P, idx, ids, 1)) continue;
            uint64_t key;  // ordered, 0 means none
            if (P->obj) {
                double T, D;
                const double U = ex_obj(P, ids, 1, f, 1, T, D);
                key = dkey(obj_j(P->lam_l64, P->m64[k], U, T, D));
            } else {
                const double cp = ex_cp(P, ids, 1, k, f, 1);
                if (!(cp <= P->slo)) continue;
                key = (uint64_t)__double_as_longlong(ex_corr(P, ids, 1)) + 1ull;
            }
            if (!pass) {
                acc = key > acc ? key : acc;
            } else if (key == target && idx < acc) {
                acc = idx;
            }
        }
        for (int o = 32; o > 0; o >>= 1) {
            const uint64_t v = __shfl_xor(acc, o);
            acc = pass ? (v < acc ? v : acc) : (v > acc ? v : acc);
        }
        if ((threadIdx.x & 63) == 0) {
            if (!pass) {
                if (acc) atomicMax((unsigned long long*)(J->fb_corr + k), (unsigned long long)acc);
            } else if (acc != ~0ull) {
                atomicMin((unsigned long long*)(J->fb_index + k), (unsigned long long)acc);
            }
        }
    }
}

__global__ void k_exhaust_final(const JobDev* __restrict__ jobs, int njobs) {
    const int j = blockIdx.x;
    if (j >= njobs) return;
    JD J = cs(jobs + j);
    PD P = cs(J->prob);
    const int k = threadIdx.x;
    if (k >= P->k || !(J->fb_levels >> k & 1u)) return;
    uint8_t ids[NMAX];
    dy_choice* o = J->out + k;
    double f[NMAX];
    if (J->fb_index[k] != ~0ull && job_ids(J, P, J->fb_index[k], ids, 1)) {
        o->index = (int64_t)J->fb_index[k];
        o->feasible = 1;
        if (P->obj) {
            double T, D;
            const double U = ex_obj(P, ids, 1, f, 1, T, D);
            o->corr = (float)obj_j(P->lam_l64, P->m64[k], U, T, D);
            o->cp = (float)T;
            o->demand = (float)D;
        } else {
            o->corr = (float)ex_corr(P, ids, 1);
            o->cp = (float)ex_cp(P, ids, 1, k, f, 1);
            o->demand = (float)ex_demand(P, ids, 1);
        }
    } else {
        o->index = -1;
        o->feasible = 0;
        o->corr = NAN;
        o->cp = NAN;
        o->demand = NAN;
    }
}

// ---------------------------------------------------------------------------
// per-plan scores (dy_plan_score)
// ---------------------------------------------------------------------------

// Tables of the score kernel staged in LDS when N * R_max <= SCORE_TAB entries
// and N <= SCORE_TAB_N: larger DAGs already load the LDS with their id and
// recurrence columns, and read the tables faster through the vector cache.
constexpr int SCORE_TAB = 2048;
constexpr int SCORE_TAB_N = 12;

// LDS of k_score for a problem of n nodes and nr table entries: a per-thread
// column of n floats (the fp32 recurrence), n id bytes per thread, and the
// staged tables.
constexpr uint64_t SCORE_PPT = 8;  // plans per thread of k_score (the tables are staged once per block)
constexpr int SCORE_ROW_TAB = 2048;      // table entries (N x R_max) of k_score_row, staged in LDS
constexpr size_t SCORE_ROW_LDS = 56 << 10;  // its dynamic LDS at most (64 KiB with the static arrays)
constexpr uint64_t SCORE_ROWS_PT = 2;    // rows per thread of k_score_row

static size_t score_lds(int n, int nr) {
    size_t b = (size_t)n * WG * sizeof(float) + (size_t)n * WG;
    b = (b + 15) & ~(size_t)15;
    if (nr <= SCORE_TAB && n <= SCORE_TAB_N) b += (size_t)nr * (sizeof(float2) + sizeof(float));
    return b;
}

__device__ __forceinline__ double wave_max_f64(double v) {
    for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o));
    return v;
}

// fp64 CP at level k of the plan held by lane L of this wave (its ids in the
// LDS column of thread wave_base + L), computed by the whole wave: lane n
// holds node n's f; each node takes the maximum of its predecessors' f (and
// 0) by a wave reduction, then adds its duration.  The maximum is exact, so
// the value equals the definition's node-order recurrence.  Every lane of the
// wave must call it with the same L and k; lane L's result is returned to all.
__device__ double wave_cp64(PD P, const uint8_t* __restrict__ s_id, int L, int k) {
    const int lane = threadIdx.x & 63, N = P->n, R = P->rmax;
    const int owner = (threadIdx.x & ~63) + L;
    double mine = 0.0;
    if (lane < N) mine = P->lat64[((size_t)k * N + lane) * R + s_id[lane * WG + owner]];
    double f = 0.0;
    for (int n = 0; n < N; ++n) {
        const bool pred = lane < n && (P->pred[n] >> lane & 1u);
        const double m = wave_max_f64(pred ? f : 0.0);
        if (lane == n) f = mine + m;
    }
    return wave_max_f64(lane < N && (P->sinks >> lane & 1u) ? f : 0.0);
}

// Exact feasibility of the levels in `amb` (lanes whose fp32 CP fell in a
// band) through wave_cp64, one ambiguous (lane, level) at a time; every lane
// of the wave must take part.  Sets the feasible ones in *bits.
__device__ void resolve_bands(PD P, const uint8_t* __restrict__ s_id, uint32_t amb, uint32_t* bits) {
    const int lane = threadIdx.x & 63;
    uint64_t lanes = __ballot(amb != 0u);
    while (lanes) {
        const int L = __builtin_ctzll(lanes);
        lanes &= lanes - 1;
        uint32_t lk = (uint32_t)__builtin_amdgcn_readlane((int)amb, L);
        while (lk) {
            const int k = __builtin_ctz(lk);
            lk &= lk - 1;
            const bool f = wave_cp64(P, s_id, L, k) <= P->slo;
            if (lane == L && f) *bits |= 1u << k;
        }
    }
}

__global__ void __launch_bounds__(WG) k_score(const JobDev job, uint64_t unit_off, uint64_t unit_end, float* corr,
                                              float* cpo, float* dem, uint32_t* feas) {
    extern __shared__ float s_dyn[];
    JD J = cs(&job);
    PD P = cs(J->prob);
    const int N = P->n, R = P->rmax, tid = threadIdx.x;
    float* s_f = s_dyn;                                    // [N][WG]
    uint8_t* s_id = (uint8_t*)(s_dyn + (size_t)N * WG);    // [N][WG]
    const size_t head = (((size_t)N * WG * sizeof(float) + (size_t)N * WG) + 15) & ~(size_t)15;
    const uint64_t n_units = J->count;  // plans of the source; this launch scores [unit_off, unit_end)
    const uint64_t first = unit_off + (uint64_t)blockIdx.x * WG, stride = (uint64_t)gridDim.x * WG;
    if (first >= unit_end) return;
    // stage the (a, tau) and demand tables
    const int NR = N * R;
    const float2* at = P->at;
    const float* dm = P->dem;
    if (NR <= SCORE_TAB && N <= SCORE_TAB_N) {
        float2* s_at = (float2*)((char*)s_dyn + head);
        float* s_dm = (float*)(s_at + NR);
        for (int i = tid; i < NR; i += WG) {
            s_at[i] = P->at[i];
            s_dm[i] = P->dem[i];
        }
        at = s_at;
        dm = s_dm;
    }
    __syncthreads();
    // several plans per thread (block-uniform loop): the table staging above is paid once
    for (uint64_t base = first; base < unit_end; base += stride) {
        const uint64_t t = base + tid;
        const bool live = t < unit_end;
        bool bad = false;  // a row id out of range (read as 0 here): NaN scores, no feasible level
        load_plan(J, P, live ? t : n_units - 1, s_id, &bad);
        const int K = P->k;
        const bool out = live && !bad;
        // 16-byte stores of the K per-level values when every row of cp is 16-byte aligned
        const bool vec = cpo && (K & 3) == 0 && ((uintptr_t)cpo & 15) == 0;
        auto put_cp = [&](auto&& value) {
            if (!cpo || !live) return;
            float* row = cpo + t * (uint64_t)K;
            if (vec) {
                for (int k = 0; k < K; k += 4)
                    *(float4*)(row + k) = make_float4(value(k), value(k + 1), value(k + 2), value(k + 3));
            } else {
                for (int k = 0; k < K; ++k) row[k] = value(k);
            }
        };
        // fp32 corr (objective mode: U), unpressured CP and demand from the (staged) tables
        float cc = 1.0f, cp0 = 0.0f, d = 0.0f, U = 0.0f;
        for (int n = 0; n < N; ++n) {
            const int e = n * R + s_id[n * WG + tid];
            const float2 v = at[e];
            if (P->obj)
                U = U + v.x;
            else
                cc = cc * v.x;
            d = d + dm[e];
            float m = 0.0f;
            uint32_t pm = P->pred[n];
            while (pm) {
                const int u = __builtin_ctz(pm);
                pm &= pm - 1;
                m = fmaxf(m, s_f[u * WG + tid]);
            }
            const float f = v.y + m;
            s_f[n * WG + tid] = f;
            if (P->sinks >> n & 1u) cp0 = fmaxf(cp0, f);
        }
        if (P->obj) {  // corr = U, cp[k] = the fp32 estimate of J_k, demand = D, every level admissible
            const float G = fmaf(-P->lam_l, cp0, U);
            put_cp([&](int k) { return out ? fmaf(-P->m32[k], d, G) : NAN; });
            if (live) {
                if (corr) corr[t] = out ? U : NAN;
                if (dem) dem[t] = out ? d : NAN;
                if (feas) feas[t] = out ? (K >= 32 ? 0xffffffffu : ((1u << K) - 1u)) : 0u;
            }
            continue;
        }
        // feasibility per level: certain in fp32 outside the band (lo, hi], else
        // the definition's fp64 CP, evaluated by the wave (resolve_bands)
        uint32_t bits = 0, amb = 0;
        if (P->uniform) {
            for (int k = 0; k < K && k < 32; ++k) {
                if (cp0 <= P->lo[k])
                    bits |= 1u << k;
                else if (cp0 <= P->hi[k])
                    amb |= 1u << k;
            }
            resolve_bands(P, s_id, out ? amb : 0u, &bits);
            put_cp([&](int k) { return out ? cp0 * P->mk[k] : NAN; });
        } else {
            // per-backend pressure: each level's own fp32 CP, one level at a time
            for (int k = 0; k < K; ++k) {
                const float cpc = eval_cp_level(P, s_id, s_f, k);
                uint32_t a = 0;
                if (k < 32) {
                    if (cpc <= P->glo)
                        bits |= 1u << k;
                    else if (cpc <= P->ghi)
                        a = 1u << k;
                }
                resolve_bands(P, s_id, out ? a : 0u, &bits);
                if (live && cpo) cpo[t * (uint64_t)K + k] = out ? cpc : NAN;
            }
        }
        if (live) {
            if (corr) corr[t] = out ? cc : NAN;
            if (feas) feas[t] = out ? bits : 0u;
            if (dem) dem[t] = out ? d : NAN;
        }
    }
}

// Per-plan scores of a RANGE source of 32-bit plan indices (uniform pressure
// or the objective) by rows: a row fixes nodes 0..N-2 and its plans are node
// y = N-1's implementations.  Phase 1: each lane takes one row and forms its
// digits, prefix product (objective: sums), demand sum and the longest paths
// into y and into the other sinks, once for the row.  Phase 2: the wave
// scores the plans of its 64 rows, which are one contiguous span of plan
// indices, 64 consecutive plans at a time; each plan adds y's terms to its
// row's, in the same operations and order as the per-plan kernels.  Lane =
// plan for the per-plan outputs; the K per-level values of the 64 plans are
// stored lane-contiguously instead (each plan's scalars pass through LDS), so
// every store instruction covers one contiguous span.  A plan's feasibility bits come from two
// tables per bin of its CP's fp32 pattern (the prefilter's bins): the levels
// every CP of the bin certainly meets, and those some CP of the bin may meet
// without certainty; only the latter are compared with the bands, and a CP
// inside a band (lo_k, hi_k] is decided in fp64 by the wave.
// Dynamic LDS: the recurrence column [N][WG] floats, the ids [N][WG], then the
// (a, tau) and demand tables (N * R_max entries).
template <bool OBJ>
__global__ void __launch_bounds__(WG) k_score_row(const JobDev job, uint64_t row_off, uint64_t row_end, float* corr,
                                                  float* cpo, float* dem, uint32_t* feas) {
    extern __shared__ float s_dyn[];
    __shared__ uint32_t s_cert[NBINS2], s_chk[NBINS2];
    __shared__ float4 s_pre[WG];  // per row: (prefix product or sum, demand sum, path into y, other sinks)
    __shared__ float2 s_v[WG];    // per plan of a step: (cp0, or G in objective mode; demand)
    __shared__ __align__(16) float s_mk[KMAX];  // per level: 1/(1 - rho_k), or lambda_ld L_k
    // the band edges per level: a lane's level index is not uniform, so they
    // are read from LDS (a global load's wait would also wait for the wave's
    // earlier stores)
    __shared__ float s_lo[KMAX], s_hi[KMAX];
    JD J = cs(&job);
    PD P = cs(J->prob);
    const int N = P->n, R = P->rmax, K = P->k, tid = threadIdx.x, lane = tid & 63, wbase = tid & ~63;
    const int y = N - 1, ry = P->radix[y];
    float* s_f = s_dyn;                                    // [N][WG]
    uint8_t* s_id = (uint8_t*)(s_dyn + (size_t)N * WG);    // [N][WG]
    const size_t head = (((size_t)N * WG * sizeof(float) + (size_t)N * WG) + 15) & ~(size_t)15;
    float2* s_at = (float2*)((char*)s_dyn + head);
    float* s_dm = (float*)(s_at + N * R);
    const uint64_t first = row_off + (uint64_t)blockIdx.x * WG, stride = (uint64_t)gridDim.x * WG;
    if (first >= row_end) return;
    for (int i = tid; i < N * R; i += WG) {
        s_at[i] = P->at[i];
        s_dm[i] = P->dem[i];
    }
    if (tid < K) {
        s_mk[tid] = OBJ ? P->m32[tid] : P->mk[tid];
        s_lo[tid] = P->lo[tid];
        s_hi[tid] = P->hi[tid];
    }
    // bins: 256 on shift 18 when they cover the CP range (P->jsh), else 64 on the problem's shift
    const bool b256 = P->jsh != 0;
    const uint32_t sh = b256 ? 18u : (uint32_t)P->bin_shift, nb = b256 ? (uint32_t)NBINS2 : (uint32_t)NBINS;
    if (!OBJ && (uint32_t)tid < nb) {
        const uint32_t blo = P->cp_lo_bits >> sh;
        const uint32_t B = blo + (((uint32_t)tid - blo) & (nb - 1u));
        uint64_t lowb = (uint64_t)B << sh, highb = (((uint64_t)B + 1) << sh) - 1;
        if (lowb < P->cp_lo_bits) lowb = P->cp_lo_bits;
        if (highb > 0x7f7fffffull) highb = 0x7f7fffffull;
        const float low = __uint_as_float((uint32_t)lowb), high = __uint_as_float((uint32_t)highb);
        uint32_t cert = 0, chk = 0;
        for (int k = 0; k < K && k < 32; ++k) {
            if (high <= P->lo[k])
                cert |= 1u << k;
            else if (low <= P->hi[k])
                chk |= 1u << k;
        }
        s_cert[tid] = cert;
        s_chk[tid] = chk;
    }
    const uint64_t row0 = J->begin / (uint64_t)ry, p_end = J->begin + J->count;
    const bool vec = cpo && (K & 3) == 0 && ((uintptr_t)cpo & 15) == 0;
    const uint32_t allk = K >= 32 ? 0xffffffffu : ((1u << K) - 1u);
    const uint32_t py = P->pred[y];
    const uint32_t kinv = (1u << 20) / (uint32_t)K + 1u;  // (f * kinv) >> 20 = f / K for f < 64 K, K <= 32
    for (uint64_t base = first; base < row_end; base += stride) {
        __syncthreads();  // tables staged; the previous batch's rows consumed
        // phase 1: lane = row
        const uint64_t rt = base + tid;
        const uint64_t row = row0 + (rt < row_end ? rt : row_end - 1);
        uint32_t x = (uint32_t)row;
        for (int n = y - 1; n >= 0; --n) {
            const uint32_t q = mdiv(x, P->rmag[n]);
            s_id[n * WG + tid] = (uint8_t)(x - q * (uint32_t)P->radix[n]);
            x = q;
        }
        float cx = OBJ ? 0.0f : 1.0f, dx = 0.0f, M = 0.0f, S2 = 0.0f;
        for (int n = 0; n < y; ++n) {
            const int e = n * R + (int)s_id[n * WG + tid];
            const float2 v = s_at[e];
            cx = OBJ ? cx + v.x : cx * v.x;
            dx = dx + s_dm[e];
            float m = 0.0f;
            uint32_t pm = P->pred[n];
            while (pm) {
                const int u = __builtin_ctz(pm);
                pm &= pm - 1;
                m = fmaxf(m, s_f[u * WG + tid]);
            }
            const float f = v.y + m;
            s_f[n * WG + tid] = f;
            if (py >> n & 1u) M = fmaxf(M, f);
            if (P->sinks >> n & 1u) S2 = fmaxf(S2, f);
        }
        s_pre[tid] = make_float4(cx, dx, M, S2);
        __syncthreads();
        // phase 2: the wave's rows are rows r0 .. r0 + 63 (those below row_end),
        // plans r0 ry .. (r0 + 64) ry - 1; 64 consecutive plans per step
        const uint64_t wrow = base + (uint64_t)wbase;  // the wave's first row (relative to row0)
        if (wrow >= row_end) continue;
        const uint32_t nrows = (uint32_t)min((uint64_t)64, row_end - wrow);
        const uint64_t pw = (row0 + wrow) * (uint64_t)ry;
        for (uint32_t q0 = 0; q0 < nrows * (uint32_t)ry; q0 += 64) {
            const uint32_t q = q0 + (uint32_t)lane;
            const uint32_t lr = mdiv(q, P->rmag[y]);  // local row
            const int j = (int)(q - lr * (uint32_t)ry);
            const uint64_t p = pw + q;
            const bool live = lr < nrows && p >= J->begin && p < p_end;
            const float4 pr = s_pre[wbase + (int)min(lr, nrows - 1)];
            const int e = y * R + j;
            const float2 v = s_at[e];
            const float cc = OBJ ? pr.x + v.x : pr.x * v.x;
            const float d = pr.y + s_dm[e];
            const float cp0 = fmaxf(v.y + pr.z, pr.w);
            const uint64_t o = p - J->begin;
            float G = 0.0f;
            uint32_t bits = allk;
            if (OBJ) {
                G = fmaf(-P->lam_l, cp0, cc);
            } else {
                const uint32_t off = b256 ? (__float_as_uint(cp0) >> 16) & 0x3fcu
                                          : (__float_as_uint(cp0) >> (sh - 2)) & 0xfcu;
                bits = *(const uint32_t*)((const char*)s_cert + off);
                uint32_t chk = *(const uint32_t*)((const char*)s_chk + off), amb = 0;
                while (chk) {
                    const int k = __builtin_ctz(chk);
                    chk &= chk - 1;
                    if (cp0 <= s_lo[k])
                        bits |= 1u << k;
                    else if (cp0 <= s_hi[k])
                        amb |= 1u << k;
                }
                if (!live) amb = 0u;
                if (__ballot(amb != 0u)) {
                    // the plan's ids into this lane's column of a second id array
                    // over s_f (free in this phase): its row's digits, which phase 1
                    // left in the row's column of s_id, and y's id
                    uint8_t* s_pid = (uint8_t*)s_f;
                    const int rc = wbase + (int)min(lr, nrows - 1);
                    for (int n = 0; n < y; ++n) s_pid[n * WG + tid] = s_id[n * WG + rc];
                    s_pid[y * WG + tid] = (uint8_t)j;
                    __builtin_amdgcn_wave_barrier();
                    resolve_bands(P, s_pid, amb, &bits);
                    __builtin_amdgcn_wave_barrier();
                }
            }
            if (live) {
                if (corr) corr[o] = cc;
                if (feas) feas[o] = bits;
                if (dem) dem[o] = d;
            }
            if (!cpo) continue;
            // the K values of each of the 64 plans: uniform pressure cp0 / (1 - rho_k)
            // in fp32 (cp0 * mk[k]), the objective G - lambda_ld L_k d (one fma);
            // each lane stores consecutive floats of the 64 plans' rows, so every
            // store covers one contiguous span
            s_v[tid] = make_float2(OBJ ? G : cp0, d);
            __builtin_amdgcn_wave_barrier();
            const uint32_t nlive = (uint32_t)min((uint64_t)nrows * (uint64_t)ry - q0, (uint64_t)64);
            const uint64_t p0 = pw + q0;  // plan of the step's first lane
            const uint32_t la = p0 < J->begin ? (uint32_t)(J->begin - p0) : 0u;
            const uint32_t lb = p0 >= p_end ? 0u : (uint32_t)min((uint64_t)nlive, p_end - p0);
            const int64_t e0 = ((int64_t)p0 - (int64_t)J->begin) * K;  // output float of the step's lane 0 (>= 0 from lane la on)
            if (vec) {
                for (int m = 0; m < K; m += 4) {
                    const uint32_t f = 4u * (uint32_t)lane + 64u * (uint32_t)m;  // float within the 64 rows
                    const uint32_t pl = (f * kinv) >> 20, k = f - pl * (uint32_t)K;
                    if (pl < la || pl >= lb) continue;
                    const float2 u = s_v[wbase + (int)pl];
                    const float4 c = *(const float4*)(s_mk + k);
                    const float4 w = OBJ ? make_float4(fmaf(-c.x, u.y, u.x), fmaf(-c.y, u.y, u.x), fmaf(-c.z, u.y, u.x),
                                                       fmaf(-c.w, u.y, u.x))
                                         : make_float4(u.x * c.x, u.x * c.y, u.x * c.z, u.x * c.w);
                    *(float4*)(cpo + e0 + f) = w;
                }
            } else {
                for (int m = 0; m < K; ++m) {
                    const uint32_t f = (uint32_t)lane + 64u * (uint32_t)m;
                    const uint32_t pl = (f * kinv) >> 20, k = f - pl * (uint32_t)K;
                    if (pl < la || pl >= lb) continue;
                    const float2 u = s_v[wbase + (int)pl];
                    cpo[e0 + f] = OBJ ? fmaf(-s_mk[k], u.y, u.x) : u.x * s_mk[k];
                }
            }
            __builtin_amdgcn_wave_barrier();  // s_v is rewritten by the next step
        }
    }
}

// ---------------------------------------------------------------------------
// launch wrappers (host)
// ---------------------------------------------------------------------------

static constexpr uint64_t MAX_GRID_X = 1ull << 22;  // workgroups per launch along x

// per-thread LDS columns of the generic kernels: ncol floats and ncol id bytes
static size_t generic_lds(int ncol) { return (size_t)ncol * WG * sizeof(float) + (size_t)ncol * WG; }

// ---------------------------------------------------------------------------
// Fixed per-call device memory for callers that cannot allocate
// ---------------------------------------------------------------------------

// The per-call buffers of dy_plan_select_static (seed slots, thresholds,
// prefilter tables, candidate lists, certification state, choices and the
// job array) live here instead of in memory the library allocates.  Every GPU
// the library runs on holds its own copy, at its own address, until the
// process ends; every such call on a GPU shares it.
constexpr size_t STATIC_SCRATCH_BYTES = 16u << 20;
static __device__ __align__(256) unsigned char scratch[STATIC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

// Device address of this device's `scratch` (the current device must be
// `device`): taken once per device with hipGetSymbolAddress and kept.  The
// array's name in host code is a host-side stand-in, never a device address.
hipError_t static_scratch(int device, char** ptr, size_t* bytes) {
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch_ptr[device] = (char*)p;
    }
    *ptr = g_scratch_ptr[device];
    *bytes = STATIC_SCRATCH_BYTES;
    return hipSuccess;
}

hipError_t launch_init(JobDev* d_jobs, int njobs, hipStream_t s) {
    hipLaunchKernelGGL(k_init, dim3(njobs), dim3(64), 0, s, d_jobs, njobs);
    return hipGetLastError();
}

// Problems above CLIMB_NODES nodes take no climb (the kernel returns for them).
// modes: bit 0 sources of corr / SLO problems climb, bit 1 of objective ones,
// bit 2 every corr / SLO one is under uniform pressure.
// The unrolled plan (NN registers per node array, NN (NN - 1) / 2 predecessor
// tests per evaluated move) is sized by the launch's largest DAG: 6 nodes or
// fewer take NN = 6, else NN = CLIMB_NODES.
template <int NN>
static hipError_t launch_climb_nn(const JobDev* d_jobs, int njobs, int kmax, int modes, int E, hipStream_t s) {
    // few (source, level) pairs: 16 waves each (latency); many: one wave
    // each, four to a block (a CU holds few blocks, so one-wave blocks would
    // leave it short of waves)
    const int nsearch = njobs * kmax;
    const bool coop = nsearch <= 1024;
    const dim3 grid = coop ? dim3(kmax, njobs) : dim3((unsigned)((nsearch + 3) / 4));
    const dim3 block(coop ? 1024 : 256);
    const int slots = coop ? 1 : 4;
    // corr mode, many sources, each under uniform pressure: one wave per
    // source climbs its levels in turn
    if ((modes & 1) && (modes & 4) && !coop)
        hipLaunchKernelGGL((k_climb<NN, false, true>), dim3((unsigned)((njobs + 3) / 4)), block,
                           slots * climb_slot_bytes(E, false), s, d_jobs, njobs, kmax, E);
    else if (modes & 1)
        hipLaunchKernelGGL((k_climb<NN, false>), grid, block, slots * climb_slot_bytes(E, false), s, d_jobs,
                           nsearch, kmax, E);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !(modes & 2)) return e;
    // objective mode, many sources: one wave per source climbs its levels in
    // turn (every plan is admissible at every level)
    if (!coop)
        hipLaunchKernelGGL((k_climb<NN, true, true>), dim3((unsigned)((njobs + 3) / 4)), block,
                           slots * climb_slot_bytes(E, true), s, d_jobs, njobs, kmax, E);
    else
        hipLaunchKernelGGL((k_climb<NN, true>), grid, block, slots * climb_slot_bytes(E, true), s, d_jobs, nsearch,
                           kmax, E);
    return hipGetLastError();
}

hipError_t launch_climb(const JobDev* d_jobs, int njobs, int kmax, int modes, int entries, int nodes, hipStream_t s) {
    if (njobs == 0) return hipSuccess;
    const int E = std::min(std::max(entries, 1), CLIMB_ENTRIES);
    return nodes <= 6 ? launch_climb_nn<6>(d_jobs, njobs, kmax, modes, E, s)
                      : launch_climb_nn<CLIMB_NODES>(d_jobs, njobs, kmax, modes, E, s);
}

hipError_t launch_table(JobDev* d_jobs, int njobs, hipStream_t s) {
    hipLaunchKernelGGL(k_table, dim3(njobs), dim3(64), 0, s, d_jobs, njobs);
    return hipGetLastError();
}

// sweep jobs: [first, first + n) of d_jobs, all with the same HAS_S2
hipError_t launch_sample_sweep(const JobDev* d_jobs, int n, bool has_s2, bool obj, uint64_t max_samples,
                               int npre_max, int npre_c, int kmax, hipStream_t s) {
    if (n == 0) return hipSuccess;
    const uint64_t gx = (max_samples + WG - 1) / WG;
    if (gx == 0) return hipSuccess;
    if (gx > MAX_GRID_X) return hipErrorInvalidValue;
    const size_t lds = (size_t)((npre_max > 0 ? npre_max : 1) + kmax) * WG * sizeof(float) +
                       (size_t)PAT_MAX * (sizeof(float2) + (obj ? sizeof(float) : 0));
    const dim3 grid((uint32_t)gx, n);
#define DYP_SAMPLE(S2, NP)                                                                                 \
    do {                                                                                                   \
        if (obj)                                                                                           \
            hipLaunchKernelGGL((k_sample_sweep_obj<S2, NP>), grid, dim3(WG), lds, s, d_jobs);             \
        else                                                                                               \
            hipLaunchKernelGGL((k_sample_sweep<S2, NP>), grid, dim3(WG), lds, s, d_jobs);                 \
    } while (0)
#define DYP_SAMPLE_NP(S2)       \
    switch (npre_c) {           \
        case 2: DYP_SAMPLE(S2, 2); break; \
        case 4: DYP_SAMPLE(S2, 4); break; \
        case 6: DYP_SAMPLE(S2, 6); break; \
        case 8: DYP_SAMPLE(S2, 8); break; \
        default: DYP_SAMPLE(S2, 0); break; \
    }
    if (has_s2) {
        DYP_SAMPLE_NP(true)
    } else {
        DYP_SAMPLE_NP(false)
    }
#undef DYP_SAMPLE_NP
#undef DYP_SAMPLE
    return hipGetLastError();
}

hipError_t launch_sweep(const JobDev* d_jobs, int n, bool has_s2, bool obj, uint64_t max_units, int npre_max,
                        int npre_c, int ry, bool b256, bool rad12, int pat, hipStream_t s) {
    if (n == 0) return hipSuccess;
    // prefix rows staged in LDS: the group's largest table (npre x rmax
    // entries), at least one entry, at most PAT_MAX (larger ones are read
    // from global memory); f_n columns only without a compile-time prefix length
    int pat_cap = std::min(std::max(pat, 1), PAT_MAX);
    const bool fixed = npre_c == 2 || npre_c == 4 || npre_c == 6 || npre_c == 8;
    const size_t lds = (fixed ? (size_t)0 : (size_t)(npre_max > 0 ? npre_max : 1) * WG * sizeof(float)) +
                       (size_t)pat_cap * (sizeof(float2) + (obj ? sizeof(float) : 0));
    for (uint64_t off = 0; off < max_units; off += MAX_GRID_X * WG) {
        uint64_t left = max_units - off;
        uint64_t gx = (left + WG - 1) / WG;
        if (gx > MAX_GRID_X) gx = MAX_GRID_X;
        const dim3 grid((uint32_t)gx, n);
#define DYP_SWEEP(S2, RYV, NP)                                                                             \
    do {                                                                                                   \
        if (obj && b256 && rad12 && RYV == 12 && NP > 0)                                                   \
            hipLaunchKernelGGL((k_sweep_obj<S2, RYV, NP, true, (RYV == 12 && NP > 0) ? 12 : 0>), grid, dim3(WG), \
                               lds, s, d_jobs, off, pat_cap);                                              \
        else if (obj && b256)                                                                              \
            hipLaunchKernelGGL((k_sweep_obj<S2, RYV, NP, true, 0>), grid, dim3(WG), lds, s, d_jobs, off,   \
                               pat_cap);                                                                   \
        else if (obj)                                                                                      \
            hipLaunchKernelGGL((k_sweep_obj<S2, RYV, NP>), grid, dim3(WG), lds, s, d_jobs, off, pat_cap); \
        else if (b256 && rad12 && RYV == 12 && NP > 0)                                                     \
            hipLaunchKernelGGL((k_sweep<S2, RYV, NP, true, (RYV == 12 && NP > 0) ? 12 : 0>), grid, dim3(WG), lds, \
                               s, d_jobs, off, pat_cap);                                                   \
        else if (b256)                                                                                     \
            hipLaunchKernelGGL((k_sweep<S2, RYV, NP, true, 0>), grid, dim3(WG), lds, s, d_jobs, off, pat_cap); \
        else                                                                                               \
            hipLaunchKernelGGL((k_sweep<S2, RYV, NP, false, 0>), grid, dim3(WG), lds, s, d_jobs, off, pat_cap); \
    } while (0)
#define DYP_SWEEP_NP(S2, RYV)            \
    switch (npre_c) {                    \
        case 2: DYP_SWEEP(S2, RYV, 2); break; \
        case 4: DYP_SWEEP(S2, RYV, 4); break; \
        case 6: DYP_SWEEP(S2, RYV, 6); break; \
        case 8: DYP_SWEEP(S2, RYV, 8); break; \
        default: DYP_SWEEP(S2, RYV, 0); break; \
    }
        if (ry == 12) {
            if (has_s2) {
                DYP_SWEEP_NP(true, 12)
            } else {
                DYP_SWEEP_NP(false, 12)
            }
        } else {
            if (has_s2) {
                DYP_SWEEP_NP(true, 0)
            } else {
                DYP_SWEEP_NP(false, 0)
            }
        }
#undef DYP_SWEEP_NP
#undef DYP_SWEEP
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_sample_generic(const JobDev* d_jobs, int n, uint64_t max_samples, int ncol, hipStream_t s) {
    if (n == 0) return hipSuccess;
    uint64_t gx = (max_samples + WG - 1) / WG;
    if (gx == 0) return hipSuccess;
    if (gx > MAX_GRID_X) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_sample_generic, dim3((uint32_t)gx, n), dim3(WG), generic_lds(ncol), s, d_jobs, ncol);
    return hipGetLastError();
}

hipError_t launch_scan(const JobDev* d_jobs, int n, uint64_t max_units, int ncol, hipStream_t s) {
    if (n == 0) return hipSuccess;
    for (uint64_t off = 0; off < max_units; off += MAX_GRID_X * WG) {
        uint64_t left = max_units - off;
        uint64_t gx = (left + WG - 1) / WG;
        if (gx > MAX_GRID_X) gx = MAX_GRID_X;
        hipLaunchKernelGGL(k_scan, dim3((uint32_t)gx, n), dim3(WG), generic_lds(ncol), s, d_jobs, off, ncol);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_certify(const JobDev* d_jobs, int njobs, int waves, int kmax, int nmax, int nrmax, hipStream_t s) {
    // LDS sized by the plan's largest DAG (a fixed 58 KB let two blocks share a CU)
    const int tab_d = 3 * nrmax * (int)sizeof(double) <= CERT_LDS_TABLES ? 3 * nrmax : 0;
    // one wave per (source, level): four to a block, CERT_PACK_CACHE
    // candidates cached per wave (the rest are read from global memory), the
    // fp64 tables in LDS up to 8 KB per wave, at most 64 KB per block
    const int tab_p = 3 * nrmax * (int)sizeof(double) <= 8192 ? 3 * nrmax : 0;
    const size_t lds_p = 4 * cert_slot_doubles(tab_p, nmax, CERT_PACK_CACHE) * sizeof(double);
    if (waves == 1 && lds_p <= 65536) {
        const int nsearch = njobs * kmax;
        hipLaunchKernelGGL(k_certify<true>, dim3((unsigned)((nsearch + 3) / 4)), dim3(256), lds_p, s, d_jobs, tab_p,
                           nmax, CERT_PACK_CACHE, nsearch, kmax);
        return hipGetLastError();
    }
    const size_t lds = cert_slot_doubles(tab_d, nmax, CERT_CACHE) * sizeof(double);
    hipLaunchKernelGGL(k_certify<false>, dim3(waves, njobs, kmax), dim3(64), lds, s, d_jobs, tab_d, nmax, CERT_CACHE,
                       0, kmax);
    return hipGetLastError();
}

// k_seed_cands, then the thresholds and tables rebuilt from the new seeds
hipError_t launch_seed_cands(const JobDev* d_jobs, int njobs, int kmax, int nmax, hipStream_t s) {
    if (njobs == 0) return hipSuccess;
    const size_t lds = (size_t)nmax * 64 * (sizeof(double) + 1);
    hipLaunchKernelGGL(k_seed_cands, dim3(njobs, kmax), dim3(64), lds, s, d_jobs);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_retable, dim3(njobs), dim3(64), 0, s, const_cast<JobDev*>(d_jobs), njobs);
    return hipGetLastError();
}

hipError_t launch_reseed(const JobDev* d_jobs, int njobs, hipStream_t s) {
    hipLaunchKernelGGL(k_reseed, dim3(njobs), dim3(64), 0, s, d_jobs);
    return hipGetLastError();
}

hipError_t launch_exhaust(const JobDev* d_jobs, int njobs, uint64_t max_units, hipStream_t s) {
    uint64_t gx = (max_units + WG - 1) / WG;
    if (gx > 4096) gx = 4096;
    if (gx == 0) gx = 1;
    for (int pass = 0; pass < 2; ++pass) {
        hipLaunchKernelGGL(k_exhaust, dim3((uint32_t)gx, njobs), dim3(WG), 0, s, d_jobs, pass);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(k_exhaust_final, dim3(njobs), dim3(KMAX), 0, s, d_jobs, njobs);
    return hipGetLastError();
}

// ry: implementations of the DAG's last node (the plans of one row)
hipError_t launch_score(const JobDev& job, uint64_t units, float* corr, float* cp, float* dem, uint32_t* feas,
                        int n_nodes, int n_entries, int ry, bool simple, bool obj, hipStream_t s) {
    const size_t lds = score_lds(n_nodes, n_entries);
    // rows of plans (nodes 0..N-2 fixed, y = N-1 swept; one row for a 1-node
    // DAG): RANGE sources of 32-bit indices, uniform pressure or the
    // objective, tables small enough for LDS
    const size_t head = (((size_t)n_nodes * WG * sizeof(float) + (size_t)n_nodes * WG) + 15) & ~(size_t)15;
    const size_t lds_row = head + (size_t)n_entries * (sizeof(float2) + sizeof(float));
    if (simple && job.kind == DY_SOURCE_RANGE && !job.big && n_entries <= SCORE_ROW_TAB && lds_row <= SCORE_ROW_LDS) {
        const uint64_t rows = (job.begin + job.count - 1) / (uint64_t)ry - job.begin / (uint64_t)ry + 1;
        for (uint64_t off = 0; off < rows; off += MAX_GRID_X * WG) {
            const uint64_t end = rows - off < MAX_GRID_X * WG ? rows : off + MAX_GRID_X * WG;
            const uint64_t gx = (end - off + WG * SCORE_ROWS_PT - 1) / (WG * SCORE_ROWS_PT);
            if (obj)
                hipLaunchKernelGGL(k_score_row<true>, dim3((uint32_t)gx), dim3(WG), lds_row, s, job, off, end, corr, cp,
                                   dem, feas);
            else
                hipLaunchKernelGGL(k_score_row<false>, dim3((uint32_t)gx), dim3(WG), lds_row, s, job, off, end, corr, cp,
                                   dem, feas);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
        return hipSuccess;
    }
    // everything else (rows, per-backend pressure, 64-bit indices, large
    // tables): the generic per-plan kernel
    for (uint64_t off = 0; off < units; off += MAX_GRID_X * WG) {
        const uint64_t end = units - off < MAX_GRID_X * WG ? units : off + MAX_GRID_X * WG;
        const uint64_t gx = (end - off + WG * SCORE_PPT - 1) / (WG * SCORE_PPT);
        hipLaunchKernelGGL(k_score, dim3((uint32_t)gx), dim3(WG), lds, s, job, off, end, corr, cp, dem, feas);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace dyp
