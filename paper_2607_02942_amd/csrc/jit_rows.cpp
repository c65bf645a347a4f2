// DAG-specialised kernels for candidate rows (streamed plans), generated as
// HIP source from one problem's structure and compiled at first use with
// hiprtc for the running device; the same module holds a per-plan score
// kernel for rows (gen_score).
//
// A row is N bytes, byte n = implementation id of node n.  Every node's table
// (factor a = 1 - w(1 - p) and duration tau, fp32) sits in LDS as 64 float2
// entries, so one ds_read_b64 per node fetches both values; on gfx950 a
// random 8-byte LDS read costs about half the issue time of a lane permute
// and a quarter of the two permutes it replaces.  The read address is the
// whole byte times 8 (one shift with a byte-select operand) plus the node's
// table offset in the instruction's immediate field.  The recurrence is unrolled
// in node order with every f_n in a register: N-1 multiplies, one add per
// node and one max per extra predecessor.  The rows stream through plain
// dword loads (on gfx950 non-temporal loads of 24-byte rows stream about 10%
// slower), three rows in flight while one is scored.
//
// Ids outside [0, R_n) are caught per byte without a lookup, two operations
// per word: bit 7 of byte n of (w + sum_n (128 - R_n) 256^n) | w is set iff
// b_n >= R_n.  For b_n < 128 the sum b_n + 128 - R_n stays below 256 (R_n <=
// 64, so no carry leaves the byte, and a carry coming in from a byte below
// cannot clear bit 7 of a byte that already has it); b_n >= 128 sets bit 7 of
// w itself.  The table array has 192 entries past node N-1's table, so a
// read for any byte value stays inside the array (an id >= 64 reads a later
// node's entries or the spare ones; its lane is dropped as invalid).  The
// arithmetic is that of the generic kernels (same fp32 operations in the
// same order), so both produce identical scores.
//
// Objective mode (the paper's additive objective): the tables hold (u, tau);
// a row's U and D are the sums of the LLM nodes' u and tau in node order, T
// the same recurrence, G = U - lambda_l T in one rounding, and the prefilter
// bin is that of D.  No early abandon: every row is evaluated in full.
#include <hip/hip_runtime.h>
#include <hip/hiprtc.h>

#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <sstream>
#include <string>
#include <vector>

#include "dyplan_internal.h"

namespace dyp {

struct JitRows {
    hipModule_t mod = nullptr;
    hipFunction_t scan = nullptr;     // rows whose words are dword aligned
    hipFunction_t scan_u = nullptr;   // any other stride / alignment (byte loads)
    hipFunction_t sample = nullptr;
    hipFunction_t score_rows = nullptr;  // per-plan scores of rows
    hipFunction_t sweep = nullptr;    // the sweep of RANGE sources (32-bit blocks)
    hipFunction_t seed = nullptr;     // its seeding pass (uniform pressure, corr mode)
};

namespace {

std::mutex g_mu;
std::map<std::string, JitRows> g_cache;  // key: device id + generated source

const char* kCommon = R"(
struct DyCand { unsigned long long index; float corr; float cp; };
__device__ __forceinline__ unsigned dy_wmax(unsigned v) {
  v = max(v, (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, false));
  v = max(v, (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, false));
  v = max(v, (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x113, 0xf, 0xf, false));
  v = max(v, (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xe, false));
  v = max(v, (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xc, false));
  v = max(v, (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false));
  v = max(v, (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false));
  return (unsigned)__builtin_amdgcn_readlane((int)v, 63);
}
// Per-wave candidate queue in LDS: the scoring loop issues no global atomic or
// store (those would make it wait for the rows in flight).  The queue goes to
// the global candidate list at the end; a full queue raises the overflow flag,
// which the host resolves exactly by reseeding and rescoring the source.
#define DY_QCAP 128
#define DY_RQCAP 64
__device__ void dy_flush(DyCand* q, unsigned qn, int lane, DyCand* cand, unsigned cap, unsigned* ncand,
                         bool* ovf) {
  if (qn == 0) return;
  unsigned base = 0;
  if (lane == 0) base = atomicAdd(ncand, qn);
  base = (unsigned)__builtin_amdgcn_readfirstlane((int)base);
  for (unsigned i = lane; i < qn; i += 64) {
    if (base + i < cap) cand[base + i] = q[i];
  }
  if (base + qn > cap) *ovf = true;
}
// Row of sample t (t < ceil(n / S)): the 64 samples of a wave read 64
// consecutive rows of the window [64 S g, min(64 S (g + 1), n)), g = t / 64,
// from a hashed offset and wrapping inside the window: whole cache lines of
// rows, where one row per window of S would fetch a line for each 24 bytes.
__device__ __forceinline__ unsigned long long dy_sample_row(unsigned long long t, unsigned long long S,
                                                            unsigned long long n) {
  const unsigned long long g = t >> 6, start = g * 64ull * S;
  const unsigned long long width = min(64ull * S, n - start);
  const unsigned h = (unsigned)(g * 0x9E3779B1ull) >> 16;
  unsigned long long r = (unsigned long long)(h % (unsigned)min(width, 0xffffffffull)) + (t & 63ull);
  if (r >= width) r %= width;
  return start + r;
}
)";

// a float as an exact hexadecimal literal
std::string flit(float x) {
    char buf[48];
    std::snprintf(buf, sizeof buf, "%af", (double)x);
    return buf;
}

float u2f(unsigned u) {
    float f;
    std::memcpy(&f, &u, 4);
    return f;
}

// nodes after which the scoring pass may abandon a wave's rows: past the
// middle of the DAG, where the remaining factors can no longer lift most rows
std::vector<int> checkpoints(int N) {
    std::vector<int> cuts;
    if (N < 8) return cuts;
    for (int m : {N / 2 - 1, N / 2 + 1, N / 2 + 3, (3 * N) / 4})
        if (m >= 2 && m < N - 1 && (cuts.empty() || m > cuts.back())) cuts.push_back(m);
    return cuts;
}

// fp64 literal
std::string dlit(double x) {
    char buf[48];
    std::snprintf(buf, sizeof buf, "%a", x);
    return buf;
}

// f_n = tau_n + max over predecessors, nodes [n0, n1), unrolled
void emit_recurrence(std::ostringstream& o, const ProbDev& D, int n0, int n1) {
    for (int n = n0; n < n1; ++n) {
        std::vector<int> preds;
        for (int u = 0; u < n; ++u)
            if (D.pred[n] >> u & 1u) preds.push_back(u);
        o << "  const float f" << n << " = e" << n << ".y";
        if (!preds.empty()) {
            std::string m = "f" + std::to_string(preds[0]);
            for (size_t k = 1; k < preds.size(); ++k) m = "fmaxf(" + m + ", f" + std::to_string(preds[k]) + ")";
            o << " + " << m;
        }
        o << "; \\\n";
    }
}

// dst = max of f_n over the sinks (declared here when `declare`)
void emit_sinks(std::ostringstream& o, const ProbDev& D, const char* dst, bool declare) {
    bool first = true;
    for (int n = 0; n < D.n; ++n) {
        if (!(D.sinks >> n & 1u)) continue;
        if (first)
            o << "  " << (declare ? "float " : "") << dst << " = f" << n << "; \\\n";
        else
            o << "  " << dst << " = fmaxf(" << dst << ", f" << n << "); \\\n";
        first = false;
    }
}

// objective mode: u_ = sum of the LLM nodes' utilities, d_ = sum of their
// durations (their d), in node order; tool nodes add nothing
void emit_obj_sums(std::ostringstream& o, const ProbDev& D, int n0, int n1) {
    o << "  float u_ = 0.0f, d_ = 0.0f; \\\n";
    for (int n = n0; n < n1; ++n)
        if (D.llm >> n & 1u) o << "  u_ = u_ + e" << n << ".x; d_ = d_ + e" << n << ".y; \\\n";
}

// Per-plan scores of rows (the values of the library's score kernels, same
// fp32 operations in the same order) with the DAG's recurrence unrolled and
// the level constants as literals (dy_score_rows: a row with an id >= R_n gets
// NaN scores and no feasible level, as in the generic kernel).  corr / SLO
// mode: a plan whose fp32 CP falls in a level's band (lo_k, hi_k] takes that
// level's fp64 recurrence here, from the fp64 duration table, against the SLO.
void gen_score(std::ostringstream& o, const ProbDev& D) {
    const int N = D.n, K = D.k, Q = (N + 3) / 4;
    o << R"(
extern "C" __global__ void __launch_bounds__(256) dy_score_rows(
    const unsigned char* __restrict__ rows, unsigned long long stride, unsigned long long count, int aligned,
    const float2* __restrict__ at, const float* __restrict__ dm, int rmax, const double* __restrict__ lat64,
    float* __restrict__ corr, float* __restrict__ cpo, float* __restrict__ demo, unsigned* __restrict__ feas,
    int vec) {)";
    o << R"(
  __shared__ float2 s_tab[DY_TAB];
  __shared__ float s_dm[DY_TAB];
  for (int i = threadIdx.x; i < DY_TAB; i += blockDim.x) {
    const int n = i >> 6, e = i & 63;
    s_dm[i] = n < DY_N && e < rmax ? dm[n * rmax + e] : 0.0f;
  }
  dy_stage(at, rmax, nullptr, s_tab, nullptr);
  const unsigned long long gstride = (unsigned long long)gridDim.x * 256ull;
  for (unsigned long long t = (unsigned long long)blockIdx.x * 256ull + threadIdx.x; t < count; t += gstride) {
)";
    o << "    unsigned ";
    for (int q = 0; q < Q; ++q) o << (q ? ", " : "") << "w" << q;
    o << ";\n    DY_LOAD(t";
    for (int q = 0; q < Q; ++q) o << ", w" << q;
    o << ")\n    unsigned bk_ = 0u;\n";
    for (int q = 0; q < Q; ++q) o << "    bk_ |= (w" << q << " + DY_K_" << q << ") | w" << q << ";\n";
    o << "    const bool bad = (bk_ & 0x80808080u) != 0u;\n";
    for (int n = 0; n < N; ++n) {
        o << "    const unsigned d" << n << " = ";
        if (n % 4) o << "(w" << n / 4 << " >> " << 8 * (n % 4) << ") & 255u;\n";
        else o << "w" << n / 4 << " & 255u;\n";
    }
    // ids below 256: the tables' spare entries keep every read in the arrays
    for (int n = 0; n < N; ++n) o << "    const float2 e" << n << " = s_tab[" << n * 64 << " + d" << n << "];\n";
    o << "    float dd = 0.0f;\n";
    for (int n = 0; n < N; ++n) o << "    dd = dd + s_dm[" << n * 64 << " + d" << n << "];\n";
    o << "    float c = " << (D.obj ? "0.0f" : "1.0f") << ";\n";
    for (int n = 0; n < N; ++n) o << "    c = c " << (D.obj ? "+" : "*") << " e" << n << ".x;\n";
    {
        std::ostringstream r;
        emit_recurrence(r, D, 0, N);
        emit_sinks(r, D, "cp", true);
        std::string body = r.str(), line;
        std::istringstream in(body);
        while (std::getline(in, line)) {  // drop the macro line continuations
            if (line.size() >= 2 && line.compare(line.size() - 2, 2, " \\") == 0) line.resize(line.size() - 2);
            o << "  " << line << "\n";
        }
    }
    o << "    const float nan_ = __builtin_nanf(\"\");\n";
    o << "    if (corr) corr[t] = bad ? nan_ : c;\n    if (demo) demo[t] = bad ? nan_ : dd;\n";
    if (D.obj) {
        o << "    const float G = fmaf(-" << flit(D.lam_l) << ", cp, c);\n";
        o << "    if (feas) feas[t] = bad ? 0u : " << (K >= 32 ? 0xffffffffu : ((1u << K) - 1u)) << "u;\n";
        o << "    if (cpo) {\n      float* row = cpo + t * " << K << "ull;\n";
        for (int k = 0; k < K; ++k) o << "      row[" << k << "] = bad ? nan_ : fmaf(-" << flit(D.m32[k]) << ", dd, G);\n";
        o << "    }\n";
    } else {
        o << "    unsigned bits = 0u, amb = 0u;\n";
        for (int k = 0; k < K && k < 32; ++k)
            o << "    if (cp <= " << flit(D.lo[k]) << ") bits |= " << (1u << k) << "u; else if (cp <= " << flit(D.hi[k])
              << ") amb |= " << (1u << k) << "u;\n";
        o << "    if (bad) bits = amb = 0u;\n";
        o << "    for (int k = 0; k < " << std::min(K, 32) << " && amb; ++k) {\n";
        o << "      if (!(amb >> k & 1u)) continue;\n";
        o << "      amb &= ~(1u << k);\n";
        o << "      const double* L = lat64 + (unsigned long long)k * " << N << "ull * (unsigned long long)rmax;\n";
        for (int n = 0; n < N; ++n) {
            std::vector<int> preds;
            for (int u = 0; u < n; ++u)
                if (D.pred[n] >> u & 1u) preds.push_back(u);
            o << "      const double g" << n << " = L[" << n << " * rmax + (int)d" << n << "]";
            if (!preds.empty()) {
                std::string m = "g" + std::to_string(preds[0]);
                for (size_t q = 1; q < preds.size(); ++q) m = "fmax(" + m + ", g" + std::to_string(preds[q]) + ")";
                o << " + " << m;
            }
            o << ";\n";
        }
        std::string c64;
        for (int n = 0; n < N; ++n)
            if (D.sinks >> n & 1u) c64 = c64.empty() ? "g" + std::to_string(n) : "fmax(" + c64 + ", g" + std::to_string(n) + ")";
        o << "      if (" << c64 << " <= " << dlit(D.slo) << ") bits |= 1u << k;\n    }\n";
        o << "    if (feas) feas[t] = bits;\n";
        o << "    if (cpo) {\n      float* row = cpo + t * " << K << "ull;\n";
        o << "      const float cq = bad ? nan_ : cp;\n";
        if (K % 4 == 0) {
            o << "      if (vec) {\n";
            for (int k = 0; k < K; k += 4)
                o << "        *(float4*)(row + " << k << ") = make_float4(cq * " << flit(D.mk[k]) << ", cq * " << flit(D.mk[k + 1])
                  << ", cq * " << flit(D.mk[k + 2]) << ", cq * " << flit(D.mk[k + 3]) << ");\n";
            o << "      } else {\n";
        }
        for (int k = 0; k < K; ++k) o << "        row[" << k << "] = cq * " << flit(D.mk[k]) << ";\n";
        if (K % 4 == 0) o << "      }\n";
        o << "    }\n";
    }
    o << "  }\n}\n";
}

// The prefix-shared sweep for RANGE sources of one problem, block indices
// below 2^32, under uniform pressure (corr / SLO mode) or the objective: the
// library's k_sweep / k_sweep_obj with the DAG fixed at compile time.  A lane
// takes one prefix block (an assignment of nodes 0..N-3): digits by constant
// division, the prefix recurrence with its exact predecessor maxima (no
// per-edge selects), then the inner pair (x, y) swept in lockstep with the y
// table in scalar registers; per plan (corr mode) one multiply, one add (and a
// max for a second sink), the bin's threshold from LDS and a compare.  A row
// with a hit is re-scored with the exact per-level test and its candidates
// appended.  Same fp32 operations in the same order as the library's sweeps,
// so both give identical candidates.
void gen_sweep(std::ostringstream& o, const ProbDev& D) {
    const int NP = D.npre, xn = D.xnode, yn = D.ynode;
    const bool obj = D.obj != 0;
    const bool exy = D.edge_xy != 0, s2 = D.pre_sinks != 0 || !exy;
    const uint32_t pmx = D.pred[xn], pmy = D.pred[yn] & ~(1u << xn), pms = D.pre_sinks;
    // byte offset of the bin's threshold: with 256 bins at shift 18, bits
    // 18..25 of the binned value times 4 = (bits >> 16) & 0x3fc, one masked
    // read of the upper half-word; else the 64 bins at the problem's shift
    const int nb = D.jsh ? NBINS2 : NBINS;
    const int sh = (D.jsh ? D.jsh : D.bin_shift) - 2;
    const unsigned msk = (unsigned)(nb - 1) << 2;
    // corr mode on 256 bins: the bins' thresholds held per implementation of
    // y, divided by its factor (rounded down, so that a plan the product test
    // admits is admitted: see the library's ydiv_threshold); a row's test is
    // then cx >= the least threshold of its plans' bins, every threshold being
    // +0, positive or +inf, so that their fp32 patterns order as the values
    const bool ydiv = !obj && D.jsh != 0 && D.ry >= 1 && D.ry <= 64;
    // objective mode on 256 bins: the first 256 entries hold the bins'
    // thresholds on G, then per implementation j of y the order keys of those
    // thresholds lowered by c_j (see the library's yshift_key); a row's test
    // is the key of its fma(-lambda_l, M, ux) >= the least key of its plans'
    // D bins, and the rare path keeps the per-plan test on G
    const bool ysh = obj && D.jsh != 0 && D.ry >= 1 && D.ry <= 64;
    auto maxof = [&](uint32_t mask, const char* pre) {
        std::string m;
        for (int u = 0; u < NP; ++u)
            if (mask >> u & 1u) m = m.empty() ? std::string(pre) + std::to_string(u) : "fmaxf(" + m + ", " + pre + std::to_string(u) + ")";
        return m.empty() ? std::string("0.0f") : m;
    };
    if (ydiv)
        o << R"(
__device__ __forceinline__ float dy_ydiv(float T, float r) {
  if (T == __builtin_inff()) return T;
  return T > 0x1p-60f ? T * r : 0.0f;
}
)";
    if (ysh)  // dy_skey: signed order key of a float (as the library's skey)
        o << R"(
__device__ __forceinline__ int dy_skey(float x) {
  const int b = __float_as_int(x);
  return b ^ ((b >> 31) & 0x7fffffff);
}
__device__ __forceinline__ int dy_yshift(float t, float c) {
  float x = t;
  if (t != __builtin_inff() && t != -__builtin_inff()) {
    x = t - c;
    if (x != -__builtin_inff()) {
      const unsigned b = __float_as_uint(x);
      if (x > 0.0f) x = __uint_as_float(b - 1u);
      else if (x < 0.0f) x = __uint_as_float(b + 1u);
    }
    if (x == 0.0f) x = -0.0f;
  }
  return dy_skey(x);
}
)";
    o << R"(
extern "C" __global__ void __launch_bounds__(256) dy_sweep(
    unsigned long long unit_off, unsigned long long blk_first, unsigned long long nblk, unsigned long long begin,
    unsigned long long count, const float2* __restrict__ at, const float2* __restrict__ atx,
    const float2* __restrict__ aty, const float* __restrict__ dem, const float* __restrict__ demx,
    const float* __restrict__ demy, const float* __restrict__ lat, int rmax, const unsigned* __restrict__ table,
    const float* __restrict__ thr, DyCand* __restrict__ cand, unsigned cap, unsigned* __restrict__ ncand,
    int* __restrict__ flags, unsigned G) {
  __shared__ float s_bins[)" << (ydiv ? D.ry * NBINS2 : ysh ? (1 + D.ry) * NBINS2 : nb) << R"(];
  __shared__ float2 s_pat[)" << NP << R"( * 64];
)";
    if (obj) o << "  __shared__ float s_pd[" << NP << " * 64];\n";
    o << R"(  const unsigned long long t0 = unit_off + (unsigned long long)blockIdx.x * 256ull;
  const unsigned long long units = nblk / G;  // runs of G blocks that share the prefix but its last node
  if (t0 >= units) return;
)";
    if (ydiv) {
        static_assert(NBINS2 == 256, "one bin per thread");
        o << "  {\n    const float T = __uint_as_float(table[threadIdx.x]);\n";
        for (int j = 0; j < D.ry; ++j)
            o << "    s_bins[" << j * NBINS2 << " + threadIdx.x] = dy_ydiv(T, " << flit(D.yinv[j]) << ");\n";
        o << "  }\n";
    } else if (ysh) {
        o << "  {\n    const float T = __uint_as_float(table[threadIdx.x]);\n    s_bins[threadIdx.x] = T;\n";
        for (int j = 0; j < D.ry; ++j)
            o << "    ((int*)s_bins)[" << (j + 1) * NBINS2 << " + threadIdx.x] = dy_yshift(T, " << flit(D.ysub[j])
              << ");\n";
        o << "  }\n";
    } else {
        o << "  for (int i = threadIdx.x; i < " << nb << "; i += 256) s_bins[i] = __uint_as_float(table[i]);\n";
    }
    o << R"(  for (int i = threadIdx.x; i < )" << NP << R"( * 64; i += 256) {
    const int n = i >> 6, e = i & 63;
    s_pat[i] = e < rmax ? at[n * rmax + e] : make_float2(1.0f, 0.0f);
)";
    if (obj) o << "    s_pd[i] = e < rmax ? dem[n * rmax + e] : 0.0f;\n";
    o << R"(  }
  __syncthreads();
  if (t0 + (threadIdx.x & ~63u) >= units) return;  // a wave past the last run (no barrier follows)
  const unsigned long long t = t0 + threadIdx.x;
  const bool live = t < units;
  const unsigned long long b0 = blk_first + (live ? t : units - 1) * G;
  unsigned x_ = (unsigned)b0;
)";
    for (int n = NP - 1; n >= 0; --n) {
        o << "  const unsigned d" << n << " = x_ % " << D.radix[n] << "u;";
        if (n > 0) o << " x_ /= " << D.radix[n] << "u;";
        o << "\n";
    }
    // prefix: corr mode the product of the factors, objective mode the sums
    // of u and of d (node order, as the library's prefix evaluation)
    // objective mode: runs of G blocks per thread, nodes 0..NP-2 once per
    // run and the last prefix node (digit + g) per block (the prefix sums
    // cost more than corr mode's products, and only they gained); corr
    // mode: one block per thread (G = 1), the whole prefix straight
    const bool runs = obj;
    o << "  float pc = " << (obj ? "0.0f" : "1.0f") << ";\n";
    if (obj) o << "  float pd = 0.0f;\n";
    for (int n = 0; n < NP; ++n) {
        std::string m;
        for (int u = 0; u < n; ++u)
            if (D.pred[n] >> u & 1u) m = m.empty() ? "f" + std::to_string(u) : "fmaxf(" + m + ", f" + std::to_string(u) + ")";
        if (runs && n == NP - 1) {
            o << "  const float ml = " << (m.empty() ? "0.0f" : m) << ";\n";
            o << "  const float pch = pc;\n";
            if (obj) o << "  const float pdh = pd;\n";
            break;
        }
        o << "  const float2 v" << n << " = s_pat[" << n * 64 << " + d" << n << "];\n";
        o << "  pc = pc " << (obj ? "+" : "*") << " v" << n << ".x;\n";
        if (obj) o << "  pd = pd + s_pd[" << n * 64 << " + d" << n << "];\n";
        o << "  const float f" << n << " = v" << n << ".y + " << (m.empty() ? "0.0f" : m) << ";\n";
    }
    o << "  float2 vy[" << D.ry << "];\n";
    if (obj) o << "  float dy[" << D.ry << "];\n";
    o << "#pragma unroll\n  for (int j = 0; j < " << D.ry << "; ++j) {\n    vy[j] = aty[j];\n";
    if (obj) o << "    dy[j] = demy[j];\n";
    o << "  }\n";
    if (!runs) {
        o << "  const unsigned long long b = b0;\n";
    } else {
        o << "#pragma unroll 1\n  for (unsigned g = 0; g < G; ++g) {\n";
        o << "  const unsigned long long b = b0 + g;\n";
        const int n = NP - 1;
        o << "  const float2 v" << n << " = s_pat[" << n * 64 << " + d" << n << " + g];\n";
        o << "  const float pc = pch " << (obj ? "+" : "*") << " v" << n << ".x;\n";
        if (obj) o << "  const float pd = pdh + s_pd[" << n * 64 << " + d" << n << " + g];\n";
        o << "  const float f" << n << " = v" << n << ".y + ml;\n";
    }
    o << "  const float px = " << maxof(pmx, "f") << ", py = " << maxof(pmy, "f") << ", ps = " << maxof(pms, "f")
      << ";\n";
    o << "#pragma unroll 1\n";  // one copy of the row and its rare path (code size)
    o << "  for (int ix = 0; ix < " << D.rx << "; ++ix) {\n";
    o << "    const float2 vx = atx[ix];\n";
    o << "    const float fx = vx.y + px;\n";
    if (obj)
        o << "    const float ux = pc + vx.x;\n    const float dx = pd + demx[ix];\n";
    else
        o << "    const float cx = pc * vx.x;\n";
    o << "    const float M = " << (exy ? "fmaxf(py, fx)" : "py") << ";\n";
    if (s2) o << "    const float S2 = " << (exy ? "ps" : "fmaxf(ps, fx)") << ";\n";
    // one plan: corr mode (cc, cp); objective mode G = u + U_x - lambda_l T
    // (one fused rounding) and D = D_x + d_y, binned by D
    // vy / dy: the register copies of y's entries (unrolled loops), or the
    // tables themselves where the loop is not unrolled (a loop index into the
    // register copy would move the whole array to scratch memory)
    auto plan = [&](const char* ind, const char* vy, const char* dy) {
        o << ind << "float cp = " << vy << "[j].y + M;\n";
        if (s2) o << ind << "cp = fmaxf(cp, S2);\n";
        if (obj) {
            o << ind << "const float cc = fmaf(" << flit(-D.lam_l) << ", cp, ux + " << vy << "[j].x);\n";
            o << ind << "const float bv = dx + " << dy << "[j];\n";
        } else {
            o << ind << "const float cc = cx * " << vy << "[j].x;\n";
            o << ind << "const float bv = cp;\n";
        }
    };
    if (ydiv) {
        // y's implementation j reads its own 256 bins (a constant offset)
        auto thr_j = [&](const char* ind, const char* j) {
            o << ind << "float cp = vy[" << j << "].y + M;\n";
            if (s2) o << ind << "cp = fmaxf(cp, S2);\n";
            o << ind << "const unsigned th = *(const unsigned*)((const char*)s_bins + " << NBINS2 * 4 << " * (" << j
              << ") + ((__float_as_uint(cp) >> 16) & 0x3fcu));\n";
        };
        o << "    unsigned m;\n    {\n";
        thr_j("      ", "0");
        o << "      m = th;\n    }\n";
        o << "#pragma unroll\n    for (int j = 1; j < " << D.ry << "; ++j) {\n";
        thr_j("      ", "j");
        o << "      m = min(m, th);\n    }\n";
        o << "    const bool mine_ = cx >= __uint_as_float(m);\n";
    } else if (ysh) {
        o << "    const float R = fmaf(" << flit(-D.lam_l) << ", M, ux);\n";
        o << "    int m = 0x7fffffff;\n";
        o << "#pragma unroll\n    for (int j = 0; j < " << D.ry << "; ++j) {\n";
        o << "      const float bv = dx + dy[j];\n";
        o << "      m = min(m, *(const int*)((const char*)s_bins + " << NBINS2 * 4
          << " * (j + 1) + ((__float_as_uint(bv) >> 16) & 0x3fcu)));\n    }\n";
        o << "    const bool mine_ = dy_skey(R) >= m;\n";
    } else {
        o << "    unsigned long long hit = 0ull;\n";
        o << "#pragma unroll\n    for (int j = 0; j < " << D.ry << "; ++j) {\n";
        plan("      ", "vy", "dy");
        o << "      const float th = *(const float*)((const char*)s_bins + ((__float_as_uint(bv) >> " << sh << "u) & "
          << msk << "u));\n";
        o << "      hit |= __builtin_amdgcn_ballot_w64(cc >= th);\n    }\n";
        o << "    const bool mine_ = hit && ((hit >> (threadIdx.x & 63)) & 1ull);\n";
    }
    o << "    if (live && mine_) {\n";
    o << "      const unsigned long long base = (b * " << D.rx << "ull + (unsigned long long)ix) * " << D.ry << "ull;\n";
    if (!obj && !D.uniform) {
        // per-backend pressure: per level, the row's exact fp32 CP_k from the
        // level's durations (prefix, x and y), skipped when no plan of the row
        // can reach the level's threshold or its band; a plan is appended
        // once, with its unpressured CP, which the bands refer to
        auto lmax = [&](uint32_t mask) {
            std::string m;
            for (int u = 0; u < NP; ++u)
                if (mask >> u & 1u) m = m.empty() ? "g" + std::to_string(u) : "fmaxf(" + m + ", g" + std::to_string(u) + ")";
            return m.empty() ? std::string("0.0f") : m;
        };
        o << "      const float cmax = cx * " << flit(D.ay_max) << ";\n";
        o << "      float cp0_lb = " << flit(D.ty_min) << " + M;\n";
        if (s2) o << "      cp0_lb = fmaxf(cp0_lb, S2);\n";
        o << "      unsigned long long done = 0ull;\n";
        o << "#pragma unroll 1\n      for (int k = 0; k < DY_K; ++k) {\n";
        o << "        const float th_k = thr[k];\n";
        o << "        if (!(cmax >= th_k && cp0_lb <= dy_hi[k])) continue;\n";
        o << "        const float* L = lat + (unsigned long long)k * DY_N * (unsigned long long)rmax;\n";
        for (int n = 0; n < NP; ++n) {
            std::string m;
            for (int u = 0; u < n; ++u)
                if (D.pred[n] >> u & 1u) m = m.empty() ? "g" + std::to_string(u) : "fmaxf(" + m + ", g" + std::to_string(u) + ")";
            o << "        const float g" << n << " = L[" << n << " * rmax + (int)d" << n << "] + " << (m.empty() ? "0.0f" : m) << ";\n";
        }
        o << "        const float qx = " << lmax(pmx) << ", qy = " << lmax(pmy) << ", qs = " << lmax(pms) << ";\n";
        o << "        const float fxk = L[" << xn << " * rmax + ix] + qx;\n";
        o << "        const float Mk = " << (exy ? "fmaxf(qy, fxk)" : "qy") << ";\n";
        if (s2) o << "        const float S2k = " << (exy ? "qs" : "fmaxf(qs, fxk)") << ";\n";
        // every CP_k of the row above the band when y's fastest entry is
        o << "        if (dy_lymin[k] + Mk > " << flit(D.ghi) << ") continue;\n";
        if (s2) o << "        if (S2k > " << flit(D.ghi) << ") continue;\n";
        // y's entries from memory, not the register copy: a loop index
        // into it would move the whole array to scratch
        // y by decreasing factor: corr falls along the loop, which stops at
        // the first plan below the level's threshold
        o << "#pragma unroll 1\n        for (int jj = 0; jj < " << D.ry << "; ++jj) {\n";
        o << "          const int j = dy_yord[jj];\n";
        o << "          const float2 wy = aty[j];\n";
        o << "          const float cc = cx * wy.x;\n";
        o << "          if (!(cc >= th_k)) break;\n";
        o << "          if (done >> j & 1ull) continue;\n";
        o << "          float cpk = L[" << yn << " * rmax + j] + Mk;\n";
        if (s2) o << "          cpk = fmaxf(cpk, S2k);\n";
        o << "          const unsigned long long idx = base + (unsigned long long)j;\n";
        o << "          if (cpk <= " << flit(D.ghi) << " && idx - begin < count) {\n";
        o << "            float cp0 = wy.y + M;\n";
        if (s2) o << "            cp0 = fmaxf(cp0, S2);\n";
        o << "            done |= 1ull << j;\n";
        o << "            const unsigned slot = atomicAdd(ncand, 1u);\n";
        o << "            if (slot < cap) {\n              cand[slot].index = idx;\n              cand[slot].corr = cc;\n"
             "              cand[slot].cp = cp0;\n            } else {\n              atomicOr(flags, " << (int)JF_OVERFLOW
          << ");\n            }\n          }\n        }\n      }\n    }\n  }\n}\n";
        return;
    }
    o << "      for (int j = 0; j < " << D.ry << "; ++j) {\n";
    plan("        ", "aty", "demy");
    o << "        const unsigned long long idx = base + (unsigned long long)j;\n";
    o << "        bool want = false;\n";
    if (ysh)
        o << "        if (!(cc >= *(const float*)((const char*)s_bins + ((__float_as_uint(bv) >> 16) & 0x3fcu)))) continue;\n";
    for (int k = 0; k < D.k; ++k) {
        if (obj)
            o << "        want = want || (fma(-" << dlit(D.m64[k]) << ", (double)bv, (double)cc) >= (double)thr[" << k << "]);\n";
        else
            o << "        want = want || (cp <= " << flit(D.hi[k]) << " && cc >= thr[" << k << "]);\n";
    }
    o << "        if (idx - begin < count && want) {\n";
    o << "          const unsigned slot = atomicAdd(ncand, 1u);\n";
    o << "          if (slot < cap) {\n            cand[slot].index = idx;\n            cand[slot].corr = cc;\n"
         "            cand[slot].cp = bv;\n          } else {\n            atomicOr(flags, " << (int)JF_OVERFLOW << ");\n"
         "          }\n        }\n      }\n    }\n  }\n" << (runs ? "  }\n" : "") << "}\n";
}

// Seeding pass of the generated sweep (uniform pressure, corr mode): one
// hashed row per window of S rows, as the library's; per level, the best corr
// among the row's plans whose CP bin certainly meets it (the bin's count of
// levels in the seeding order), reduced per workgroup into one slot.
void gen_sweep_seed(std::ostringstream& o, const ProbDev& D) {
    const int NP = D.npre, xn = D.xnode, yn = D.ynode, K = D.k;
    const bool exy = D.edge_xy != 0, s2 = D.pre_sinks != 0 || !exy;
    const uint32_t pmx = D.pred[xn], pmy = D.pred[yn] & ~(1u << xn), pms = D.pre_sinks;
    auto maxof = [&](uint32_t mask) {
        std::string m;
        for (int u = 0; u < NP; ++u)
            if (mask >> u & 1u) m = m.empty() ? "f" + std::to_string(u) : "fmaxf(" + m + ", f" + std::to_string(u) + ")";
        return m.empty() ? std::string("0.0f") : m;
    };
    o << "__device__ __constant__ const int dy_lvl_order[DY_K] = {";
    for (int k = 0; k < K; ++k) o << (k ? ", " : "") << D.lvl_order[k];
    o << "};\n";
    o << R"(
extern "C" __global__ void __launch_bounds__(256) dy_sweep_seed(
    unsigned long long nsamp, unsigned long long S, unsigned long long units, unsigned long long blk_first,
    unsigned long long begin, unsigned long long count, const float2* __restrict__ at,
    const float2* __restrict__ atx, const float2* __restrict__ aty, int rmax, const unsigned* __restrict__ jtab,
    unsigned* __restrict__ scert) {
  __shared__ float2 s_pat[)" << NP << R"( * 64];
  __shared__ int s_jt[64];
  __shared__ unsigned s_red[DY_K][4];
  const unsigned long long t0 = (unsigned long long)blockIdx.x * 256ull;
  if (t0 >= nsamp) return;
  for (int i = threadIdx.x; i < )" << NP << R"( * 64; i += 256) {
    const int n = i >> 6, e = i & 63;
    s_pat[i] = e < rmax ? at[n * rmax + e] : make_float2(1.0f, 0.0f);
  }
  if (threadIdx.x < 64) s_jt[threadIdx.x] = (int)jtab[threadIdx.x];
  __syncthreads();
  const unsigned long long t = t0 + threadIdx.x;
  const bool live = t < nsamp;
  const unsigned long long tj = live ? t : nsamp - 1;
  const unsigned long long st = tj * S;
  const unsigned wd = (unsigned)(S < units - st ? S : units - st);
  const unsigned hh = (unsigned)(tj * 0x9E3779B1ull) >> 16;
  const unsigned u = (unsigned)(st + (unsigned long long)(hh % wd));
  const unsigned qb = u / )" << D.rx << R"(u;
  const int ix = (int)(u - qb * )" << D.rx << R"(u);
  const unsigned long long b = blk_first + qb;
  unsigned x_ = (unsigned)b;
)";
    for (int n = NP - 1; n >= 0; --n) {
        o << "  const unsigned d" << n << " = x_ % " << D.radix[n] << "u;";
        if (n > 0) o << " x_ /= " << D.radix[n] << "u;";
        o << "\n";
    }
    o << "  float pc = 1.0f;\n";
    for (int n = 0; n < NP; ++n) {
        o << "  const float2 v" << n << " = s_pat[" << n * 64 << " + d" << n << "];\n";
        o << "  pc = pc * v" << n << ".x;\n";
        std::string m;
        for (int u = 0; u < n; ++u)
            if (D.pred[n] >> u & 1u) m = m.empty() ? "f" + std::to_string(u) : "fmaxf(" + m + ", f" + std::to_string(u) + ")";
        o << "  const float f" << n << " = v" << n << ".y + " << (m.empty() ? "0.0f" : m) << ";\n";
    }
    o << "  const float px = " << maxof(pmx) << ", py = " << maxof(pmy) << ", ps = " << maxof(pms) << ";\n";
    o << "  const float2 vx = atx[ix];\n  const float fx = vx.y + px;\n  const float cx = pc * vx.x;\n";
    o << "  const float M = " << (exy ? "fmaxf(py, fx)" : "py") << ";\n";
    if (s2) o << "  const float S2 = " << (exy ? "ps" : "fmaxf(ps, fx)") << ";\n";
    o << "  const unsigned long long base = (b * " << D.rx << "ull + (unsigned long long)ix) * " << D.ry << "ull;\n";
    for (int k = 0; k < K; ++k) o << "  float bst" << k << " = -1.0f;\n";
    o << "#pragma unroll\n  for (int j = 0; j < " << D.ry << "; ++j) {\n";
    o << "    const float2 vy = aty[j];\n    float cp = vy.y + M;\n";
    if (s2) o << "    cp = fmaxf(cp, S2);\n";
    o << "    const float cc = cx * vy.x;\n";
    o << "    const int nj = (live && base + (unsigned long long)j - begin < count) ? s_jt[(__float_as_uint(cp) >> "
      << D.bin_shift << "u) & 63u] : 0;\n";
    for (int k = 0; k < K; ++k) o << "    bst" << k << " = fmaxf(bst" << k << ", nj > " << k << " ? cc : -1.0f);\n";
    o << "  }\n";
    o << "  const int lane = threadIdx.x & 63;\n";
    for (int k = 0; k < K; ++k) {
        o << "  { const unsigned e = dy_wmax(bst" << k << " >= 0.0f ? __float_as_uint(bst" << k << ") + 1u : 0u);\n";
        o << "    if (lane == 0) s_red[" << k << "][threadIdx.x >> 6] = e; }\n";
    }
    o << R"(  __syncthreads();
  if (threadIdx.x < DY_K) {
    const unsigned* r = s_red[threadIdx.x];
    const unsigned e = max(max(r[0], r[1]), max(r[2], r[3]));
    if (e) atomicMax(scert + dy_lvl_order[threadIdx.x] * 64 + (blockIdx.x % 64), e);
  }
}
)";
}

std::string gen_source(const ProbDev& D) {
    const int N = D.n;
    const int Q = (N + 3) / 4;
    std::ostringstream o;
    o << kCommon;
    o << "#define DY_N " << N << "\n#define DY_K " << D.k << "\n";
    // node tables: 64 entries each, then 192 spare ones (read by byte ids past 63)
    o << "#define DY_TAB (DY_N * 64 + 192)\n";
    // per-word constants of the id range check (bytes past node N-1 are zero)
    for (int q = 0; q < Q; ++q) {
        unsigned kk = 0;
        for (int b = 0; b < 4 && 4 * q + b < N; ++b) kk |= (unsigned)(0x80 - D.radix[4 * q + b]) << (8 * b);
        o << "#define DY_K_" << q << " 0x" << std::hex << kk << std::dec << "u\n";
    }
    // node tables (and the prefilter bins) into LDS
    o << R"(
__device__ __forceinline__ void dy_stage(const float2* __restrict__ at, int rmax,
                                         const unsigned* __restrict__ table, float2* s_tab, float* s_bins) {
  for (int i = threadIdx.x; i < DY_TAB; i += blockDim.x) {
    const int n = i >> 6, e = i & 63;
    s_tab[i] = n < DY_N && e < rmax ? at[n * rmax + e] : make_float2(__builtin_nanf(""), __builtin_nanf(""));
  }
  if (table != nullptr && threadIdx.x < 64) s_bins[threadIdx.x] = __uint_as_float(table[threadIdx.x]);
  __syncthreads();
}
)";
    auto wl = [&](const char* p) {
        std::string r;
        for (int q = 0; q < Q; ++q) r += (q ? ", " : "") + std::string(p) + std::to_string(q);
        return r;
    };
    if (!D.obj && !D.uniform) {
        // per-backend pressure: level k's fp32 CP of the row in words w0..,
        // from that level's durations L (the generic kernel's order), inlined
        // at every use
        o << "__device__ __forceinline__ float dy_cpk(";
        for (int q = 0; q < Q; ++q) o << "unsigned w" << q << ", ";
        o << "const float* __restrict__ L, int rmax) {\n";
        for (int n = 0; n < N; ++n) {
            const int q = n / 4, b = n % 4;
            std::vector<int> preds;
            for (int u = 0; u < n; ++u)
                if (D.pred[n] >> u & 1u) preds.push_back(u);
            o << "  const float h" << n << " = L[" << n << " * rmax + (int)((w" << q;
            if (b) o << " >> " << 8 * b;
            o << ") & 255u)]";
            if (!preds.empty()) {
                std::string m = "h" + std::to_string(preds[0]);
                for (size_t k = 1; k < preds.size(); ++k) m = "fmaxf(" + m + ", h" + std::to_string(preds[k]) + ")";
                o << " + " << m;
            }
            o << ";\n";
        }
        std::string ck;
        for (int n = 0; n < N; ++n)
            if (D.sinks >> n & 1u) ck = ck.empty() ? "h" + std::to_string(n) : "fmaxf(" + ck + ", h" + std::to_string(n) + ")";
        o << "  return " << ck << ";\n}\n";
        o << "__device__ __constant__ const float dy_hi[DY_K] = {";
        for (int k = 0; k < D.k; ++k) o << (k ? ", " : "") << flit(D.hi[k]);
        o << "};\n";
        o << "__device__ __constant__ const float dy_lymin[DY_K] = {";
        for (int k = 0; k < D.k; ++k) o << (k ? ", " : "") << flit(D.lymin[k]);
        o << "};\n";
        if (D.ry >= 1 && D.ry <= 64) {
            o << "__device__ __constant__ const unsigned char dy_yord[" << D.ry << "] = {";
            for (int j = 0; j < D.ry; ++j) o << (j ? ", " : "") << (int)D.yord[j];
            o << "};\n";
        }
    }
    auto load_body = [&](const char* dst, const char* cond) {
        o << "  if (" << cond << ") { \\\n";
        for (int q = 0; q < Q; ++q)
            o << "    " << dst << q << " = ((const unsigned*)p_)[" << q << "]; \\\n";
        o << "  } else { \\\n";
        for (int q = 0; q < Q; ++q) {
            o << "    " << dst << q << " = 0u";
            for (int b = 0; b < 4 && 4 * q + b < N; ++b)
                o << " | ((unsigned)p_[" << 4 * q + b << "] << " << 8 * b << ")";
            o << "; \\\n";
        }
        o << "  }";
    };
    // row loads: whole dwords when aligned, else bytes
    o << "#define DY_LOAD(rr, " << wl("w") << ") { \\\n  const unsigned char* p_ = rows + (rr) * stride; \\\n";
    load_body("w", "aligned");
    o << " }\n";
    o << "#define DY_LOADP(pp, " << wl("x") << ") { const unsigned char* p_ = (pp); \\\n";
    load_body("x", "ALIGNED");
    o << " __builtin_amdgcn_sched_barrier(0); }\n";
    // objective mode: the level weights as literals
    if (D.obj) {
        o << "#define DY_LAM " << flit(D.lam_l) << "\n";
        o << "__device__ __constant__ const float dy_m32[DY_K] = {";
        for (int k = 0; k < D.k; ++k) o << (k ? ", " : "") << flit(D.m32[k]);
        o << "};\n__device__ __constant__ const double dy_m64[DY_K] = {";
        for (int k = 0; k < D.k; ++k) o << (k ? ", " : "") << dlit(D.m64[k]);
        o << "};\n";
        o << "__device__ __forceinline__ unsigned dy_fkey(float x) {\n"
             "  const unsigned b = __float_as_uint(x);\n"
             "  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);\n}\n";
    }
    // evaluation of one row held in words w0..
    o << "#define DY_EVAL(" << wl("w") << ", c, cp, bad) { \\\n  unsigned bk_ = 0u; \\\n";
    for (int q = 0; q < Q; ++q)
        o << "  bk_ |= (w" << q << " + DY_K_" << q << ") | w" << q << "; \\\n";
    o << "  bad = (bk_ & 0x80808080u) != 0u; \\\n";
    for (int n = 0; n < N; ++n) {
        const int q = n / 4, b = n % 4;
        o << "  const float2 e" << n << " = s_tab[" << n * 64 << " + ((w" << q;
        if (b) o << " >> " << 8 * b;
        o << ") & 255u)]; \\\n";
    }
    if (D.obj) {
        emit_obj_sums(o, D, 0, N);
    } else {
        o << "  c = e0.x; \\\n";
        for (int n = 1; n < N; ++n) o << "  c = c * e" << n << ".x; \\\n";
    }
    emit_recurrence(o, D, 0, N);
    emit_sinks(o, D, D.obj ? "t_" : "cp", D.obj != 0);
    if (D.obj) o << "  c = fmaf(-DY_LAM, t_, u_); \\\n  cp = d_; \\\n";
    o << "}\n";
    // one row of the scoring pass.  The nodes are evaluated in segments; at
    // the end of each but the last the wave abandons its rows when none can
    // still become a candidate: the corr so far times corr_tail (an upper
    // bound on the final fp32 corr) is below the prefilter threshold of a
    // lower bound on the final fp32 CP (the largest f_n + lat_tail[n] over the
    // evaluated nodes without an evaluated successor, less 2^-18 relative,
    // and never below the smallest CP).  Thresholds below 2^-60 never
    // abandon, so every product the bound reasons about is a normal number.
    // Rows that reach the end take the prefilter by the bin of their CP, the
    // exact per-level test, then the wave's LDS candidate queue.
    {
        const std::vector<int> cuts = D.obj ? std::vector<int>() : checkpoints(N);
        o << "#define DY_HANDLE(" << wl("y") << ", rr, LIVE) { \\\n  const bool live = (LIVE); \\\n"
          << "  unsigned bk_ = 0u; \\\n";
        for (int q = 0; q < Q; ++q)
            o << "  bk_ |= (y" << q << " + DY_K_" << q << ") | y" << q << "; \\\n";
        o << "  const bool bad = (bk_ & 0x80808080u) != 0u; \\\n  badmask |= __builtin_amdgcn_ballot_w64(live && bad); \\\n"
          << "  const bool ok = live && !bad; \\\n  do { \\\n  float c, cp; \\\n";
        int n0 = 0;
        std::vector<int> ends = cuts;
        ends.push_back(N);
        for (int m : ends) {
            for (int n = n0; n < m; ++n) {
                const int q = n / 4, bb = n % 4;
                o << "  const float2 e" << n << " = s_tab[" << n * 64 << " + ((y" << q;
                if (bb) o << " >> " << 8 * bb;
                o << ") & 255u)]; \\\n";
            }
            if (!D.obj)
                for (int n = n0; n < m; ++n)
                    o << (n == 0 ? "  c = e0.x; \\\n" : "  c = c * e") << (n == 0 ? "" : std::to_string(n) + ".x; \\\n");
            emit_recurrence(o, D, n0, m);
            if (m < N) {
                std::string lb;
                for (int n = 0; n < m; ++n) {
                    bool inner = false;
                    for (int v = n + 1; v < m; ++v)
                        if (D.pred[v] >> n & 1u) inner = true;
                    if (inner) continue;
                    std::string term = "f" + std::to_string(n);
                    if (D.lat_tail[n] > 0.0f) term = "(" + term + " + " + flit(D.lat_tail[n]) + ")";
                    lb = lb.empty() ? term : "fmaxf(" + lb + ", " + term + ")";
                }
                o << "  { const float lb_ = fmaxf(" << lb << " * " << flit(1.0f - 0x1p-18f) << ", "
                  << flit(u2f(D.cp_lo_bits)) << "); \\\n"
                  << "    const float th_ = s_bins[(__float_as_uint(lb_) >> bin_shift) & 63u]; \\\n"
                  << "    if (!__builtin_amdgcn_ballot_w64(ok && (c * " << flit(D.corr_tail[m]) << " >= th_ || th_ < 0x1p-60f))) break; } \\\n";
            }
            n0 = m;
        }
        if (D.obj) {
            emit_obj_sums(o, D, 0, N);
            emit_sinks(o, D, "t_", true);
            o << "  c = fmaf(-DY_LAM, t_, u_); \\\n  cp = d_; \\\n";
        } else {
            emit_sinks(o, D, "cp", false);
        }
    }
    // objective mode: c = G, cp = D, and a level's exact test is its one-rounding
    // estimate fma(-m_k, D, G) against its threshold
    o << R"(  const float th = s_bins[(__float_as_uint(cp) >> bin_shift) & 63u]; \
  bool want = ok && c >= th; \
  if (__builtin_amdgcn_ballot_w64(want)) { \
    if (want) { \
      bool w2 = false; \
)";
    if (D.obj)
        o << "      for (int k = 0; k < DY_K; ++k) if (fma(-dy_m64[k], (double)cp, (double)c) >= (double)thr[k]) w2 = true; \\\n";
    else
        o << "      for (int k = 0; k < DY_K; ++k) if (cp <= hi[k] && c >= thr[k]) w2 = true; \\\n";
    o << R"(      want = w2; \
    } \
)";
    if (!D.obj && !D.uniform) {
        // per-backend pressure: the bands above are those of the unpressured
        // CP; a row that passes them is parked in the wave's refine queue and
        // takes each level's exact fp32 CP_k (its durations from the level's
        // table) after the row loop, where that code adds no register
        // pressure to the loop; a full refine queue sends the rows straight
        // to the candidate list (certification decides them exactly)
        o << R"(    { const unsigned long long r_ = __builtin_amdgcn_ballot_w64(want); \
      if (r_) { \
        const unsigned rn_ = (unsigned)__builtin_popcountll(r_); \
        if (rqn + rn_ <= DY_RQCAP) { \
          if (want) { \
            const unsigned o_ = rqn + __builtin_amdgcn_mbcnt_hi((unsigned)(r_ >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)r_, 0u)); \
            rq[o_].index = (rr); rq[o_].corr = c; rq[o_].cp = cp; \
          } \
          rqn += rn_; \
          want = false; \
        } \
      } } \
)";
    }
    o << R"(    const unsigned long long m_ = __builtin_amdgcn_ballot_w64(want); \
    if (m_) { \
      const unsigned n_ = (unsigned)__builtin_popcountll(m_); \
      if (qn + n_ > DY_QCAP) { \
        ovf = true; /* queue full: the source is rescored after reseeding */ \
      } else { \
        if (want) { \
          const unsigned o_ = qn + __builtin_amdgcn_mbcnt_hi((unsigned)(m_ >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)m_, 0u)); \
          q[o_].index = index_base + (rr); q[o_].corr = c; q[o_].cp = cp; \
        } \
        qn += n_; \
      } \
    } \
  } \
  } while (0); }
)";
    // The load method is a template parameter and every load is issued
    // unconditionally (pointers clamped to the last row), so the compiler can
    // count the loads in flight and waits only for the row it scores.
    o << R"(
template <int ALIGNED>
__device__ __forceinline__ void dy_scan_body(
    const unsigned char* __restrict__ rows, unsigned long long stride, unsigned long long count,
    unsigned long long index_base, const float2* __restrict__ at, int rmax,
    const unsigned* __restrict__ table, int bin_shift, const float* __restrict__ hi,
    const float* __restrict__ thr, const float* __restrict__ lat, DyCand* __restrict__ cand, unsigned cap,
    unsigned* __restrict__ ncand, int* __restrict__ flags) {
  __shared__ float2 s_tab[DY_TAB];
  __shared__ float s_bins[64];
  __shared__ DyCand s_q[4][DY_QCAP];
)";
    if (!D.obj && !D.uniform)
        o << "  __shared__ DyCand s_rq[4][DY_RQCAP];\n  DyCand* rq = s_rq[threadIdx.x >> 6];\n  unsigned rqn = 0;\n";
    o << R"(  dy_stage(at, rmax, table, s_tab, s_bins);
  const int lane = threadIdx.x & 63;
  DyCand* q = s_q[threadIdx.x >> 6];
  unsigned qn = 0;
  bool ovf = false;
  unsigned long long badmask = 0;
  const unsigned long long G = (unsigned long long)gridDim.x * 256ull;
  const unsigned long long wbase = (unsigned long long)blockIdx.x * 256ull + (threadIdx.x & ~63u);
  if (wbase >= count) return;
  unsigned long long iters = (count - wbase + G - 1) / G;
  iters = ((unsigned long long)__builtin_amdgcn_readfirstlane((int)(iters >> 32)) << 32) |
          (unsigned)__builtin_amdgcn_readfirstlane((int)iters);
  unsigned long long r = wbase + lane;
  const unsigned long long step = G * stride;
  const unsigned char* p = rows + r * stride;
  unsigned )" << wl("u0") << ", " << wl("u1") << ", " << wl("u2") << ", " << wl("u3") << R"(;
  // Rows j < iters - 1 of the wave are whole (every lane in range, as G >= 256),
  // so the main loop, which touches rows up to it + 6 <= iters - 2, needs no
  // clamp and no range test; a ring of four row buffers keeps three rows in
  // flight while one is scored.  The last rows go one at a time.
  unsigned long long it = 0;
  if (iters >= 8) {
    DY_LOADP(p, )" << wl("u0") << R"()
    DY_LOADP(p + step, )" << wl("u1") << R"()
    DY_LOADP(p + 2 * step, )" << wl("u2") << R"()
    for (; it + 8 <= iters; it += 4) {
      DY_LOADP(p + 3 * step, )" << wl("u3") << R"()
      DY_HANDLE()" << wl("u0") << R"(, r, true)
      DY_LOADP(p + 4 * step, )" << wl("u0") << R"()
      DY_HANDLE()" << wl("u1") << R"(, r + G, true)
      DY_LOADP(p + 5 * step, )" << wl("u1") << R"()
      DY_HANDLE()" << wl("u2") << R"(, r + 2 * G, true)
      DY_LOADP(p + 6 * step, )" << wl("u2") << R"()
      DY_HANDLE()" << wl("u3") << R"(, r + 3 * G, true)
      p += 4 * step;
      r += 4 * G;
    }
  }
  const unsigned char* const plast = rows + (count - 1) * stride;
  for (; it < iters; ++it) {
    DY_LOADP((r < count ? p : plast), )" << wl("u0") << R"()
    DY_HANDLE()" << wl("u0") << R"(, r, r < count)
    p += step;
    r += G;
  }
)";
    if (!D.obj && !D.uniform) {
        // the parked rows: reload each, then its exact fp32 CP_k at every
        // level whose threshold and band it meets
        o << R"(  for (unsigned i0 = 0; i0 < rqn; i0 += 64) {
    const unsigned i = i0 + lane;
    bool keep = false;
    DyCand e = {0ull, 0.0f, 0.0f};
    if (i < rqn) {
      e = rq[i];
      unsigned )" << wl("v") << R"(;
      DY_LOADP(rows + e.index * stride, )" << wl("v") << R"()
      for (int k = 0; k < DY_K && !keep; ++k)
        if (e.corr >= thr[k] && e.cp <= dy_hi[k] &&
            dy_cpk()" << wl("v") << R"(, lat + (unsigned long long)k * DY_N * (unsigned long long)rmax, rmax) <= )"
          << flit(D.ghi) << R"()
          keep = true;
    }
    const unsigned long long m_ = __builtin_amdgcn_ballot_w64(keep);
    if (m_) {
      const unsigned n_ = (unsigned)__builtin_popcountll(m_);
      if (qn + n_ > DY_QCAP) {
        ovf = true;
      } else {
        if (keep) {
          const unsigned o_ = qn + __builtin_amdgcn_mbcnt_hi((unsigned)(m_ >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)m_, 0u));
          q[o_].index = index_base + e.index; q[o_].corr = e.corr; q[o_].cp = e.cp;
        }
        qn += n_;
      }
    }
  }
)";
    }
    o << R"(  dy_flush(q, qn, lane, cand, cap, ncand, &ovf);
  if (lane == 0 && (badmask || ovf)) atomicOr(flags, (badmask ? 2 : 0) | (ovf ? 1 : 0));
}

#define DY_SCAN_ARGS \
    const unsigned char* __restrict__ rows, unsigned long long stride, unsigned long long count, \
    unsigned long long index_base, const float2* __restrict__ at, int rmax, \
    const unsigned* __restrict__ table, int bin_shift, const float* __restrict__ hi, \
    const float* __restrict__ thr, const float* __restrict__ lat, DyCand* __restrict__ cand, unsigned cap, \
    unsigned* __restrict__ ncand, int* __restrict__ flags
#define DY_SCAN_PASS rows, stride, count, index_base, at, rmax, table, bin_shift, hi, thr, lat, cand, cap, ncand, flags
extern "C" __global__ void __launch_bounds__(256) dy_rows_scan_a(DY_SCAN_ARGS) { dy_scan_body<1>(DY_SCAN_PASS); }
extern "C" __global__ void __launch_bounds__(256) dy_rows_scan_u(DY_SCAN_ARGS) { dy_scan_body<0>(DY_SCAN_PASS); }

)";
    // seeding pass: hashed sample rows, grid-stride; per level the largest
    // certified corr (ordered bits + 1) of the thread, reduced per wave at the
    // end; objective mode: the largest estimate fma(-m_k, D, G) (ordered key)
    if (D.obj)
        o << "#define DY_SEED_UPDATE(k) best[k] = max(best[k], dy_fkey(fmaf(-dy_m32[k], cp, c)))\n";
    else if (!D.uniform)  // a CP inside the bands takes the level's exact fp32 CP_k against SLO (1 - (N+2)u),
                          // only for a sample that would raise the thread's value
        o << "#define DY_SEED_UPDATE(k) { const unsigned e_ = __float_as_uint(c) + 1u; if (e_ > best[k] && "
             "(cp <= lo[k] || (cp <= dy_hi[k] && dy_cpk(" << wl("w")
          << ", lat + (unsigned long long)(k) * DY_N * (unsigned long long)rmax, rmax) <= " << flit(D.glo)
          << "))) best[k] = e_; }\n";
    else
        o << "#define DY_SEED_UPDATE(k) if (cp <= lo[k]) best[k] = max(best[k], __float_as_uint(c) + 1u)\n";
    o << R"(extern "C" __global__ void __launch_bounds__(256) dy_rows_sample(
    const unsigned char* __restrict__ rows, unsigned long long stride, unsigned long long count,
    const float2* __restrict__ at, int rmax, const float* __restrict__ lo, const float* __restrict__ lat,
    unsigned* __restrict__ scert, unsigned long long S, int aligned) {
  __shared__ float2 s_tab[DY_TAB];
  dy_stage(at, rmax, nullptr, s_tab, nullptr);
  const int lane = threadIdx.x & 63;
  const unsigned long long nsamp = (count + S - 1) / S;
  const unsigned long long G = (unsigned long long)gridDim.x * 256ull;
  unsigned best[DY_K];
  for (int k = 0; k < DY_K; ++k) best[k] = 0u;
  for (unsigned long long t = (unsigned long long)blockIdx.x * 256ull + threadIdx.x; t < nsamp; t += G) {
    const unsigned long long rr = dy_sample_row(t, S, count);
    unsigned )" << wl("w") << R"(;
    DY_LOAD(rr, )" << wl("w") << R"()
    float c, cp; bool bad;
    DY_EVAL()" << wl("w") << R"(, c, cp, bad)
    if (!bad)
      for (int k = 0; k < DY_K; ++k)
        DY_SEED_UPDATE(k);
  }
  // wave maxima, then the workgroup's through LDS: one atomic per level and
  // workgroup (same-address atomics serialise across the device)
  __shared__ unsigned s_red[DY_K][4];
  for (int k = 0; k < DY_K; ++k) {
    const unsigned e = dy_wmax(best[k]);
    if (lane == 0) s_red[k][threadIdx.x >> 6] = e;
  }
  __syncthreads();
  if (threadIdx.x < DY_K) {
    const unsigned* r = s_red[threadIdx.x];
    const unsigned e = max(max(r[0], r[1]), max(r[2], r[3]));
    if (e) atomicMax(scert + threadIdx.x * 64 + (blockIdx.x % 64), e);
  }
}
)";
    if (D.uniform || D.obj) {
        gen_score(o, D);
    }
    if (D.npre >= 1 && D.xnode >= 0) gen_sweep(o, D);
    if (D.uniform && !D.obj && D.npre >= 1 && D.xnode >= 0) gen_sweep_seed(o, D);
    return o.str();
}

}  // namespace

// Compile (or fetch from the process cache) the rows kernels of problem D for
// `device`.  Returns false with a message when the problem does not qualify
// or runtime compilation is unavailable.
bool jit_rows_get(int device, const ProbDev& D, JitRows* out, std::string* err) {
    for (int n = 0; n < D.n; ++n)
        if (D.radix[n] > 64) {
            *err = "a node has more than 64 implementations";
            return false;
        }
    static_assert(NSLOT == 64, "generated sampler writes 64 slots per level");
    const std::string src = gen_source(D);
    const std::string key = std::to_string(device) + "\n" + src;
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_cache.find(key);
    if (it != g_cache.end()) {
        *out = it->second;
        return true;
    }
    hiprtcProgram prog;
    if (hiprtcCreateProgram(&prog, src.c_str(), "dyplan_rows.hip", 0, nullptr, nullptr) != HIPRTC_SUCCESS) {
        *err = "hiprtcCreateProgram failed";
        return false;
    }
    hipDeviceProp_t prop;
    std::string arch = "--offload-arch=gfx950";
    if (hipGetDeviceProperties(&prop, device) == hipSuccess) arch = std::string("--offload-arch=") + prop.gcnArchName;
    const char* opts[] = {arch.c_str(), "-O3", "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang",
                          "-packed-fp32-ops"};
    const hiprtcResult rc = hiprtcCompileProgram(prog, 7, opts);
    if (rc != HIPRTC_SUCCESS) {
        size_t n = 0;
        hiprtcGetProgramLogSize(prog, &n);
        std::string log(n, '\0');
        if (n) hiprtcGetProgramLog(prog, &log[0]);
        *err = std::string("hiprtc compile failed: ") + log.substr(0, 400);
        hiprtcDestroyProgram(&prog);
        return false;
    }
    size_t sz = 0;
    hiprtcGetCodeSize(prog, &sz);
    std::vector<char> code(sz);
    hiprtcGetCode(prog, code.data());
    hiprtcDestroyProgram(&prog);
    JitRows j;
    if (hipModuleLoadData(&j.mod, code.data()) != hipSuccess ||
        hipModuleGetFunction(&j.scan, j.mod, "dy_rows_scan_a") != hipSuccess ||
        hipModuleGetFunction(&j.scan_u, j.mod, "dy_rows_scan_u") != hipSuccess ||
        hipModuleGetFunction(&j.sample, j.mod, "dy_rows_sample") != hipSuccess ||
        ((D.uniform || D.obj) && hipModuleGetFunction(&j.score_rows, j.mod, "dy_score_rows") != hipSuccess) ||
        (D.npre >= 1 && D.xnode >= 0 && hipModuleGetFunction(&j.sweep, j.mod, "dy_sweep") != hipSuccess) ||
        (D.uniform && !D.obj && D.npre >= 1 && D.xnode >= 0 &&
         hipModuleGetFunction(&j.seed, j.mod, "dy_sweep_seed") != hipSuccess)) {
        *err = "loading the compiled rows kernels failed";
        return false;
    }
    g_cache[key] = j;  // modules stay loaded for the life of the process
    *out = j;
    return true;
}

// Source of the kernels for a problem (diagnostics and tests).
std::string jit_rows_source(const ProbDev& D) { return gen_source(D); }

}  // namespace dyp
