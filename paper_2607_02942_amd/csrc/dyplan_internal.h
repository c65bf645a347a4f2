// Internal layout shared by the host side (host.cpp) and the kernels
// (kernels.hip) of the plan scorer.  Not part of the public ABI.
#pragma once

#include <stdint.h>

#include "dyplan.h"

namespace dyp {

constexpr int WG = 256;          // threads per workgroup of the scoring kernels
constexpr int NMAX = DY_MAX_NODES;
constexpr int KMAX = DY_MAX_LEVELS;
constexpr int NBINS = 64;        // lane-resident prefilter table: one bin per lane
constexpr int NBINS2 = 256;      // bins of the generated sweep's prefilter (one shift-and-mask operation)
constexpr int NSLOT = 64;        // per-level atomic slots of the seeding pass (spreads contention)
constexpr int CERT_WAVES = 8;    // waves per source in certification when sources are few
constexpr int CLIMB_ENTRIES = 512;  // local search: largest sum of a problem's radices (its tables in LDS), else none

// Unsigned 32-bit division by an invariant divisor (Granlund & Montgomery,
// PLDI 1994, Fig. 4.1): q = (t + ((x - t) >> sh1)) >> sh2, t = mulhi(m, x).
struct Magic {
    uint32_t m;
    uint32_t sh1;
    uint32_t sh2;
    uint32_t d;
};

// Static, per problem; built once by dy_plan_create.
struct ProbDev {
    int32_t n, k, b, rmax;
    int32_t npre;             // prefix nodes 0..npre-1 (the nodes before the inner pair)
    int32_t xnode, ynode;     // inner pair x = N-2, y = N-1 (x = -1 for a 1-node DAG)
    int32_t rx, ry;           // their radices (rx = 1 when x is virtual)
    int32_t uniform;          // every level presses all used backends equally
    int32_t edge_xy;          // edge x -> y exists
    int32_t x_sink;           // x has no successor
    uint32_t pre_sinks;       // sinks among prefix nodes (bit mask)
    uint32_t sinks;           // sinks among all nodes
    uint32_t pred[NMAX];      // predecessor bit mask of each node
    int32_t radix[NMAX];
    Magic rmag[NMAX];         // division by radix[n]
    Magic pvmag[NMAX];        // division by the place value of prefix node n within a block index
    uint32_t pv_big[NMAX];    // place value >= 2^32: the digit of this prefix node is 0 for 32-bit blocks
    uint64_t pv64[NMAX];      // place value of prefix node n within a block index (saturated)
    uint64_t n_plans;         // number of plans (saturated at 2^64-1)
    float lo[KMAX];           // certainly feasible at level k if the fp32 CP compared is <= lo[k]
    float hi[KMAX];           // possibly feasible at level k only if it is <= hi[k]
    float mk[KMAX];           // uniform mode: fp32 1/(1 - rho_k), for per-plan CP outputs
    double slo;
    uint32_t cp_lo_bits, cp_hi_bits;  // fp32 bounds of the unpressured CP over all plans
    int32_t bin_shift;        // prefilter bin = (bits(CP) >> bin_shift) mod 64
    int32_t jsh;              // generated sweep: prefilter bin = (bits(CP) >> jsh) mod 256 (jsh = 18), 0: unused
    // seeding pass (uniform mode): levels sorted by lo (descending); for a CP
    // in bin j, jtab[j] levels of that order are certainly feasible (a lower
    // bound: the bin's largest CP decides)
    uint32_t jtab[NBINS];
    int32_t lvl_order[KMAX];
    // bounds for abandoning a streamed row part-way (uniform mode):
    // corr_tail[m] >= the fp32 product of every node m..N-1's largest factor,
    // with slack for N roundings; lat_tail[n] <= the fp32 sum of the smallest
    // durations along the cheapest path from n's successors to a sink
    float corr_tail[NMAX + 1];
    float lat_tail[NMAX];
    // device tables
    const float2* at;         // [n][rmax] (factor a = 1 - w(1-p), duration tau), fp32
    const float2* atx;        // rows of x and y in `at` (x: a 1-entry (1, 0) row when virtual)
    const float2* aty;
    const float* dem;         // [n][rmax] demand term tau * size, fp32
    const float* lat;         // general mode: [k][n][rmax] fp32 tau / (1 - rho_{k,b})
    // fp64 terms of the definition, each rounded exactly as the definition
    // writes it (the re-evaluation only multiplies, adds and compares them)
    const double* a64;        // [n][rmax] 1 - w (1 - p)
    const double* lat64;      // [k][n][rmax] tau / (1 - rho_{k,b})
    const double* dem64;      // [n][rmax] tau * size
    // Objective mode (the paper's additive objective, Sec. 4.3-4.4): the same
    // tables hold at = (u, tau), dem = d (tau for LLM nodes, 0 for tool
    // nodes), a64 = u in fp64, dem64 = d in fp64, lat / lat64 = tau (one
    // level); cp_lo_bits / cp_hi_bits / bin_shift then describe the range of
    // the fp32 D, which indexes the prefilter bins.
    int32_t obj;
    uint32_t llm;             // LLM nodes (bit mask): only they add utility and demand
    float lam_l;              // lambda_l (the fp32 input)
    int32_t pad1;
    double lam_l64;
    float m32[KMAX];          // lambda_ld L_k rounded to fp32
    double m64[KMAX];         // lambda_ld L_k (exact in fp64)
    double err2[KMAX];        // twice a bound on |estimate - J_k| for every fp32 estimate of a plan's J_k
    const float* demx;        // rows of x and y in `dem` (x: a 1-entry 0 row when virtual)
    const float* demy;
    // Per-backend pressure (uniform == 0): lo / hi are bands on the fp32
    // unpressured CP implied by every level's largest / smallest multiplier
    // (a conservative prefilter, as in uniform mode); glo / ghi are the bands
    // of the exact per-level test on the fp32 CP_k itself.
    float glo, ghi;
    float ay_max;             // largest factor a of node y (fp32 table)
    float ty_min;             // smallest duration tau of node y
    uint8_t yord[64];         // ids of node y by decreasing fp32 factor a (ties by id), radix <= 64
    float lymin[KMAX];        // per-backend pressure: per level, node y's smallest fp32 duration
    // per implementation j of node y (j < 64): r_j <= 1 / (a_j (1 + 2^-22)),
    // rounded down to fp32; 0 when a_j < 2^-20.  A bin threshold T scaled by
    // r_j is a threshold on the rest of the product: fp32(c a_j) >= T implies
    // c >= fp32(T r_j) for T > 2^-60 (see ydiv_threshold).
    float yinv[64];
    // objective mode, per implementation j of y (j < 64): c_j >= u_j -
    // lambda_l tau_j + E (E bounds the roundings of a plan's G and of its
    // row's fma(-lambda_l, M, ux)), rounded up to fp32; see yshift_key
    float ysub[64];
};

struct Cand {
    uint64_t index;
    float corr;
    float cp;
};

enum JobFlags : int32_t { JF_OVERFLOW = 1, JF_BAD_ROW = 2 };

// Per source, per call.
struct JobDev {
    const ProbDev* prob;
    int32_t kind;             // DY_SOURCE_RANGE / DY_SOURCE_ROWS
    int32_t big;              // RANGE: some block (or plan) index needs 64 bits
    uint64_t begin, count;    // RANGE: plan indices [begin, begin + count); ROWS: count rows
    const uint8_t* rows;
    uint64_t stride;
    uint64_t index_base;
    uint64_t blk_first, nblk; // RANGE sweep: inner-pair blocks covering the range
    uint64_t units;           // work units of the main kernel (blocks for the sweep, plans otherwise)
    uint32_t sample_stride;
    uint32_t cap;             // candidate slots
    uint32_t* scert;          // [KMAX][NSLOT] best certainly-feasible fp32 corr found by the pre-pass, bits + 1 (0: none)
    float* thr;               // [KMAX] candidate thresholds
    uint32_t* table;          // [NBINS] prefilter thresholds (fp32 bits)
    uint32_t* table2;         // [NBINS2] the same on the generated sweep's finer bins (P->jsh)
    Cand* cand;               // [cap]
    uint32_t* ncand;
    int32_t* flags;
    dy_choice* out;           // [KMAX]
    uint64_t* fb_corr;        // [KMAX] exhaustive fp64 path: best corr bits
    uint64_t* fb_index;       // [KMAX] exhaustive fp64 path: lowest index at that corr
    uint32_t fb_levels;       // exhaustive path: bit mask of levels to decide
    int32_t cert_waves;       // waves of certification for this source
    double* cert_c;           // [KMAX][CERT_WAVES] per-wave best fp64 corr of certification
    uint64_t* cert_i;         // [KMAX][CERT_WAVES] its index
    double* cert_cp;          // [KMAX][CERT_WAVES] its fp64 CP at the level
    double* cert_d;           // [KMAX][CERT_WAVES] its fp64 demand
    uint32_t* sync;           // certification blocks finished (re-armed to 0 by the last)
    dy_choice* hout;          // [KMAX] host-mapped copy of the choices (null: copied back instead)
    uint32_t* hncand;         // host-mapped copies of ncand and flags (with hout)
    int32_t* hflags;
    uint32_t* hdone;          // host-mapped completion word of the call (with hout), set last
    int32_t climb;            // RANGE source over its problem's whole plan space: local-search seeds
    int32_t gblk;             // library sweep: consecutive blocks per thread (units = nblk / gblk)
};

}  // namespace dyp
