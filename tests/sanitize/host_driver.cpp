// Runs the library's host-only code (validation, the dry staging behind
// dy_kernel_source and the kernel-source generator, suffix recompilation,
// bundle annotations, the switching simulator, the self checks) for a build
// under AddressSanitizer and UBSan.  The device-side launchers are stubs that
// fail: no path exercised here reaches them.  Exit status 0 when every call
// behaved as documented.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <string>
#include <vector>

#include "dyplan.h"
#include "dyplan_internal.h"

namespace dyp {
struct JitRows;
#define STUB return hipErrorNotSupported;
hipError_t launch_init(JobDev*, int, hipStream_t) { STUB }
hipError_t launch_table(JobDev*, int, hipStream_t) { STUB }
hipError_t launch_sample_sweep(const JobDev*, int, bool, bool, uint64_t, int, int, int, hipStream_t) { STUB }
hipError_t launch_sweep(const JobDev*, int, bool, bool, uint64_t, int, int, int, bool, bool, int, hipStream_t) { STUB }
hipError_t launch_sample_generic(const JobDev*, int, uint64_t, int, hipStream_t) { STUB }
hipError_t launch_scan(const JobDev*, int, uint64_t, int, hipStream_t) { STUB }
hipError_t launch_certify(const JobDev*, int, int, int, int, int, hipStream_t) { STUB }
hipError_t launch_exhaust(const JobDev*, int, uint64_t, hipStream_t) { STUB }
hipError_t launch_reseed(const JobDev*, int, hipStream_t) { STUB }
hipError_t launch_seed_cands(const JobDev*, int, int, int, hipStream_t) { STUB }
hipError_t launch_climb(const JobDev*, int, int, int, int, int, hipStream_t) { STUB }
hipError_t static_scratch(int, char**, size_t*) { STUB }
hipError_t launch_score(const JobDev&, uint64_t, float*, float*, float*, uint32_t*, int, int, int, bool, bool, hipStream_t) {
    STUB
}
}  // namespace dyp

static uint64_t st = 0x243F6A8885A308D3ull;
static double urand() {
    st += 0x9E3779B97F4A7C15ull;
    uint64_t z = st;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    return (double)(z >> 11) * 0x1p-53;
}

struct Prob {
    int N, R, K, B;
    std::vector<int32_t> edges, radix, backend, is_tool, model;
    std::vector<float> p, tau, size, w, rho, cost, levels;
    dy_objective obj{};
    dy_problem pb{};
};

static void make(Prob& P, int N, int R, int K, int B, bool objective, double edge_p) {
    P.N = N, P.R = R, P.K = K, P.B = B;
    for (int i = 0; i < N; ++i)
        for (int j = i + 1; j < N; ++j)
            if (urand() < edge_p) {
                P.edges.push_back(i);
                P.edges.push_back(j);
            }
    P.radix.resize(N);
    P.w.resize(N);
    P.is_tool.resize(N);
    for (int n = 0; n < N; ++n) {
        P.radix[n] = 1 + (int)(urand() * R);
        P.w[n] = (float)urand();
        P.is_tool[n] = urand() < 0.2;
    }
    for (int e = 0; e < N * R; ++e) {
        P.p.push_back((float)(0.4 + 0.6 * urand()));
        P.tau.push_back((float)(0.1 + 3.0 * urand()));
        P.size.push_back((float)(1 + (int)(urand() * 6)));
        P.cost.push_back(P.tau.back() * P.size.back());
        P.backend.push_back((int)(urand() * B));
        P.model.push_back((int)(urand() * 3));
    }
    for (int k = 0; k < K; ++k) {
        P.levels.push_back((float)(1.5 * k));
        for (int b = 0; b < B; ++b) P.rho.push_back((float)(0.9 * urand()));
    }
    P.obj = dy_objective{P.cost.data(), P.is_tool.data(), 1.0f, 0.01f, 0.05f, 0.05f, 1.0f, 0.5f, K, P.levels.data()};
    P.pb = dy_problem{N, (int32_t)(P.edges.size() / 2), P.edges.data(), P.radix.data(), R, P.p.data(), P.tau.data(),
                      P.size.data(), P.backend.data(), P.w.data(), K, B, P.rho.data(), 4.0f,
                      objective ? &P.obj : nullptr};
}

int main() {
    int bad = 0;
    bad += dy_selftest() != 0;
    for (int s = 1; s >= -6; --s) bad += dy_status_str(s) == nullptr;
    for (int trial = 0; trial < 40; ++trial) {
        Prob P;
        const int N = 1 + trial % 24;
        make(P, N, 1 + trial % 40, 1 + trial % 8, 1 + trial % 3, trial % 3 == 2, trial % 2 ? 0.15 : 0.5);
        // generated kernel source, host-only
        uint64_t len = 0;
        bad += dy_kernel_source(&P.pb, nullptr, 0, &len) != DY_OK;
        std::string buf(len + 1, '\0');
        uint64_t len2 = 0;
        bad += dy_kernel_source(&P.pb, &buf[0], len + 1, &len2) != DY_OK || len2 != len;
        char small[16];
        bad += dy_kernel_source(&P.pb, small, sizeof small, &len2) != DY_OK || small[15] != '\0';
        // suffix recompilation on a random committed set
        std::vector<uint8_t> committed(N);
        std::vector<int32_t> cimpl(N), full(N);
        int ncom = 0;
        for (int n = 0; n < N; ++n) {
            committed[n] = n < N / 2;
            ncom += committed[n];
            cimpl[n] = committed[n] ? (int)(urand() * P.radix[n]) : 0;
        }
        dy_suffix* sx = nullptr;
        const int rc = dy_suffix_create(&P.pb, committed.data(), &sx);
        if (ncom == N) {
            bad += rc != DY_EINVAL;
        } else {
            bad += rc != DY_OK;
            std::vector<int32_t> map(N);
            const int nr = dy_suffix_nodes(sx, map.data());
            bad += nr != N - ncom;
            bad += dy_suffix_problem(sx) == nullptr;
            int64_t fi = 0;
            bad += dy_suffix_merge(sx, cimpl.data(), 0, full.data(), &fi) != DY_OK;
            bad += dy_suffix_merge(sx, cimpl.data(), -1, full.data(), &fi) != DY_EINVAL;
            const dy_problem* rp = dy_suffix_problem(sx);
            bad += dy_kernel_source(rp, nullptr, 0, &len) != DY_OK;
        }
        dy_suffix_destroy(sx);
        // bundle annotation and switching
        std::vector<int32_t> impl(N);
        for (int n = 0; n < N; ++n) impl[n] = (int)(urand() * P.radix[n]);
        double dem[3], q = 0.0;
        int32_t dom = 0;
        bad += dy_bundle_annotate(&P.pb, P.model.data(), 3, impl.data(), dem, &dom, &q) != DY_OK;
        dy_variant vars[3] = {{0, 0.9}, {1, 0.85}, {2, 0.8}};
        std::vector<double> times(50), loads(150);
        for (int t = 0; t < 50; ++t) {
            times[t] = t;
            for (int m = 0; m < 3; ++m) loads[t * 3 + m] = urand();
        }
        dy_switch_rules rules{0.7, 0.3, 0.2, 0.1, 2.0};
        std::vector<int32_t> active(50);
        int32_t nsw = 0;
        bad += dy_switch_simulate(vars, 3, 3, times.data(), loads.data(), 50, &rules, active.data(), &nsw) != DY_OK;
        // validation errors, reported before any device call
        Prob Q;
        make(Q, N, 3, 2, 2, false, 0.3);
        Q.radix[0] = 0;
        dy_plan* h = nullptr;
        bad += dy_plan_create(&Q.pb, 1, 0, &h) != DY_EINVAL || h != nullptr;
        bad += dy_kernel_source(&Q.pb, nullptr, 0, &len) != DY_EINVAL;
        Q.radix[0] = 1;
        Q.tau[0] = NAN;
        bad += dy_plan_create(&Q.pb, 1, 0, &h) != DY_EINVAL;
        bad += std::string(dy_plan_last_error(nullptr)).empty();
    }
    dy_plan_destroy(nullptr);
    std::printf("host driver: %d failed checks\n", bad);
    return bad != 0;
}
