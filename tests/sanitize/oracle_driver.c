/* Runs every entry point of the fp64 oracle (oracle.c, objective.c) on small
 * seeded problems, for a build under AddressSanitizer and UBSan.  The two
 * sources are included whole so the driver sees their types.  Exit status 0
 * when every call returned success; the sanitizers report anything else. */
#include "../../oracle/oracle.c"
#include "../../oracle/objective.c"

#include <stdio.h>

static uint64_t st = 0x243F6A8885A308D3ull;
static double urand(void) {
    st += 0x9E3779B97F4A7C15ull;
    uint64_t z = st;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    return (double)(z >> 11) * 0x1p-53;
}

int main(void) {
    int bad = 0;
    for (int trial = 0; trial < 40; ++trial) {
        const int N = 1 + trial % 7, R = 1 + trial % 5, K = 1 + trial % 4, B = 1 + trial % 3;
        int32_t edges[64][2], radix[8], backend[8 * 8], is_tool[8];
        float p[64], tau[64], size[64], cost[64], w[8], rho[16 * 4], levels[4];
        int E = 0;
        for (int i = 0; i < N; ++i)
            for (int j = i + 1; j < N; ++j)
                if (urand() < 0.4) {
                    edges[E][0] = i;
                    edges[E][1] = j;
                    ++E;
                }
        for (int n = 0; n < N; ++n) {
            radix[n] = 1 + (int)(urand() * R);
            w[n] = (float)urand();
            is_tool[n] = urand() < 0.2;
            for (int i = 0; i < R; ++i) {
                p[n * R + i] = (float)(0.4 + 0.6 * urand());
                tau[n * R + i] = (float)(0.1 + 3.0 * urand());
                size[n * R + i] = (float)(1 + (int)(urand() * 6));
                cost[n * R + i] = tau[n * R + i] * size[n * R + i];
                backend[n * R + i] = (int)(urand() * B);
            }
        }
        for (int k = 0; k < K; ++k) {
            levels[k] = (float)(1.5 * k);
            for (int b = 0; b < B; ++b) rho[k * B + b] = (float)(0.9 * urand());
        }
        or_problem pb = {N, E, &edges[0][0], radix, R, p, tau, size, backend, w, K, B, rho, 4.0f};
        uint64_t total = 1;
        for (int n = 0; n < N; ++n) total *= (uint64_t)radix[n];
        or_choice ch[4];
        bad += or_select_range(&pb, 0, total, ch) != 0;
        uint8_t rows[512 * 10];
        uint64_t idx[512];
        const uint64_t nr = total < 512 ? total : 512;
        int32_t impl[64];
        for (uint64_t j = 0; j < nr; ++j) {
            or_decode(&pb, j, impl);
            for (int n = 0; n < N; ++n) rows[j * 10 + (uint64_t)n] = (uint8_t)impl[n];
            idx[j] = nr - 1 - j;
        }
        bad += or_select_rows(&pb, rows, nr, 10, 7, ch) != 0;
        double corr[512], cp[512 * 4], dem[512];
        uint32_t feas[512];
        bad += or_score_range(&pb, 0, nr, corr, cp, dem, feas) != 0;
        bad += or_score_rows(&pb, rows, nr, 10, corr, cp, dem, feas) != 0;
        bad += or_score_indices(&pb, idx, nr, corr, cp, dem, feas) != 0;
        uint64_t hist[1 << 8] = {0};
        bad += or_cp0_hist(&pb, 0, NULL, 0, 0, nr, 8, hist) != 0;
        bad += or_cp0_hist(&pb, 1, rows, 10, 0, nr, 8, hist) != 0;
        double vals[512];
        bad += or_cp0_collect(&pb, 1, rows, 10, 0, nr, 8, 0, vals, 512) < 0;
        bad += or_cp0_range(&pb, 0, NULL, 0, 0, nr, vals) != 0;
        (void)or_corr(&pb, impl);
        (void)or_cp(&pb, impl, -1);
        (void)or_demand(&pb, impl);
        op_problem ob = {N, E, &edges[0][0], radix, R, p, tau, cost, w, (trial & 1) ? is_tool : NULL,
                         1.0f, 0.01f, 0.05f, 0.05f, 1.0f, 0.5f, K, levels};
        op_choice oc[4];
        double reach[8], U, T, D, J[4];
        bad += op_reach(&ob, reach) != 0;
        bad += op_eval(&ob, impl, &U, &T, &D, J) != 0;
        bad += op_select_range(&ob, 0, total, oc) != 0;
        bad += op_select_rows(&ob, rows, nr, 10, 0, oc) != 0;
        double su[512], st_[512], sd[512], sj[512 * 4];
        bad += op_score(&ob, 0, NULL, 0, 0, nr, su, st_, sd, sj) != 0;
        bad += op_score(&ob, 1, rows, 10, 0, nr, su, st_, sd, sj) != 0;
    }
    printf("oracle driver: %d failed calls\n", bad);
    return bad != 0;
}
