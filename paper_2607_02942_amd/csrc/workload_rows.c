/*
 * Candidate-row generator for the streamed workload: uniform implementation
 * ids drawn with a counter-based SplitMix64 (Steele, Lea & Flood, OOPSLA 2014).
 * Input generation only; no scoring arithmetic lives here.
 *
 *   draw(key, c) = mix(key + (c + 1) * 0x9E3779B97F4A7C15)
 *   id(row, n)   = ((draw(key, row * n_nodes + n) >> 32) * radix) >> 32
 */
#include <stdint.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static inline uint64_t dw_mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

uint64_t dw_draw(uint64_t key, uint64_t ctr) {
    return dw_mix(key + (ctr + 1) * 0x9E3779B97F4A7C15ULL);
}

/* Fill out[r * stride + n] for rows [row_begin, row_begin + n_rows); bytes
 * n_nodes..stride-1 of each row are zeroed.  threads <= 0: OpenMP default. */
int32_t dw_rows(uint64_t key, uint64_t row_begin, uint64_t n_rows, int32_t n_nodes,
                int32_t radix, uint64_t stride, uint8_t* out, int32_t threads) {
    if (!out || n_nodes <= 0 || radix <= 0 || radix > 256 || stride < (uint64_t)n_nodes) return -1;
#ifdef _OPENMP
    if (threads > 0) omp_set_num_threads(threads);
#else
    (void)threads;
#endif
    int64_t nr = (int64_t)n_rows;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < nr; ++r) {
        uint8_t* row = out + (uint64_t)r * stride;
        uint64_t base = (row_begin + (uint64_t)r) * (uint64_t)n_nodes;
        for (int32_t n = 0; n < n_nodes; ++n) {
            uint64_t hi = dw_draw(key, base + (uint64_t)n) >> 32;
            row[n] = (uint8_t)((hi * (uint64_t)radix) >> 32);
        }
        if (stride > (uint64_t)n_nodes) memset(row + n_nodes, 0, stride - (uint64_t)n_nodes);
    }
    return 0;
}
