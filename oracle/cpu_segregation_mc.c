/* Multi-core CPU segregation: classify + partition of a mini-batch on the
 * host's cores, the CPU-side alternative whose cost and core scaling Sec. III
 * measures before moving segregation into the accelerator -- TEST
 * INFRASTRUCTURE.
 *
 * This is not the oracle.  The benchmark times it, labelled as a multi-core CPU
 * baseline, beside the single-threaded oracle; the tests check its results bit
 * for bit against the oracle's ho_gids, ho_classify and ho_partition.  It
 * shares no code with the HIP library.
 *
 * Per mini-batch:
 * - each lookup's global id: table base + row (Sec. V-A, Address Registers);
 * - hot-set membership of each id: one bit of a bitmap over all rows, built
 *   once per hot set, as a learning phase would;
 * - a sample is popular iff every one of its lookups is hot (Eq. 2); the scan
 *   of a sample stops at its first cold lookup;
 * - the popular and non-popular lists, in ascending sample order (Eq. 3).
 * Each thread takes one contiguous slice of the samples and counts its popular
 * ones.  A prefix over the threads' counts places every slice in the two
 * lists, and each thread then writes its own slice.
 */
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define MC_MAX_THREADS 256

/* Bits of the hot ids in bm (n_rows bits, (n_rows+63)/64 words, cleared
 * here).  Returns 0, or 2 when a hot id is >= n_rows (that id is skipped). */
int mc_hot_bitmap(const uint32_t* hot_ids, int64_t n_hot, uint64_t n_rows, uint64_t* bm) {
    int rc = 0;
    memset(bm, 0, (size_t)((n_rows + 63) / 64) * sizeof(uint64_t));
    for (int64_t i = 0; i < n_hot; ++i) {
        uint64_t g = hot_ids[i];
        if (g >= n_rows) {
            rc = 2;
            continue;
        }
        bm[g >> 6] |= 1ull << (g & 63);
    }
    return rc;
}

/* flags[b] (n_samples bytes), pop and nonpop (n_samples entries each); returns
 * the number of popular samples, or -1 on a bad argument.  Bag j belongs to
 * table j mod n_tables and sample b owns bags b*bps .. b*bps+bps-1; a row
 * outside its table makes its sample non-popular (its id names no hot row). */
int32_t mc_segregate(int32_t n_tables, const uint32_t* rows_per_table, const uint32_t* rows,
                     const int32_t* bag_ptr, int32_t n_samples, int32_t bps, const uint64_t* bm,
                     int32_t n_threads, uint8_t* flags, int32_t* pop, int32_t* nonpop) {
    if (n_tables < 1 || n_samples < 0 || bps < 1 || n_threads < 1) return -1;
    if (n_threads > MC_MAX_THREADS) n_threads = MC_MAX_THREADS;
    uint64_t* base = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)n_tables);
    if (!base) return -1;
    uint64_t acc = 0;
    for (int32_t t = 0; t < n_tables; ++t) {
        base[t] = acc;
        acc += rows_per_table[t];
    }
    int32_t cnt[MC_MAX_THREADS];
    int32_t total = 0;
#pragma omp parallel num_threads(n_threads)
    {
        const int th = omp_get_thread_num(), T = omp_get_num_threads();
        const int32_t lo = (int32_t)((int64_t)n_samples * th / T);
        const int32_t hi = (int32_t)((int64_t)n_samples * (th + 1) / T);
        int32_t c = 0;
        for (int32_t b = lo; b < hi; ++b) {
            uint8_t p = 1;
            for (int64_t j = (int64_t)b * bps; p && j < (int64_t)(b + 1) * bps; ++j) {
                const int32_t t = (int32_t)(j % n_tables);
                for (int32_t i = bag_ptr[j]; i < bag_ptr[j + 1]; ++i) {
                    const uint32_t r = rows[i];
                    const uint64_t g = base[t] + r;
                    if (r >= rows_per_table[t] || !((bm[g >> 6] >> (g & 63)) & 1u)) {
                        p = 0;
                        break;
                    }
                }
            }
            flags[b] = p;
            c += p;
        }
        cnt[th] = c;
#pragma omp barrier
        int32_t before = 0;
        for (int u = 0; u < th; ++u) before += cnt[u];
        int32_t a = before, q = lo - before;
        for (int32_t b = lo; b < hi; ++b) {
            if (flags[b])
                pop[a++] = b;
            else
                nonpop[q++] = b;
        }
#pragma omp barrier
#pragma omp single
        for (int u = 0; u < T; ++u) total += cnt[u];
    }
    free(base);
    return total;
}
