/*
 * Hotline hot-path ORACLE -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, single-threaded, obviously-correct CPU statement of what the hot
 * path of "Heterogeneous Acceleration Pipeline for Recommendation System
 * Training" (Hotline, arXiv 2204.05436) computes for one mini-batch.  It is
 * used by the test-suite, by the smoke check and by the benchmark's CPU
 * baseline leg only; the product path (the HIP library) never links, loads or
 * calls it, and the two share no code, header, table or constant.
 *
 * Floating point: sums in fp64, one rounding to the storage type at the end.
 * Build: gcc -O2 -ffp-contract=off -shared -fPIC (no FMA contraction, so every
 * expression rounds exactly as written).
 *
 * Readings of points the paper leaves open (ties, empty samples, slot order,
 * partition order, update timing) are stated at the function that takes them.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define HO_DT_F32 0
#define HO_DT_BF16 1

/* ------------------------------------------------------------------ helpers */
static int cmp_u32(const void* a, const void* b) {
    uint32_t x = *(const uint32_t*)a, y = *(const uint32_t*)b;
    return (x > y) - (x < y);
}

/* index of key in ascending array v[0..n) or -1 */
static int64_t find_u32(const uint32_t* v, int64_t n, uint32_t key) {
    const uint32_t* p = (const uint32_t*)bsearch(&key, v, (size_t)n, sizeof(uint32_t), cmp_u32);
    return p ? (int64_t)(p - v) : -1;
}

static double widen(const void* base, int dtype, int64_t elem) {
    if (dtype == HO_DT_F32) return (double)((const float*)base)[elem];
    uint32_t bits = (uint32_t)((const uint16_t*)base)[elem] << 16;
    float f;
    memcpy(&f, &bits, 4);
    return (double)f;
}

/* Round a double to bfloat16 (8 significant bits) to nearest, ties to even,
 * directly from the double (no intermediate fp32 rounding). */
static uint16_t round_bf16(double x) {
    uint16_t sign = signbit(x) ? 0x8000 : 0;
    double a = fabs(x);
    if (a == 0.0) return sign;
    int e;
    frexp(a, &e);                 /* a = m * 2^e, 0.5 <= m < 1 */
    int q = e - 8;                /* quantum of 8 significant bits */
    if (q < -133) q = -133;       /* bf16 subnormal quantum */
    double r = nearbyint(ldexp(a, -q));   /* default rounding mode: nearest-even */
    float f = (float)ldexp(r, q); /* exact (<= 8 significant bits), or inf on overflow */
    uint32_t bits;
    memcpy(&bits, &f, 4);
    return (uint16_t)((bits >> 16) | sign);
}

static void store(void* base, int dtype, int64_t elem, double v) {
    if (dtype == HO_DT_F32) ((float*)base)[elem] = (float)v;   /* nearest-even */
    else ((uint16_t*)base)[elem] = round_bf16(v);
}

/* Row pointer selection for a slot code: [0, k_cap) names a hot-cache slot,
 * [k_cap, ...) a row of the staging buffer that holds gathered cold rows. */
static int row_of(int32_t code, uint32_t k_cap, int64_t n_hot_rows, int64_t n_stg_rows,
                  int* in_staging, int64_t* row) {
    if (code < 0) return 0;
    if ((uint32_t)code < k_cap) {
        if (code >= n_hot_rows) return 0;
        *in_staging = 0;
        *row = code;
        return 1;
    }
    int64_t s = (int64_t)code - (int64_t)k_cap;
    if (s >= n_stg_rows) return 0;
    *in_staging = 1;
    *row = s;
    return 1;
}

/* ------------------------------------------------------------------ 1. ids */
/* Global row id of every lookup: the table's base (the exclusive prefix sum of
 * the row counts, the "Address Registers" holding each table's base, Sec. V-A
 * Data Dispatcher) plus the table-local row.  The table of bag j is j mod T
 * (bag index = (b*steps + s)*T + t).  A row outside its table is an error: the
 * id is set to 0xFFFFFFFF and 2 is returned. */
int ho_gids(int32_t n_tables, const uint32_t* rows_per_table, const uint32_t* rows,
            const int32_t* bag_ptr, int64_t n_bags, uint32_t* gids) {
    uint64_t* base = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)(n_tables > 0 ? n_tables : 1));
    uint64_t acc = 0;
    int rc = 0;
    for (int32_t t = 0; t < n_tables; ++t) {
        base[t] = acc;
        acc += rows_per_table[t];
    }
    for (int64_t j = 0; j < n_bags; ++j) {
        int32_t t = (int32_t)(j % n_tables);
        for (int32_t i = bag_ptr[j]; i < bag_ptr[j + 1]; ++i) {
            if (rows[i] >= rows_per_table[t]) {
                gids[i] = 0xFFFFFFFFu;
                rc = 2;
            } else {
                gids[i] = (uint32_t)(base[t] + rows[i]);
            }
        }
    }
    free(base);
    return rc;
}

/* ------------------------------------------------------------------ 2. count */
/* Access counting over profiling batches: one increment per lookup (the EAL's
 * per-entry frequency counter, Sec. V-B, in its exact "Oracle LFU" form).
 * Repeated ids inside a bag count with multiplicity.  Ids >= n_rows are
 * skipped and reported by a nonzero return. */
int ho_count(uint64_t n_rows, const uint32_t* gids, int64_t n, uint32_t* counts) {
    int rc = 0;
    for (int64_t i = 0; i < n; ++i) {
        if (gids[i] >= n_rows) { rc = 2; continue; }
        counts[gids[i]] += 1;
    }
    return rc;
}

/* ------------------------------------------------------------------ 3. select */
typedef struct { uint32_t cnt, gid; } cand_t;

static int cmp_cand(const void* a, const void* b) {
    const cand_t* x = (const cand_t*)a;
    const cand_t* y = (const cand_t*)b;
    if (x->cnt != y->cnt) return x->cnt > y->cnt ? -1 : 1;   /* count descending */
    return (x->gid > y->gid) - (x->gid < y->gid);            /* then id ascending */
}

/* Hot set: the k most frequently accessed rows (Sec. V-B; Oracle LFU of Fig.
 * "SRRIP-based tracker as compared to the Oracle LFU scheme").  Readings: only
 * rows accessed at least once are candidates; ties broken by ascending id; the
 * hot-cache slot of a hot row is its rank in ascending id order, so the output
 * list is ascending.  Returns n_hot = min(k, #candidates). */
int64_t ho_topk(uint64_t n_rows, const uint32_t* counts, uint64_t k, uint32_t* hot_ids) {
    int64_t nc = 0;
    for (uint64_t g = 0; g < n_rows; ++g) nc += counts[g] >= 1;
    cand_t* c = (cand_t*)malloc(sizeof(cand_t) * (size_t)(nc > 0 ? nc : 1));
    int64_t j = 0;
    for (uint64_t g = 0; g < n_rows; ++g)
        if (counts[g] >= 1) { c[j].cnt = counts[g]; c[j].gid = (uint32_t)g; ++j; }
    qsort(c, (size_t)nc, sizeof(cand_t), cmp_cand);
    int64_t nh = (int64_t)k < nc ? (int64_t)k : nc;
    for (int64_t i = 0; i < nh; ++i) hot_ids[i] = c[i].gid;
    qsort(hot_ids, (size_t)nh, sizeof(uint32_t), cmp_u32);
    free(c);
    return nh;
}

/* ------------------------------------------------------------------ 4. classify */
/* A sample is popular iff every one of its lookups names a hot row; a single
 * non-hot lookup makes it non-popular (Sec. I, insight 2; Sec. V-C Lookup
 * Engine).  A sample with no lookups is popular (the "every" is vacuous). */
void ho_classify(const uint32_t* hot_ids, int64_t n_hot, const uint32_t* gids,
                 const int32_t* bag_ptr, int32_t n_samples, int32_t bps, uint8_t* flags) {
    for (int32_t b = 0; b < n_samples; ++b) {
        uint8_t pop = 1;
        int64_t lo = bag_ptr[(int64_t)b * bps], hi = bag_ptr[(int64_t)(b + 1) * bps];
        for (int64_t i = lo; i < hi; ++i)
            if (find_u32(hot_ids, n_hot, gids[i]) < 0) pop = 0;
        flags[b] = pop;
    }
}

/* ------------------------------------------------------------------ 5. partition */
/* Split the mini-batch M into the popular mu-batch O and the non-popular X with
 * O u X = M and O n X = {} (Eq. 3).  Reading: both lists keep ascending sample
 * order.  Returns |O|. */
int32_t ho_partition(const uint8_t* flags, int32_t n, int32_t* pop, int32_t* nonpop) {
    int32_t a = 0, b = 0;
    for (int32_t i = 0; i < n; ++i) {
        if (flags[i]) pop[a++] = i;
        else nonpop[b++] = i;
    }
    return a;
}

/* ------------------------------------------------------------------ 6. remap */
/* Hot-cache address of every lookup: its slot (rank among the ascending hot
 * ids) when hot, else -1 (a row to be fetched from host memory). */
void ho_remap(const uint32_t* hot_ids, int64_t n_hot, const uint32_t* gids, int64_t n,
              int32_t* codes) {
    for (int64_t i = 0; i < n; ++i) codes[i] = (int32_t)find_u32(hot_ids, n_hot, gids[i]);
}

/* ------------------------------------------------------------------ 7. cold plan */
typedef struct { uint32_t gid; int64_t pos; } cpos_t;

static int cmp_cpos_gid(const void* a, const void* b) {
    const cpos_t* x = (const cpos_t*)a;
    const cpos_t* y = (const cpos_t*)b;
    if (x->gid != y->gid) return (x->gid > y->gid) - (x->gid < y->gid);
    return (x->pos > y->pos) - (x->pos < y->pos);
}

static int cmp_cpos_pos(const void* a, const void* b) {
    const cpos_t* x = (const cpos_t*)a;
    const cpos_t* y = (const cpos_t*)b;
    return (x->pos > y->pos) - (x->pos < y->pos);
}

/* Working parameters of a mu-batch (Sec. V-A: DMA reads for non-hot rows, in
 * the order the dispatcher streams the mu-batch).  The cold rows are the
 * distinct ids of the selected samples' lookups whose slot is -1, listed in
 * order of first occurrence in the mini-batch's CSR lookup order (for a
 * selection in ascending sample order, as the partition produces, that is the
 * order a stream over the mu-batch meets them); each such lookup's code
 * becomes k_cap + (position of its id in that list).  sel == NULL selects
 * samples 0..n_sel-1.  Returns the number of cold rows. */
int64_t ho_cold_plan(const uint32_t* gids, int32_t* codes, const int32_t* bag_ptr,
                     const int32_t* sel, int32_t n_sel, int32_t bps, uint32_t k_cap,
                     uint32_t* cold_ids) {
    int64_t m = 0;
    for (int32_t q = 0; q < n_sel; ++q) {
        int64_t b = sel ? sel[q] : q;
        m += bag_ptr[(b + 1) * bps] - bag_ptr[b * bps];
    }
    cpos_t* c = (cpos_t*)malloc(sizeof(cpos_t) * (size_t)(m > 0 ? m : 1));
    int64_t n = 0;
    for (int32_t q = 0; q < n_sel; ++q) {
        int64_t b = sel ? sel[q] : q;
        for (int64_t i = bag_ptr[b * bps]; i < bag_ptr[(b + 1) * bps]; ++i)
            if (codes[i] == -1) { c[n].gid = gids[i]; c[n].pos = i; ++n; }
    }
    /* first occurrence of each id: sort by (id, position), keep the first of each run */
    qsort(c, (size_t)n, sizeof(cpos_t), cmp_cpos_gid);
    int64_t u = 0;
    for (int64_t i = 0; i < n; ++i)
        if (i == 0 || c[i].gid != c[i - 1].gid) c[u++] = c[i];
    /* list the distinct ids by first position */
    qsort(c, (size_t)u, sizeof(cpos_t), cmp_cpos_pos);
    for (int64_t i = 0; i < u; ++i) cold_ids[i] = c[i].gid;
    /* id -> list position, through an id-sorted copy */
    cpos_t* byid = (cpos_t*)malloc(sizeof(cpos_t) * (size_t)(u > 0 ? u : 1));
    for (int64_t i = 0; i < u; ++i) { byid[i].gid = cold_ids[i]; byid[i].pos = i; }
    qsort(byid, (size_t)u, sizeof(cpos_t), cmp_cpos_gid);
    for (int32_t q = 0; q < n_sel; ++q) {
        int64_t b = sel ? sel[q] : q;
        for (int64_t i = bag_ptr[b * bps]; i < bag_ptr[(b + 1) * bps]; ++i) {
            if (codes[i] != -1) continue;
            int64_t lo = 0, hi = u;   /* binary search for the id */
            while (lo < hi) {
                int64_t mid = (lo + hi) / 2;
                if (byid[mid].gid < gids[i]) lo = mid + 1; else hi = mid;
            }
            codes[i] = (int32_t)((int64_t)k_cap + byid[lo].pos);
        }
    }
    free(byid);
    free(c);
    return u;
}

/* ------------------------------------------------------------------ 8. gather */
/* Row copy from the host table (dma_rd of the ISA table): out[u] = table[ids[u]]
 * bit for bit. */
void ho_gather(const void* table, uint64_t row_bytes, const uint32_t* ids, int64_t n, void* out) {
    for (int64_t u = 0; u < n; ++u)
        memcpy((char*)out + (size_t)u * row_bytes, (const char*)table + (size_t)ids[u] * row_bytes,
               (size_t)row_bytes);
}

/* Write-back of updated working parameters (non-hot rows are updated in CPU
 * main memory, Sec. IV; dma_wr of the ISA table): table[ids[u]] = rows[u] bit
 * for bit.  The ids are distinct. */
void ho_scatter(void* table, uint64_t row_bytes, const uint32_t* ids, int64_t n, const void* rows) {
    for (int64_t u = 0; u < n; ++u)
        memcpy((char*)table + (size_t)ids[u] * row_bytes, (const char*)rows + (size_t)u * row_bytes,
               (size_t)row_bytes);
}

/* ------------------------------------------------------------------ 9. forward */
/* Sum pooling (the Reducer's sparse-length element-wise sum, Sec. V-D, v_add of
 * the ISA): out[bag] = sum of the bag's rows, in fp64 in CSR order, rounded once
 * to fp32.  Rows come from the hot cache or the staging buffer by code.  An
 * empty bag pools to zero.  sel == NULL selects samples 0..n_sel-1.  If scale is
 * non-NULL it receives sum |term| per element (the summation error scale).
 * Returns 0, or 3 if a code names no row. */
int ho_embbag_fwd(int32_t dim, int32_t dtype, const void* w_hot, uint32_t k_cap, int64_t n_hot_rows,
                  const void* staging, int64_t n_stg_rows, const int32_t* codes,
                  const int32_t* bag_ptr, const int32_t* sel, int32_t n_sel, int32_t bps,
                  float* out, double* scale) {
    double* acc = (double*)malloc(sizeof(double) * (size_t)dim);
    double* aab = (double*)malloc(sizeof(double) * (size_t)dim);
    int rc = 0;
    for (int32_t q = 0; q < n_sel; ++q) {
        int64_t b = sel ? sel[q] : q;
        for (int32_t j = 0; j < bps; ++j) {
            int64_t bag = b * bps + j;
            for (int32_t d = 0; d < dim; ++d) acc[d] = aab[d] = 0.0;
            for (int64_t i = bag_ptr[bag]; i < bag_ptr[bag + 1]; ++i) {
                int st;
                int64_t r;
                if (!row_of(codes[i], k_cap, n_hot_rows, n_stg_rows, &st, &r)) { rc = 3; continue; }
                const void* src = st ? staging : w_hot;
                for (int32_t d = 0; d < dim; ++d) {
                    double v = widen(src, dtype, r * dim + d);
                    acc[d] += v;
                    aab[d] += fabs(v);
                }
            }
            for (int32_t d = 0; d < dim; ++d) {
                out[bag * dim + d] = (float)acc[d];
                if (scale) scale[bag * dim + d] = aab[d];
            }
        }
    }
    free(acc);
    free(aab);
    return rc;
}

/* Unsplit reference: the same pooling with every row read from one flat table by
 * global id (no hot/cold distinction).  Eq. 5 says the mu-batch split must give
 * the same result. */
void ho_embbag_fwd_flat(int32_t dim, int32_t dtype, const void* table, const uint32_t* gids,
                        const int32_t* bag_ptr, int64_t n_bags, float* out) {
    double* acc = (double*)malloc(sizeof(double) * (size_t)dim);
    for (int64_t bag = 0; bag < n_bags; ++bag) {
        for (int32_t d = 0; d < dim; ++d) acc[d] = 0.0;
        for (int64_t i = bag_ptr[bag]; i < bag_ptr[bag + 1]; ++i)
            for (int32_t d = 0; d < dim; ++d) acc[d] += widen(table, dtype, (int64_t)gids[i] * dim + d);
        for (int32_t d = 0; d < dim; ++d) out[bag * dim + d] = (float)acc[d];
    }
    free(acc);
}

/* ------------------------------------------------------------------ 10. backward */
typedef struct { int32_t code; int64_t lookup; int64_t bag; } occ_t;

static int cmp_occ(const void* a, const void* b) {
    const occ_t* x = (const occ_t*)a;
    const occ_t* y = (const occ_t*)b;
    if (x->code != y->code) return (x->code > y->code) - (x->code < y->code);
    return (x->lookup > y->lookup) - (x->lookup < y->lookup);
}

/* Gradient of sum pooling and one plain SGD step, with duplicate rows
 * coalesced: for every distinct code c among the selected bags' lookups,
 * G_c = sum of dY[bag(i)] over lookups i with code c (fp64, ascending lookup
 * order), then row_c <- round_storage(row_c - lr * G_c).  Rows no lookup names
 * are untouched.  Hot rows are updated in the hot cache and cold rows in the
 * staging buffer (Sec. IV: hot embeddings are updated on the GPU, the rest
 * where they live).  Reading of the update timing: one step per mini-batch over
 * both mu-batches, after both forwards, which is what gives gradients identical
 * to the unsplit mini-batch (Eq. 5).
 * Optional outputs: the distinct codes (ascending) and, per code and element,
 * |row| + lr * sum |dY| (the error scale of the update).  Returns the number of
 * distinct codes, or -3 if a code names no row. */
int64_t ho_embbag_bwd_sgd(int32_t dim, int32_t dtype, void* w_hot, uint32_t k_cap,
                          int64_t n_hot_rows, void* staging, int64_t n_stg_rows,
                          const int32_t* codes, const int32_t* bag_ptr, const int32_t* sel,
                          int32_t n_sel, int32_t bps, const float* dY, float lr,
                          int32_t* uniq_out, double* scale_out) {
    int64_t m = 0;
    for (int32_t q = 0; q < n_sel; ++q) {
        int64_t b = sel ? sel[q] : q;
        m += bag_ptr[(b + 1) * bps] - bag_ptr[b * bps];
    }
    occ_t* o = (occ_t*)malloc(sizeof(occ_t) * (size_t)(m > 0 ? m : 1));
    int64_t k = 0;
    for (int32_t q = 0; q < n_sel; ++q) {
        int64_t b = sel ? sel[q] : q;
        for (int64_t bag = b * bps; bag < (b + 1) * bps; ++bag)
            for (int64_t i = bag_ptr[bag]; i < bag_ptr[bag + 1]; ++i) {
                o[k].code = codes[i];
                o[k].lookup = i;
                o[k].bag = bag;
                ++k;
            }
    }
    qsort(o, (size_t)m, sizeof(occ_t), cmp_occ);
    double* g = (double*)malloc(sizeof(double) * (size_t)dim);
    double* ga = (double*)malloc(sizeof(double) * (size_t)dim);
    int64_t nu = 0, rc = 0;
    for (int64_t s = 0; s < m;) {
        int64_t e = s;
        while (e < m && o[e].code == o[s].code) ++e;
        int st;
        int64_t r;
        if (!row_of(o[s].code, k_cap, n_hot_rows, n_stg_rows, &st, &r)) {
            rc = -3;
            s = e;
            continue;
        }
        for (int32_t d = 0; d < dim; ++d) g[d] = ga[d] = 0.0;
        for (int64_t t = s; t < e; ++t)
            for (int32_t d = 0; d < dim; ++d) {
                double v = (double)dY[o[t].bag * dim + d];
                g[d] += v;
                ga[d] += fabs(v);
            }
        void* dst = st ? staging : w_hot;
        for (int32_t d = 0; d < dim; ++d) {
            double w0 = widen(dst, dtype, r * dim + d);
            if (scale_out) scale_out[nu * dim + d] = fabs(w0) + (double)lr * ga[d];
            store(dst, dtype, r * dim + d, w0 - (double)lr * g[d]);
        }
        if (uniq_out) uniq_out[nu] = o[s].code;
        ++nu;
        s = e;
    }
    free(g);
    free(ga);
    free(o);
    return rc ? rc : nu;
}

/* Unsplit reference of the update: every row addressed by global id in one flat
 * table. */
void ho_embbag_bwd_sgd_flat(int32_t dim, int32_t dtype, void* table, const uint32_t* gids,
                            const int32_t* bag_ptr, int64_t n_bags, const float* dY, float lr) {
    int64_t m = bag_ptr[n_bags];
    occ_t* o = (occ_t*)malloc(sizeof(occ_t) * (size_t)(m > 0 ? m : 1));
    for (int64_t bag = 0; bag < n_bags; ++bag)
        for (int64_t i = bag_ptr[bag]; i < bag_ptr[bag + 1]; ++i) {
            o[i].code = (int32_t)gids[i];   /* ids < 2^31 in every use of this function */
            o[i].lookup = i;
            o[i].bag = bag;
        }
    qsort(o, (size_t)m, sizeof(occ_t), cmp_occ);
    double* g = (double*)malloc(sizeof(double) * (size_t)dim);
    for (int64_t s = 0; s < m;) {
        int64_t e = s;
        while (e < m && o[e].code == o[s].code) ++e;
        for (int32_t d = 0; d < dim; ++d) g[d] = 0.0;
        for (int64_t t = s; t < e; ++t)
            for (int32_t d = 0; d < dim; ++d) g[d] += (double)dY[o[t].bag * dim + d];
        int64_t r = o[s].code;
        for (int32_t d = 0; d < dim; ++d)
            store(table, dtype, r * dim + d, widen(table, dtype, r * dim + d) - (double)lr * g[d]);
        s = e;
    }
    free(g);
    free(o);
}

/* ------------------------------------------------------------------ 11. re-learning */
/* The learning phase recurs during training (Sec. V-B: the EAL periodically
 * switches back to learning; Sec. VI: twice per epoch; Sec. IV: hot rows are
 * updated on the GPU, the others in CPU memory).  When a new hot set
 * new_ids replaces old_ids (both ascending, distinct; slot = position):
 *   - a row that leaves the cache (in old_ids, not in new_ids) goes back to the
 *     host table with its trained value: host[id] = w_hot_old[old slot];
 *   - a row that stays moves to its new slot with its trained value;
 *   - a row that enters is read from the host table.
 * Reading: nothing else changes, so the table as the path sees it (a hot row
 * from the cache, any other from the host table) is the same before and after,
 * bit for bit.  w_hot_new receives n_new rows; host is updated in place.
 * Returns the number of rows written back. */
int64_t ho_migrate(uint64_t row_bytes, const uint32_t* old_ids, int64_t n_old, const void* w_hot_old,
                   const uint32_t* new_ids, int64_t n_new, void* w_hot_new, void* host) {
    int64_t wb = 0;
    for (int64_t s = 0; s < n_old; ++s)
        if (find_u32(new_ids, n_new, old_ids[s]) < 0) {
            memcpy((char*)host + (size_t)old_ids[s] * row_bytes, (const char*)w_hot_old + (size_t)s * row_bytes,
                   (size_t)row_bytes);
            ++wb;
        }
    for (int64_t s = 0; s < n_new; ++s) {
        const int64_t o = find_u32(old_ids, n_old, new_ids[s]);
        const char* src = o >= 0 ? (const char*)w_hot_old + (size_t)o * row_bytes
                                 : (const char*)host + (size_t)new_ids[s] * row_bytes;
        memcpy((char*)w_hot_new + (size_t)s * row_bytes, src, (size_t)row_bytes);
    }
    return wb;
}

/* ------------------------------------------------------------------ 12. SRRIP tracker */
/* The Embedding Access Logger of Sec. V-B: a cache of embedding indices with
 * SRRIP replacement and a 2-bit re-reference prediction value (RRPV) instead
 * of per-row counters.  Readings (the paper gives no geometry that fits its own
 * numbers): n_sets sets of `ways` ways; id g lives in set mix(g) % n_sets,
 * where mix is the 32-bit finalizer of MurmurHash3 (Appleby, public domain);
 * accesses are taken in stream order (batch by batch, lookup order); a hit
 * sets the way's RRPV to 0; a miss takes the first way whose RRPV is 3, ageing
 * every way of the set by one until one is, and inserts the id with RRPV 2
 * (SRRIP's long re-reference insertion, one below the maximum).  An empty way
 * holds the id 0xFFFFFFFF and RRPV 3, and an access with that id (the id of a
 * row out of range) is not logged.  The hot set the tracker yields is every id
 * held at the end, ascending. */
uint32_t ho_mix32(uint32_t x) {
    x ^= x >> 16;
    x *= 0x85EBCA6Bu;
    x ^= x >> 13;
    x *= 0xC2B2AE35u;
    x ^= x >> 16;
    return x;
}

void ho_eal_init(int64_t n_sets, int32_t ways, uint32_t* tag, uint8_t* rrpv) {
    for (int64_t i = 0; i < n_sets * ways; ++i) {
        tag[i] = 0xFFFFFFFFu;
        rrpv[i] = 3;
    }
}

void ho_eal_access(int64_t n_sets, int32_t ways, uint32_t* tag, uint8_t* rrpv, const uint32_t* gids, int64_t n) {
    for (int64_t i = 0; i < n; ++i) {
        const uint32_t g = gids[i];
        if (g == 0xFFFFFFFFu) continue;
        const int64_t set = (int64_t)(ho_mix32(g) % (uint32_t)n_sets);
        uint32_t* t = tag + set * ways;
        uint8_t* r = rrpv + set * ways;
        int32_t hit = -1;
        for (int32_t w = 0; w < ways; ++w)
            if (t[w] == g) hit = w;
        if (hit >= 0) {
            r[hit] = 0;
            continue;
        }
        for (;;) {
            int32_t v = -1;
            for (int32_t w = 0; w < ways && v < 0; ++w)
                if (r[w] == 3) v = w;
            if (v >= 0) {
                t[v] = g;
                r[v] = 2;
                break;
            }
            for (int32_t w = 0; w < ways; ++w) ++r[w];
        }
    }
}

int64_t ho_eal_hot(int64_t n_sets, int32_t ways, const uint32_t* tag, uint32_t* out) {
    int64_t n = 0;
    for (int64_t i = 0; i < n_sets * ways; ++i)
        if (tag[i] != 0xFFFFFFFFu) out[n++] = tag[i];
    qsort(out, (size_t)n, sizeof(uint32_t), cmp_u32);
    return n;
}

/* bf16 rounding exposed for its own pin (ties-to-even cases). */
uint16_t ho_round_bf16(double x) { return round_bf16(x); }
