// The backward's grouping of a one-hot mini-batch (one lookup per bag, the
// layout of the DLRM-shaped workloads) table by table.
//
// The reduction needs the (key, bag) pairs of every distinct key contiguous,
// in ascending lookup order, hot keys first.  Hot slots are ranks of the
// ascending hot ids and a table's rows are one id range, so the hot slots of
// table t form one range [lo_t, hi_t); a staging row holds a row of one
// table.  Sorting each table's lookups by key, and placing the tables' hot
// pairs one after another at the front and their other pairs one before
// another at the back, gives such an order without a sort over the whole
// mini-batch.  Two launches:
//
//  gt_prep  -- the keys in table-major order (bag j = s T + t goes to
//              position t E + s, E = bags per table; the bag is implied by
//              the position): a block takes GT_S consecutive bag rows s,
//              reads their offsets and codes (coalesced), forms the keys (the
//              fused plan's cold-code rewrite included), and writes each
//              table's GT_S keys through LDS; it also stores, for its rows,
//              the number of hot keys of the tables before each table.
//  gt_sort  -- one block per table:
//              the table's E keys, compressed to [0, R_t) for hot slots
//              (R_t = hi_t - lo_t) and above for staging rows, sorted with
//              their positions in LDS by an LSD radix of as many 9-bit digits
//              as the largest key needs; then the table's hot pairs go to the
//              front of the output after those of the earlier tables, its
//              others to the back before those of the earlier tables (both
//              offsets from the prep blocks' counts).
//
// Ranks inside a wave: the lanes that hold the wave's first lane's digit
// advance its counter once, together (stable by construction); every other
// lane adds 1 to its digit's counter and takes the old value, an order among
// same-digit lanes of one instruction that nothing specifies.  So the sorted
// table is checked (keys ascending, positions ascending among equal keys:
// the stable order, and the only one that passes) and, if the check fails,
// sorted again with every rank formed from ballot peer masks.
#include "hl_group_sort.h"

// ----------------------------------------------------------------------------- prep
__global__ void __launch_bounds__(256)
gt_prep(int32_t* codes, const int32_t* __restrict__ bag_ptr, int64_t n_bags, int32_t T, uint32_t E, uint32_t n_hot,
        uint32_t k_cap, int32_t stg_rows, const uint32_t* __restrict__ tb, uint32_t* __restrict__ keys_tm,
        uint32_t* __restrict__ cum, int64_t n_lookups, uint32_t* sflag, uint32_t sv, uint32_t* err,
        hl_cg_fused cf) {
  __shared__ uint32_t lk[GT_TMAX][GT_S];
  __shared__ uint32_t hcnt[GT_TMAX];
  __shared__ uint32_t stb[GT_TMAX + 1];
  __shared__ uint32_t s_bad;
  bw_start_signal(sflag, sv);
  const int tid = threadIdx.x;
  if (tid == 0) s_bad = 0;
  if (tid <= T) stb[tid] = tb[tid];
  if (tid < T) hcnt[tid] = 0;
  const bool fits = cf.table && *cf.ncold <= (uint32_t)cf.cap;
  if (blockIdx.x == 0 && tid == 0) {
    if (bag_ptr[n_bags] != n_lookups) hl_flag(err, HL_DEVERR_SHAPE);
    if (cf.table && !fits) hl_flag(err, HL_DEVERR_CAPACITY);
  }
  __syncthreads();
  const uint32_t s0 = blockIdx.x * GT_S;
  const uint32_t ns = min((uint32_t)GT_S, E - s0);
  const int64_t j0 = (int64_t)s0 * T;
  const uint32_t nb = ns * (uint32_t)T;
  bool bad = false, badc = false;
  // every load of the thread's bags in flight before any is used
  int32_t lo[GT_PI], hi[GT_PI], cc[GT_PI];
#pragma unroll
  for (int i = 0; i < GT_PI; ++i) {
    const uint32_t q = tid + i * 256;
    const int64_t j = j0 + min(q, nb - 1);
    lo[i] = bag_ptr[j];
    hi[i] = bag_ptr[j + 1];
    cc[i] = codes[j];
  }
#pragma unroll
  for (int i = 0; i < GT_PI; ++i) {
    const uint32_t q = tid + i * 256;
    if (q >= nb) continue;
    const int64_t j = j0 + q;
    uint32_t key = EB_SENT;
    // one lookup per bag: bag j holds lookup j
    if (lo[i] != j || hi[i] != j + 1) {
      bad = true;
    } else {
      int32_t c = cc[i];
      if (cf.table && c == -1) {
        const uint32_t sl = cf.slotof[j];
        c = bw_fused_code(c, (uint32_t)j, cf, k_cap, fits);
        if (c != -1) codes[j] = c;
        if (sl < cf.S) cf.table[sl] = 0;
      }
      key = bw_key((uint32_t)c, n_hot, k_cap, stg_rows);
      badc = badc || key == EB_SENT;
    }
    const uint32_t t = q % (uint32_t)T;
    lk[t][q / (uint32_t)T] = key;
    // hot keys per table: those gt_sort places at the front (a hot slot of
    // the table's own range)
    if (key < n_hot && key - stb[t] < stb[t + 1] - stb[t]) atomicAdd(&hcnt[t], 1u);
  }
  if (bad) s_bad = 1;  // (every writer stores 1)
  if (badc) hl_flag(err, HL_DEVERR_BAD_CODE);
  __syncthreads();
  if (tid == 0 && s_bad) hl_flag(err, HL_DEVERR_SHAPE);
  for (uint32_t q = tid; q < nb; q += blockDim.x) {
    const uint32_t t = q / ns, s = q - t * ns;
    const uint64_t p = (uint64_t)t * E + s0 + s;
    keys_tm[p] = lk[t][s];  // (a row of GT_S keys of one table)
  }
  // for each table the hot keys of the tables before it (T <= 64: one wave's
  // scan; the last entry, T, is the total)
  if (tid < 64) {
    const uint32_t v = tid < T ? hcnt[tid] : 0u;
    uint32_t x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = __shfl_up(x, o);
      if (tid >= o) x += y;
    }
    uint32_t* c = cum + (uint64_t)blockIdx.x * (T + 1);
    if (tid <= T) c[tid] = x - v;
    if (T == 64 && tid == 63) c[64] = x;
  }
}

// ----------------------------------------------------------------------------- sort
template <int ITEMS>
__global__ void __launch_bounds__(GT_THREADS)
gt_sort(const uint32_t* __restrict__ keys_tm, const uint32_t* __restrict__ cum, uint32_t nblk, uint32_t E,
        int32_t T, uint32_t n, const uint32_t* __restrict__ tb, uint32_t n_hot, uint32_t* __restrict__ kout,
        uint32_t* __restrict__ vout, uint32_t* err, int ballot_only, hl_hook hk) {
  hl_hook_head(hk);  // a handover signal: the codes are complete (gt_prep has ended)
  gt_sort_body<ITEMS>(blockIdx.x, keys_tm, cum, nblk, E, T, n, tb, n_hot, kout, vout, err, ballot_only);
}

// ----------------------------------------------------------------------------- host
bool hl_group_by_table_ok(const hl_handle* h, int64_t n_lookups, int64_t n_bags) {
  const int32_t T = h->n_tables;
  if (n_lookups != n_bags || n_bags == 0 || T > GT_TMAX || n_bags % T != 0) return false;
  const int64_t E = n_bags / T;
  // the prep blocks' counts go where the table-major bags would
  return E <= (int64_t)GT_IMAX * GT_THREADS && hl_div_up(E, GT_S) * (T + 1) <= n_lookups;
}

uint32_t hl_group_prep(hl_handle* h, int32_t* codes, const int32_t* bag_ptr, int64_t n_bags, int32_t stg_rows,
                       uint32_t* k_tm, uint32_t* cum, uint32_t* sflag, uint32_t sv, const hl_cg_fused* cf,
                       hipStream_t s) {
  const int32_t T = h->n_tables;
  const uint32_t E = (uint32_t)(n_bags / T);
  const uint32_t nblk = hl_div_up(E, GT_S);
  HL_KERNEL(h, s, "gt_prep", gt_prep, dim3(nblk), dim3(256), 0, s, codes, bag_ptr, n_bags, T, E, h->n_hot, h->k_cap,
            stg_rows, h->d_tb, k_tm, cum, n_bags, sflag, sv, h->d_err, cf ? *cf : hl_cg_fused{});
  return nblk;
}

hl_status hl_group_by_table(hl_handle* h, int32_t* codes, const int32_t* bag_ptr, int64_t n_bags, int32_t stg_rows,
                            uint32_t* k_tm, uint32_t* cum, uint32_t* kout, uint32_t* vout, uint32_t* sflag,
                            uint32_t sv, const hl_cg_fused* cf, hipStream_t s) {
  const int32_t T = h->n_tables;
  const uint32_t E = (uint32_t)(n_bags / T);
  const hl_hook hk = hl_hook_take(h);  // carried by gt_sort (the first sort pass takes it on the other path)
  const uint32_t nblk = hl_group_prep(h, codes, bag_ptr, n_bags, stg_rows, k_tm, cum, sflag, sv, cf, s);
#define GTS(I)                                                                                                    \
  HL_KERNEL(h, s, "gt_sort", gt_sort<I>, dim3(T), dim3(GT_THREADS), 0, s, k_tm, cum, nblk, E, T, (uint32_t)n_bags, \
            h->d_tb, h->n_hot, kout, vout, h->d_err, h->ballot_ranks, hk)
  if (E <= 4 * GT_THREADS) GTS(4);
  else GTS(8);
#undef GTS
  HL_LAUNCHED();
  return HL_OK;
}
