// The backward's grouping of a one-hot mini-batch (one lookup per bag, the
// layout of the DLRM- and TBSM-shaped workloads) table by table.
//
// The reduction needs the (key, bag) pairs of every distinct key contiguous,
// in ascending lookup order, hot keys first.  Hot slots are ranks of the
// ascending hot ids and a table's rows are one id range, so the hot slots of
// table t form one range [lo_t, hi_t); a staging row holds a row of one
// table.  Sorting each table's lookups by key, and placing the tables' hot
// pairs one after another at the front and their other pairs one before
// another at the back, gives such an order without a sort over the whole
// mini-batch.  A table's E = n_bags / T lookups (bag j = s T + t is its s-th)
// are cut into chunks of GC; two launches, every block independent:
//
//  gt_chunk -- a block per (table, chunk): reads its lookups' codes (strided
//              by T), forms the keys (the fused plan's cold-code rewrite
//              included), compresses them to [0, R_t) for hot slots (R_t =
//              hi_t - lo_t) and above for staging rows, sorts the chunk by
//              key in LDS (LSD radix of as many 9-bit digits as its largest
//              key needs; each pass checked for stability and redone with
//              ballot ranks if it broke an order), and writes the sorted
//              chunk and its count of hot keys.
//  gt_merge -- a block per (table, chunk): the table's sorted chunks into
//              LDS; each pair's rank in its table is its rank in its chunk
//              plus, in every other chunk, the keys below it (and the equal
//              ones of earlier chunks: lookup order) by binary search; the
//              tables' offsets from the chunks' hot counts.
#include "hl_internal.h"

#define GC 1024           // lookups per chunk (gt_merge's searches take 11 halving steps)
#define GC_THREADS 256
#define GC_ITEMS (GC / GC_THREADS)
#define GC_WAVES (GC_THREADS / 64)
#define GT_TMAX 64        // tables the path takes
#define GT_CMAX 32        // chunks per table
#define GT_DBITS 9        // largest digit of the chunk sort
#define GT_NB (1 << GT_DBITS)

// Exclusive scan of one value per thread over the block; *total receives the sum.
__device__ __forceinline__ uint32_t gt_scan(uint32_t v, uint32_t* ws, uint32_t* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) ws[w] = x;
  __syncthreads();
  uint32_t off = 0, tot = 0;
  for (int q = 0; q < (int)(blockDim.x >> 6); ++q) {
    const uint32_t c = ws[q];
    off += q < w ? c : 0u;
    tot += c;
  }
  *total = tot;
  __syncthreads();  // ws may be reused
  return x - v + off;
}

// ----------------------------------------------------------------------------- chunk sort
__global__ void __launch_bounds__(GC_THREADS)
gt_chunk(int32_t* codes, const int32_t* __restrict__ bag_ptr, int64_t n_bags, int32_t T, uint32_t E, uint32_t C,
         uint32_t n_hot, uint32_t k_cap, int32_t stg_rows, const uint32_t* __restrict__ tb, uint32_t* __restrict__ ck,
         uint32_t* __restrict__ cv, uint32_t* __restrict__ hcnt, uint32_t* __restrict__ lor, int64_t n_lookups,
         uint32_t* sflag, uint32_t sv, uint32_t* err, hl_cg_fused cf, int ballot_only) {
  __shared__ uint32_t sk[GC], sval[GC], spos[GC];
  __shared__ uint32_t wcnt[GC_WAVES][GT_NB];
  __shared__ uint32_t dofs[GT_NB];
  __shared__ uint32_t scan_ws[GC_WAVES];
  __shared__ uint32_t s_lo, s_hi, s_max, s_bad;
  bw_start_signal(sflag, sv);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const uint32_t t = blockIdx.x / C, c = blockIdx.x - t * C;
  const uint32_t s0 = c * GC;
  const uint32_t ns = min((uint32_t)GC, E - s0);
  const bool fits = cf.table && *cf.ncold <= (uint32_t)cf.cap;
  if (tid == 0) {
    s_lo = tb[t];  // the table's hot slots
    s_hi = tb[t + 1];
    s_max = 0;
    s_bad = 0;
    if (blockIdx.x == 0 && bag_ptr[n_bags] != n_lookups) hl_flag(err, HL_DEVERR_SHAPE);
    if (blockIdx.x == 0 && cf.table && !fits) hl_flag(err, HL_DEVERR_CAPACITY);
  }
  for (int j = tid; j < GC_WAVES * GT_NB; j += GC_THREADS) (&wcnt[0][0])[j] = 0;
  // the chunk's lookups: item k of thread (w, lane) is the chunk's lookup
  // r = w * 64 ITEMS + 64 k + lane (lookup order)
  uint32_t key[GC_ITEMS], val[GC_ITEMS];
  bool bad = false, badc = false;
#pragma unroll
  for (int k = 0; k < GC_ITEMS; ++k) {
    const uint32_t r = (uint32_t)w * (GC_ITEMS * 64) + k * 64 + lane;
    key[k] = EB_SENT;
    val[k] = 0;
    if (r >= ns) continue;
    const int64_t j = (int64_t)(s0 + r) * T + t;
    val[k] = (uint32_t)j;
    if (bag_ptr[j] != j || bag_ptr[j + 1] != j + 1) {  // one lookup per bag: bag j holds lookup j
      bad = true;
      continue;
    }
    int32_t cc = codes[j];
    if (cf.table && cc == -1) {
      const uint32_t sl = cf.slotof[j];
      cc = bw_fused_code(cc, (uint32_t)j, cf, k_cap, fits);
      if (cc != -1) codes[j] = cc;
      if (sl < cf.S) cf.table[sl] = 0;
    }
    key[k] = bw_key((uint32_t)cc, n_hot, k_cap, stg_rows);
    badc = badc || key[k] == EB_SENT;
  }
  if (bad) s_bad = 1;  // (every writer stores 1)
  __syncthreads();
  if (tid == 0 && s_bad) hl_flag(err, HL_DEVERR_SHAPE);
  const uint32_t lo = s_lo, R = s_hi - s_lo;
  // compressed keys: hot slot - lo, R + staging row; skipped lookups (an
  // invalid code, or a hot slot of another table's row) R + stg_rows, after
  // every other
  const uint32_t sent = R + (uint32_t)stg_rows;
  uint32_t kmax = 0;
  bool foreign = false;
#pragma unroll
  for (int k = 0; k < GC_ITEMS; ++k) {
    const uint32_t r = (uint32_t)w * (GC_ITEMS * 64) + k * 64 + lane;
    uint32_t x = sent;
    if (key[k] < n_hot) {
      if (key[k] - lo < R) x = key[k] - lo;
      else foreign = true;
    } else if (key[k] != EB_SENT) {
      x = R + (key[k] - n_hot);
    }
    key[k] = x;
    if (r < ns) kmax = max(kmax, x);
  }
  if (badc || foreign) hl_flag(err, HL_DEVERR_BAD_CODE);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) kmax = max(kmax, (uint32_t)__shfl_xor(kmax, o));
  if (lane == 0) atomicMax(&s_max, kmax);
  __syncthreads();
  const int bits = 32 - __clz(s_max);
  const int passes = (bits + GT_DBITS - 1) / GT_DBITS;  // 0: every key is 0, already in order
  const int b = passes ? (bits + passes - 1) / passes : 1;
  const uint32_t mask = (1u << b) - 1u;
  const uint64_t lt = (1ull << lane) - 1ull;
  for (int p = 0; p < passes; ++p) {
    const int shift = p * b;
    uint32_t dg[GC_ITEMS];
#pragma unroll
    for (int k = 0; k < GC_ITEMS; ++k) dg[k] = (key[k] >> shift) & mask;
    // The pass is stable iff the items of one digit keep their order.  First
    // try: every item adds 1 to its digit's counter of the wave and takes the
    // old value as its rank inside the wave; the order that gives to lanes of
    // one instruction with the same digit is not specified, so the pass is
    // checked after its scatter (equal digits next to each other must come
    // from increasing positions) and, if an order was broken, done again with
    // ranks that are stable by construction (ballot peer masks).
    for (int stable = ballot_only ? 1 : 0; stable < 2; ++stable) {
      uint32_t rk[GC_ITEMS];
#pragma unroll
      for (int k = 0; k < GC_ITEMS; ++k) {
        const uint32_t r = (uint32_t)w * (GC_ITEMS * 64) + k * 64 + lane;
        const bool valid = r < ns;
        if (!stable) {
          rk[k] = valid ? atomicAdd(&wcnt[w][dg[k]], 1u) : 0u;
        } else {
          const uint64_t peers = hl_match_digit(dg[k], b, valid);
          const int leader = __ffsll((unsigned long long)peers) - 1;
          uint32_t bs = 0;
          if (valid && lane == leader) bs = atomicAdd(&wcnt[w][dg[k]], (uint32_t)__popcll(peers));
          bs = __shfl(bs, leader < 0 ? 0 : leader);
          rk[k] = bs + (uint32_t)__popcll(peers & lt);
        }
      }
      __syncthreads();
      // per digit: offsets of the waves, then of the digits
      for (uint32_t d = tid; d <= mask; d += GC_THREADS) {
        uint32_t run = 0;
        for (int q = 0; q < GC_WAVES; ++q) {
          const uint32_t x = wcnt[q][d];
          wcnt[q][d] = run;
          run += x;
        }
        dofs[d] = run;
      }
      __syncthreads();
      // exclusive scan of the digit totals (GT_NB / GC_THREADS per thread)
      constexpr int PD = GT_NB / GC_THREADS;
      uint32_t loc[PD], sum = 0;
#pragma unroll
      for (int q = 0; q < PD; ++q) {
        const uint32_t d = tid * PD + q;
        loc[q] = d <= mask ? dofs[d] : 0u;
        sum += loc[q];
      }
      uint32_t all;
      uint32_t ex = gt_scan(sum, scan_ws, &all);
#pragma unroll
      for (int q = 0; q < PD; ++q) {
        const uint32_t d = tid * PD + q;
        if (d <= mask) dofs[d] = ex;
        ex += loc[q];
      }
      __syncthreads();
#pragma unroll
      for (int k = 0; k < GC_ITEMS; ++k) {
        const uint32_t r = (uint32_t)w * (GC_ITEMS * 64) + k * 64 + lane;
        if (r < ns) {
          const uint32_t q = dofs[dg[k]] + wcnt[w][dg[k]] + rk[k];
          sk[q] = key[k];
          sval[q] = val[k];
          spos[q] = r;
        }
      }
      __syncthreads();
      for (int j = tid; j < GC_WAVES * GT_NB; j += GC_THREADS) (&wcnt[0][0])[j] = 0;
      if (stable) break;
      bool broken = false;
#pragma unroll
      for (int k = 0; k < GC_ITEMS; ++k) {
        const uint32_t q = (uint32_t)w * (GC_ITEMS * 64) + k * 64 + lane;
        if (q > 0 && q < ns && ((sk[q] >> shift) & mask) == ((sk[q - 1] >> shift) & mask) && spos[q] < spos[q - 1])
          broken = true;
      }
      if (!__syncthreads_or(broken)) break;  // (also orders the counters' clearing before the next ranks)
    }
#pragma unroll
    for (int k = 0; k < GC_ITEMS; ++k) {
      const uint32_t r = (uint32_t)w * (GC_ITEMS * 64) + k * 64 + lane;
      if (r < ns) {
        key[k] = sk[r];
        val[k] = sval[r];
      }
    }
    __syncthreads();
  }
  uint32_t hc = 0;
  const uint64_t o = (uint64_t)t * E + s0;
#pragma unroll
  for (int k = 0; k < GC_ITEMS; ++k) {
    const uint32_t r = (uint32_t)w * (GC_ITEMS * 64) + k * 64 + lane;
    if (r < ns) {
      ck[o + r] = key[k];
      cv[o + r] = val[k];
      hc += key[k] < R ? 1u : 0u;
    }
  }
  uint32_t h;
  (void)gt_scan(hc, scan_ws, &h);
  if (tid == 0) {
    hcnt[blockIdx.x] = h;
    if (c == 0) {
      lor[2 * t] = lo;
      lor[2 * t + 1] = R;
    }
  }
}

// ----------------------------------------------------------------------------- merge
__global__ void __launch_bounds__(GC_THREADS)
gt_merge(const uint32_t* __restrict__ ck, const uint32_t* __restrict__ cv, int32_t T, uint32_t E, uint32_t C,
         uint32_t n, uint32_t n_hot, int32_t stg_rows, const uint32_t* __restrict__ hcnt,
         const uint32_t* __restrict__ lor, uint32_t* __restrict__ kout, uint32_t* __restrict__ vout, uint32_t* err,
         hl_hook hk) {
  extern __shared__ uint32_t lk[];  // the table's E sorted keys, chunk by chunk
  __shared__ uint32_t scan_ws[GC_WAVES];
  hl_hook_head(hk);  // a handover signal: the codes are complete (gt_chunk has ended)
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const uint32_t t = blockIdx.x / C, c = blockIdx.x - t * C;
  const uint64_t tb = (uint64_t)t * E;
  // the table's keys into LDS, 8 loads in flight per thread (tb is a multiple
  // of 4 when E is: 16-byte loads then)
  if ((E & 3) == 0) {
    const uint4* src = reinterpret_cast<const uint4*>(ck + tb);
    uint4* dst = reinterpret_cast<uint4*>(lk);
    const uint32_t n4 = E >> 2;
    for (uint32_t i0 = tid; i0 < n4; i0 += 8 * GC_THREADS) {
      uint4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = src[min(i0 + u * GC_THREADS, n4 - 1)];  // (all in flight)
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (i0 + u * GC_THREADS < n4) dst[i0 + u * GC_THREADS] = v[u];
    }
  } else {
    for (uint32_t i0 = tid; i0 < E; i0 += 8 * GC_THREADS) {
      uint32_t v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = ck[tb + min(i0 + u * GC_THREADS, E - 1)];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (i0 + u * GC_THREADS < E) lk[i0 + u * GC_THREADS] = v[u];
    }
  }
  // the hot pairs of the earlier tables and of this one
  uint32_t eh = 0, th = 0;
  for (uint32_t q = tid; q < (t + 1) * C; q += GC_THREADS) {
    const uint32_t x = hcnt[q];
    if (q < t * C) eh += x;
    else th += x;
  }
  uint32_t H, h;
  (void)gt_scan(eh, scan_ws, &H);
  (void)gt_scan(th, scan_ws, &h);  // (its barriers also order the LDS fill above)
  const uint32_t lo = lor[2 * t], R = lor[2 * t + 1];
  const uint32_t sent = R + (uint32_t)stg_rows;
  const uint64_t NH = (uint64_t)t * E - H;          // the earlier tables' other pairs
  const uint64_t nb0 = (uint64_t)n - NH - (E - h);  // this table's other pairs, before theirs
  const uint32_t s0 = c * GC;
  const uint32_t ns = min((uint32_t)GC, E - s0);
  // rank in the table: the chunk's own, plus the other chunks' keys before it
  uint32_t x[GC_ITEMS], g[GC_ITEMS];
#pragma unroll
  for (int k = 0; k < GC_ITEMS; ++k) {
    const uint32_t r = (uint32_t)w * (GC_ITEMS * 64) + k * 64 + lane;
    x[k] = r < ns ? lk[s0 + r] : 0u;
    g[k] = r;
  }
  // a chunk's keys not above x if it precedes this one (lookup order), below
  // x if it follows (keys are far below 2^32 - 1, so "not above x" is "below
  // x + 1"): a fixed number of halving steps written without branches, the
  // searches of the GC_ITEMS pairs interleaved
  const uint32_t cu = __builtin_amdgcn_readfirstlane(c);
  for (uint32_t c2 = 0; c2 < C; ++c2) {
    if (c2 == cu) continue;
    const uint32_t b0 = c2 * GC, n2 = min((uint32_t)GC, E - b0);
    const uint32_t inc = c2 < cu ? 1u : 0u;
    uint32_t pos[GC_ITEMS], xb[GC_ITEMS];
#pragma unroll
    for (int k = 0; k < GC_ITEMS; ++k) {
      pos[k] = 0;
      xb[k] = x[k] + inc;
    }
#pragma unroll
    for (int e = 10; e >= 0; --e) {  // steps 1024 .. 1 (GC = 1024)
      const uint32_t step = 1u << e;
#pragma unroll
      for (int k = 0; k < GC_ITEMS; ++k) {
        const uint32_t m = pos[k] + step;
        const uint32_t v = lk[b0 + min(m, n2) - 1];
        const uint32_t take = (uint32_t)(m <= n2) & (uint32_t)(v < xb[k]);
        pos[k] += take * step;
      }
    }
#pragma unroll
    for (int k = 0; k < GC_ITEMS; ++k) g[k] += pos[k];
  }
#pragma unroll
  for (int k = 0; k < GC_ITEMS; ++k) {
    const uint32_t r = (uint32_t)w * (GC_ITEMS * 64) + k * 64 + lane;
    if (r >= ns) continue;
    const uint32_t v = cv[tb + s0 + r];
    uint64_t p;
    uint32_t kk;
    if (x[k] < R) {
      p = (uint64_t)H + g[k];
      kk = x[k] + lo;
    } else {
      p = nb0 + (g[k] - h);
      kk = x[k] >= sent ? EB_SENT : n_hot + (x[k] - R);
    }
    if (p < n) {
      kout[p] = kk;
      vout[p] = v;
    } else {
      hl_flag(err, HL_DEVERR_INTERNAL);
    }
  }
}

// ----------------------------------------------------------------------------- host
bool hl_group_by_table_ok(const hl_handle* h, int64_t n_lookups, int64_t n_bags) {
  const int32_t T = h->n_tables;
  if (n_lookups != n_bags || n_bags == 0 || T > GT_TMAX || n_bags % T != 0) return false;
  return n_bags / T <= (int64_t)GT_CMAX * GC;
}

hl_status hl_group_by_table(hl_handle* h, int32_t* codes, const int32_t* bag_ptr, int64_t n_bags, int32_t stg_rows,
                            uint32_t* k_tm, uint32_t* v_tm, uint32_t* kout, uint32_t* vout, uint32_t* small,
                            uint32_t* sflag, uint32_t sv, const hl_cg_fused* cf, hipStream_t s) {
  const int32_t T = h->n_tables;
  const uint32_t E = (uint32_t)(n_bags / T);
  const uint32_t C = hl_div_up(E, GC);
  static_assert(HL_GROUP_SMALL >= GT_TMAX * GT_CMAX + 2 * GT_TMAX, "grouping counters");
  uint32_t* hcnt = small;                     // [T * C]
  uint32_t* lor = small + GT_TMAX * GT_CMAX;  // [2 T]
  const size_t lds = (size_t)E * sizeof(uint32_t);
  if (lds > 64 * 1024 &&
      hipFuncSetAttribute((const void*)gt_merge, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return HL_ERR_HIP;
  const hl_hook hk = hl_hook_take(h);  // carried by gt_merge (the first sort pass takes it on the other path)
  HL_KERNEL(h, s, "gt_chunk", gt_chunk, dim3(T * C), dim3(GC_THREADS), 0, s, codes, bag_ptr, n_bags, T, E, C,
            h->n_hot, h->k_cap, stg_rows, h->d_tb, k_tm, v_tm, hcnt, lor,
            n_bags, sflag, sv, h->d_err, cf ? *cf : hl_cg_fused{}, h->ballot_ranks);
  HL_KERNEL(h, s, "gt_merge", gt_merge, dim3(T * C), dim3(GC_THREADS), lds, s, k_tm, v_tm, T, E,
            C, (uint32_t)n_bags, h->n_hot, stg_rows, hcnt, lor, kout, vout, h->d_err, hk);
  HL_LAUNCHED();
  return HL_OK;
}
