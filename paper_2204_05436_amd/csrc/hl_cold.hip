// Cold-row gather of a mu-batch: the distinct non-hot rows its lookups need,
// in ascending id order, fetched from the pinned host table by the GPU over the
// host link, with the lookups' codes pointed at the staging rows.
//
//   collect  : (gid, lookup) of every selected lookup with code -1, appended
//              with one atomic per wave (order irrelevant: the result depends
//              only on the set of ids)
//   sort     : radix sort by gid (hl_sort.hip)
//   unique   : head flags in sorted order, decoupled look-back scan -> the
//              staging index of every sorted entry, and the count of cold rows
//   finalize : capacity check, then code rewrite, cold id list and row copy
#include "hl_internal.h"

#define CG_UTILE 2048  // 256 threads x 8 items
#define CG_C_COLLECT 0
#define CG_C_NCOLD 1
#define CG_C_UTILE 2
#define CG_C_SNAP 3

struct cg_ws {
  hl_sort_ws sort;
  uint32_t* ctr;     // [16]
  uint32_t* uidx;    // [n_max]
  uint64_t* ustat;   // [tiles]
  uint32_t utiles;
};

static void cg_carve(hl_carver& c, cg_ws& ws, uint32_t n_max) {
  hl_sort_ws_carve(c, ws.sort, n_max);
  ws.ctr = c.base ? c.header() + HL_HDR_COLD : nullptr;
  ws.uidx = c.take<uint32_t>(n_max);
  ws.utiles = n_max ? hl_div_up(n_max, CG_UTILE) : 1;
  ws.ustat = c.take<uint64_t>(ws.utiles);
}

size_t hl_cold_ws_bytes(const hl_handle* h, int64_t max_lookups) {
  (void)h;
  hl_carver c = hl_carver::after_header(nullptr, 0);
  cg_ws ws;
  cg_carve(c, ws, (uint32_t)max_lookups);
  return c.off;
}

// A block owns `spb` selected samples; their lookup ranges are laid end to end
// in LDS (start, exclusive prefix of lengths) and threads walk the
// concatenation, finding their sample by binary search.  Candidates are
// buffered in LDS and appended to the global list with one atomic per block
// (per flush), which keeps same-address atomics rare.
#define CG_MAX_SPB 512
#define CG_BUF 2048
__global__ void __launch_bounds__(256)
cg_collect(const uint32_t* __restrict__ gids, const int32_t* __restrict__ codes,
           const int32_t* __restrict__ bag_ptr, int32_t n_samples, int32_t bps,
           const int32_t* __restrict__ sample_ids, const int32_t* n_sel_dev, int32_t n_sel_max, int32_t spb,
           uint64_t n_rows, uint32_t* __restrict__ out_k, uint32_t* __restrict__ out_v, uint32_t n_max,
           uint32_t* ctr, uint64_t* ustat, uint32_t utiles, uint32_t* err) {
  __shared__ int32_t st[CG_MAX_SPB], pre[CG_MAX_SPB + 1];
  __shared__ uint32_t bk[CG_BUF], bv[CG_BUF];
  __shared__ uint32_t bn, bbase;
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < utiles; i += gridDim.x * blockDim.x) ustat[i] = 0;
  int32_t n_sel = n_sel_max;
  if (sample_ids && n_sel_dev) n_sel = min(max(*n_sel_dev, 0), n_sel_max);
  const int64_t q0 = (int64_t)blockIdx.x * spb;
  const int ns = (int)max((int64_t)0, min((int64_t)spb, (int64_t)n_sel - q0));
  for (int j = threadIdx.x; j < ns; j += blockDim.x) {
    const int64_t s = sample_ids ? sample_ids[q0 + j] : q0 + j;
    int32_t a = 0, b = 0;
    if (s >= 0 && s < n_samples) {
      a = bag_ptr[s * bps];
      b = bag_ptr[(s + 1) * bps];
    } else {
      hl_flag(err, HL_DEVERR_OUT_OF_RANGE);
    }
    st[j] = a;
    pre[j + 1] = b - a;
  }
  if (threadIdx.x == 0) {
    pre[0] = 0;
    bn = 0;
  }
  __syncthreads();
  if (threadIdx.x == 0)
    for (int j = 0; j < ns; ++j) pre[j + 1] += pre[j];
  __syncthreads();
  const int32_t total = pre[ns];
  const int lane = threadIdx.x & 63;
  const uint64_t lt = (1ull << lane) - 1ull;
  for (int32_t t0 = 0; t0 < total + (int32_t)blockDim.x; t0 += blockDim.x) {
    // flush when the next chunk might not fit, and once after the last chunk;
    // the barrier makes every wave see the same buffer fill
    __syncthreads();
    const bool last = t0 >= total;
    if (last || bn + blockDim.x > CG_BUF) {
      const uint32_t cnt = bn;
      if (threadIdx.x == 0 && cnt) bbase = atomicAdd(ctr + CG_C_COLLECT, cnt);
      __syncthreads();
      if (cnt) {
        for (uint32_t j = threadIdx.x; j < cnt; j += blockDim.x) {
          const uint32_t p = bbase + j;
          if (p < n_max) {  // a sample listed twice could overflow the buffer
            out_k[p] = bk[j];
            out_v[p] = bv[j];
          } else {
            hl_flag(err, HL_DEVERR_OUT_OF_RANGE);
          }
        }
      }
      __syncthreads();
      if (threadIdx.x == 0) bn = 0;
      __syncthreads();
    }
    if (last) break;
    const int32_t t = t0 + threadIdx.x;
    bool take = false;
    uint32_t g = 0;
    int32_t i = 0;
    if (t < total) {
      int a = 0, b = ns;
      while (b - a > 1) {
        int m = (a + b) >> 1;
        if (pre[m] <= t) a = m; else b = m;
      }
      i = st[a] + (t - pre[a]);
      if (codes[i] == -1) {
        g = gids[i];
        if (g < n_rows) take = true;
        else hl_flag(err, HL_DEVERR_OUT_OF_RANGE);
      }
    }
    const uint64_t m = __ballot(take);
    if (m) {
      uint32_t base = 0;
      if (lane == 0) base = atomicAdd(&bn, (uint32_t)__popcll(m));
      base = __shfl(base, 0);
      if (take) {
        const uint32_t p = base + (uint32_t)__popcll(m & lt);
        bk[p] = g;
        bv[p] = (uint32_t)i;
      }
    }
  }
}

__global__ void __launch_bounds__(256)
cg_unique(const uint32_t* __restrict__ keys, uint32_t* ctr, uint32_t n_host, uint64_t* ustat,
          uint32_t* __restrict__ uidx, int32_t* n_cold_dev, uint32_t epoch, uint32_t* err) {
  __shared__ uint32_t s_tile, wt[4];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  if (tid == 0) s_tile = atomicInc(ctr + CG_C_UTILE, gridDim.x - 1);
  __syncthreads();
  const uint32_t n = min(__hip_atomic_load(ctr + CG_C_COLLECT, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT), n_host);
  const uint32_t tile = s_tile;
  if (n == 0) {
    if (tile == 0 && tid == 0) {
      ctr[CG_C_NCOLD] = 0;
      ctr[CG_C_SNAP] = 0;
      *n_cold_dev = 0;
    }
    return;
  }
  const uint64_t tb = (uint64_t)tile * CG_UTILE;
  if (tb >= n) return;
  const uint64_t lt = (1ull << lane) - 1ull;
  bool hd[8];
  uint32_t wsum = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const uint64_t idx = tb + (uint64_t)w * 512 + k * 64 + lane;
    bool h = false;
    if (idx < n) h = idx == 0 || keys[idx] != keys[idx - 1];
    hd[k] = h;
    wsum += (uint32_t)__popcll(__ballot(h));
  }
  if (lane == 0) wt[w] = wsum;
  __syncthreads();
  uint32_t before = 0, tc = 0;
  for (int j = 0; j < 4; ++j) {
    if (j < w) before += wt[j];
    tc += wt[j];
  }
  __shared__ uint32_t s_excl;
  if (tid == 0) {
    uint64_t* st = ustat;
    hl_st_store(st + tile, hl_st_pack(epoch, tile == 0 ? HL_ST_PRE : HL_ST_AGG, tc));
    uint32_t ex = 0;
    if (tile > 0) {
      ex = hl_lookback(st, tile, 1, epoch, err);
      hl_st_store(st + tile, hl_st_pack(epoch, HL_ST_PRE, ex + tc));
    }
    s_excl = ex;
  }
  __syncthreads();
  uint32_t run = s_excl + before;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const uint64_t idx = tb + (uint64_t)w * 512 + k * 64 + lane;
    const uint64_t m = __ballot(hd[k]);
    const uint32_t incl = run + (uint32_t)__popcll(m & lt) + (hd[k] ? 1u : 0u);
    if (idx < n) uidx[idx] = incl - 1;
    if (idx == (uint64_t)n - 1) {
      ctr[CG_C_NCOLD] = incl;
      ctr[CG_C_SNAP] = n;
      *n_cold_dev = (int32_t)incl;
    }
    run += (uint32_t)__popcll(m);
  }
}

// Units of `U` bytes: thread (entry e, unit c).  Unit 0 of an entry rewrites the
// lookup's code; heads (first entry of each id) also record the id and copy
// their row from the host table.
template <typename V>
__global__ void __launch_bounds__(256)
cg_finalize(const uint32_t* __restrict__ keys, const uint32_t* __restrict__ vals,
            const uint32_t* __restrict__ uidx, uint32_t* ctr, int32_t cap, uint32_t k_cap,
            int32_t* __restrict__ codes, uint32_t* __restrict__ cold_ids, const V* __restrict__ src,
            V* __restrict__ dst, uint32_t upr, uint32_t* err) {
  const uint32_t n = ctr[CG_C_SNAP], ncold = ctr[CG_C_NCOLD];
  if (blockIdx.x == 0 && threadIdx.x == 0) ctr[CG_C_COLLECT] = 0;  // ready for the next call
  if (ncold > (uint32_t)cap) {
    if (blockIdx.x == 0 && threadIdx.x == 0) hl_flag(err, HL_DEVERR_CAPACITY);
    return;
  }
  const uint64_t total = (uint64_t)n * upr;
  for (uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
       t += (uint64_t)gridDim.x * blockDim.x) {
    const uint32_t e = (uint32_t)(t / upr), c = (uint32_t)(t - (uint64_t)e * upr);
    const uint32_t g = keys[e];
    const bool head = e == 0 || keys[e - 1] != g;
    const uint32_t u = uidx[e];
    if (c == 0) {
      codes[vals[e]] = (int32_t)(k_cap + u);
      if (head) cold_ids[u] = g;
    }
    if (head) dst[(uint64_t)u * upr + c] = src[(uint64_t)g * upr + c];
  }
}

extern "C" hl_status hl_cold_gather(hl_handle* h, const uint32_t* gids, int32_t* codes, const int32_t* bag_ptr,
                                    int32_t n_samples, int32_t bps, int64_t n_lookups,
                                    const int32_t* sample_ids, const int32_t* n_sel_dev, int32_t n_sel_max,
                                    const void* w_host, void* staging, int32_t cap, uint32_t* cold_ids_out,
                                    int32_t* n_cold_dev, void* workspace, size_t ws_bytes,
                                    hl_stream stream) {
  if (!h || n_samples < 0 || bps < 1 || n_lookups < 0 || n_sel_max < 0 || cap < 0) return HL_ERR_INVALID_ARG;
  if (!n_cold_dev || !bag_ptr || !workspace) return HL_ERR_INVALID_ARG;
  if (!sample_ids && n_sel_max > n_samples) return HL_ERR_INVALID_ARG;
  if (n_lookups > 0 && (!gids || !codes || !w_host || (cap > 0 && (!staging || !cold_ids_out))))
    return HL_ERR_INVALID_ARG;
  if (n_lookups >= (1ll << 30) || (uint64_t)h->k_cap + (uint64_t)cap >= (1ull << 31)) return HL_ERR_UNSUPPORTED;
  if (ws_bytes < hl_cold_ws_bytes(h, n_lookups)) return HL_ERR_CAPACITY;
  hipStream_t s = (hipStream_t)stream;
  hl_carver c = hl_carver::after_header(workspace, ws_bytes);
  cg_ws ws;
  cg_carve(c, ws, (uint32_t)n_lookups);
  const uint32_t n_max = (uint32_t)n_lookups;
  int64_t spb = n_lookups > 0 && n_samples > 0 ? (512ll * n_samples + n_lookups - 1) / n_lookups : CG_MAX_SPB;
  spb = spb < 1 ? 1 : (spb > CG_MAX_SPB ? CG_MAX_SPB : spb);
  const uint32_t cblocks = n_sel_max > 0 ? hl_div_up(n_sel_max, spb) : 1;
  HL_KERNEL(h, s, "cg_collect", cg_collect, dim3(cblocks), dim3(256), 0, s, gids, codes, bag_ptr, n_samples, bps, sample_ids,
                     n_sel_dev, n_sel_max, (int32_t)spb, h->n_rows, ws.sort.k0, ws.sort.v0, n_max, ws.ctr, ws.ustat,
                     ws.utiles, h->d_err);
  HL_LAUNCHED();
  uint32_t *sk, *sv;
  hl_status st = hl_sort_pairs(h, ws.sort, ws.ctr + CG_C_COLLECT, n_max, hl_bit_width(h->n_rows), s, &sk, &sv);
  if (st != HL_OK) return st;
  const uint32_t epoch = hl_next_epoch(h);
  const uint32_t ut = n_max ? hl_div_up(n_max, CG_UTILE) : 1;
  HL_KERNEL(h, s, "cg_unique", cg_unique, dim3(ut), dim3(256), 0, s, sk, ws.ctr, n_max, ws.ustat, ws.uidx, n_cold_dev,
                     epoch, h->d_err);
  const uint32_t rb = h->row_bytes;
  uint64_t total;
  uint32_t g;
#define CG_FIN(V)                                                                                      \
  total = (uint64_t)(n_max ? n_max : 1) * (rb / sizeof(V));                                            \
  g = hl_div_up(total, 256);                                                                           \
  if (g > 8192) g = 8192;                                                                              \
  HL_KERNEL(h, s, "cg_finalize", cg_finalize<V>, dim3(g), dim3(256), 0, s, sk, sv, ws.uidx, ws.ctr, cap, h->k_cap, \
                     codes, cold_ids_out, (const V*)w_host, (V*)staging, (uint32_t)(rb / sizeof(V)), h->d_err);
  if (rb % 16 == 0) { CG_FIN(uint4) }
  else if (rb % 8 == 0) { CG_FIN(uint2) }
  else if (rb % 4 == 0) { CG_FIN(uint32_t) }
  else { CG_FIN(uint16_t) }
#undef CG_FIN
  HL_LAUNCHED();
  return HL_OK;
}
