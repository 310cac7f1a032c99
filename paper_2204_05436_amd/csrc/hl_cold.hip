// Cold-row gather of a mu-batch: the distinct non-hot rows its lookups need,
// in order of first occurrence in the mini-batch's lookup order, fetched from
// the pinned host table by the GPU over the host link, with the lookups'
// codes pointed at the staging rows.
//
//   insert   : every selected lookup with code -1 enters an open-addressing
//              hash table keyed by row id; a 64-bit atomic min keeps the
//              smallest lookup index per id; the lookup is also appended to a
//              list (one atomic per block)
//   rank     : a scan over all lookups in index order (decoupled look-back)
//              numbers the first occurrences: staging row u of each id
//   codes    : capacity check, code rewrite and the cold id list
//   copy     : the row copy between the pinned host table and the staging
//              rows, in either direction (fetch before the mu-batch runs,
//              write-back of the updated rows after it)
// The plan (insert, rank, codes) uses the workspace, which is shared with
// other calls, so its table is cleared at the start of every call.  The copy
// reads only the cold id list and count, so it can run on a stream of its own
// while the popular mu-batch and the backward's grouping proceed (the overlap
// of the paper's pipeline, Sec. IV and Fig. "hotlinepipe").
#include "hl_internal.h"

#define CG_C_LIST 0
#define CG_C_NCOLD 1
#define CG_C_RTILE 2
#define CG_C_SNAP 3
#define CG_RTILE 8192     // lookups per rank tile (512 threads x 16)
#define CG_MAX_SPB 2048   // selected samples per insert block
#define CG_FIRST 0x80000000u

struct cg_ws {
  uint32_t* ctr;      // header counters
  uint64_t* table;    // [S] (id + 1) << 32 | smallest lookup index; 0 = empty
  uint32_t* uidx;     // [S] staging row of the id in the slot
  uint32_t* slotof;   // [n_max] slot of a cold lookup
  uint32_t* list;     // [n_max] lookup indices of the cold lookups
  uint32_t* fst;      // [n_max] id of staging row u
  uint64_t* rstat;    // [rtiles] look-back status of the rank scan
  uint32_t S, rtiles;
};

static uint32_t cg_table_slots(uint32_t n_max) {
  uint32_t s = 1024;
  while (s < 2u * n_max) s <<= 1;
  return s;
}

static void cg_carve(hl_carver& c, cg_ws& ws, uint32_t n_max) {
  ws.S = cg_table_slots(n_max);
  ws.rtiles = n_max ? hl_div_up(n_max, CG_RTILE) : 1;
  ws.ctr = c.base ? c.header() + HL_HDR_COLD : nullptr;
  ws.table = c.take<uint64_t>(ws.S);
  ws.uidx = c.take<uint32_t>(ws.S);
  ws.slotof = c.take<uint32_t>(n_max);
  ws.list = c.take<uint32_t>(n_max);
  ws.fst = c.take<uint32_t>(n_max);
  ws.rstat = c.take<uint64_t>(ws.rtiles);
}

size_t hl_cold_ws_bytes(const hl_handle* h, int64_t max_lookups) {
  (void)h;
  hl_carver c = hl_carver::after_header(nullptr, 0);
  cg_ws ws;
  cg_carve(c, ws, (uint32_t)max_lookups);
  return c.off;
}

__device__ __forceinline__ uint32_t cg_hash(uint32_t x) {  // 32-bit finalising mix
  x ^= x >> 16;
  x *= 0x85EBCA6Bu;
  x ^= x >> 13;
  x *= 0xC2B2AE35u;
  x ^= x >> 16;
  return x;
}

__global__ void __launch_bounds__(256) cg_clear(cg_ws ws) {
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < ws.S; i += gridDim.x * blockDim.x) ws.table[i] = 0;
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < ws.rtiles; i += gridDim.x * blockDim.x)
    ws.rstat[i] = 0;
}

// A block owns `spb` consecutive selected samples; their lookup ranges are laid
// end to end in LDS (start, inclusive prefix of lengths) and threads walk the
// concatenation in rounds of 8 positions per thread, finding their sample by
// binary search.  Each round issues its loads stage by stage for all 8
// positions (codes, then ids, then the first hash probe) so that they overlap.
#define CG_IPT 8
__global__ void __launch_bounds__(256)
cg_insert(const uint32_t* __restrict__ gids, const int32_t* __restrict__ codes,
          const int32_t* __restrict__ bag_ptr, int32_t n_samples, int32_t bps,
          const int32_t* __restrict__ sample_ids, const int32_t* n_sel_dev, int32_t n_sel_max, int32_t spb,
          uint64_t n_rows, cg_ws ws, uint32_t n_max, uint32_t* err) {
  __shared__ int32_t st[CG_MAX_SPB], pre[CG_MAX_SPB + 1];
  __shared__ uint32_t buf[256 * CG_IPT];
  __shared__ uint32_t bn, bbase, wsum[4];
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
  if (threadIdx.x == 0) pre[0] = 0;
  __syncthreads();
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  {  // block-wide inclusive scan of the lengths (up to 8 per thread, blocked)
    const int per = (ns + 255) / 256;
    uint32_t loc = 0;
    for (int k = 0; k < per; ++k) {
      const int j = threadIdx.x * per + k;
      if (j < ns) loc += (uint32_t)pre[j + 1];
    }
    uint32_t inc = loc;
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t t = __shfl_up(inc, o);
      if (lane >= o) inc += t;
    }
    if (lane == 63) wsum[w] = inc;
    __syncthreads();
    uint32_t run = inc - loc;
    for (int j = 0; j < w; ++j) run += wsum[j];
    for (int k = 0; k < per; ++k) {
      const int j = threadIdx.x * per + k;
      if (j < ns) {
        run += (uint32_t)pre[j + 1];
        pre[j + 1] = (int32_t)run;
      }
    }
  }
  __syncthreads();
  const int32_t total = pre[ns];
  const uint64_t lt = (1ull << lane) - 1ull;
  const uint32_t smask = ws.S - 1;
  for (int32_t r0 = 0; r0 < total; r0 += 256 * CG_IPT) {
    if (threadIdx.x == 0) bn = 0;
    int32_t idx[CG_IPT];
    int32_t cd[CG_IPT];
    uint32_t g[CG_IPT], slot[CG_IPT];
    uint64_t cur[CG_IPT];
#pragma unroll
    for (int k = 0; k < CG_IPT; ++k) {
      const int32_t t = r0 + k * 256 + threadIdx.x;
      idx[k] = -1;
      if (t < total) {
        int a = 0, b = ns;
        while (b - a > 1) {
          int m = (a + b) >> 1;
          if (pre[m] <= t) a = m; else b = m;
        }
        idx[k] = st[a] + (t - pre[a]);
      }
    }
#pragma unroll
    for (int k = 0; k < CG_IPT; ++k) cd[k] = idx[k] >= 0 ? codes[idx[k]] : 0;
#pragma unroll
    for (int k = 0; k < CG_IPT; ++k) g[k] = (idx[k] >= 0 && cd[k] == -1) ? gids[idx[k]] : 0xFFFFFFFFu;
#pragma unroll
    for (int k = 0; k < CG_IPT; ++k) {
      if (idx[k] >= 0 && cd[k] == -1 && g[k] >= n_rows) hl_flag(err, HL_DEVERR_OUT_OF_RANGE);
      slot[k] = cg_hash(g[k]) & smask;
      cur[k] = g[k] < n_rows ? ws.table[slot[k]] : 0ull;
    }
    bool take[CG_IPT];
#pragma unroll
    for (int k = 0; k < CG_IPT; ++k) {
      take[k] = g[k] < n_rows;
      if (!take[k]) continue;
      const uint64_t want = ((uint64_t)(g[k] + 1) << 32) | (uint32_t)idx[k];
      uint64_t c = cur[k];
      for (uint32_t probe = 0; probe <= smask; ++probe) {
        if ((c >> 32) == 0) {
          c = atomicCAS((unsigned long long*)(ws.table + slot[k]), 0ull, (unsigned long long)want);
          if (c == 0) break;
        }
        if ((uint32_t)(c >> 32) == g[k] + 1) {
          atomicMin((unsigned long long*)(ws.table + slot[k]), (unsigned long long)want);
          break;
        }
        slot[k] = (slot[k] + 1) & smask;
        c = ws.table[slot[k]];
      }
      ws.slotof[idx[k]] = slot[k];
    }
    __syncthreads();  // bn reset visible
#pragma unroll
    for (int k = 0; k < CG_IPT; ++k) {
      const uint64_t m = __ballot(take[k]);
      if (m) {
        uint32_t base = 0;
        if (lane == 0) base = atomicAdd(&bn, (uint32_t)__popcll(m));
        base = __shfl(base, 0);
        if (take[k]) buf[base + (uint32_t)__popcll(m & lt)] = (uint32_t)idx[k];
      }
    }
    __syncthreads();
    const uint32_t cnt = bn;
    if (threadIdx.x == 0 && cnt) bbase = atomicAdd(ws.ctr + CG_C_LIST, cnt);
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < cnt; j += blockDim.x) {
      const uint32_t p = bbase + j;
      if (p < n_max) ws.list[p] = buf[j];
      else hl_flag(err, HL_DEVERR_OUT_OF_RANGE);  // a sample listed twice
    }
    __syncthreads();
  }
}

// Scan over the mini-batch's lookups in index order.  Lookup i is a first
// occurrence iff it is a cold lookup of this call whose slot holds (its id,
// i); the running count of first occurrences numbers the staging rows.  Tiles
// of 8192 lookups (512 threads x 16), so one look-back window reaches tile 0.
#define CG_RT_THREADS 512
#define CG_RT_ITEMS 16
__global__ void __launch_bounds__(CG_RT_THREADS)
cg_rank(const uint32_t* __restrict__ gids, const int32_t* __restrict__ codes, uint32_t n_lookups, cg_ws ws,
        int32_t* n_cold_dev, uint32_t epoch, uint32_t* err) {
  __shared__ uint32_t s_tile, wt[CG_RT_THREADS / 64], s_excl;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  if (tid == 0) s_tile = atomicInc(ws.ctr + CG_C_RTILE, gridDim.x - 1);
  __syncthreads();
  const uint32_t tile = s_tile;
  if (tile == 0 && tid == 0) ws.ctr[CG_C_SNAP] = ws.ctr[CG_C_LIST];
  if (n_lookups == 0) {
    if (tile == 0 && tid == 0) {
      ws.ctr[CG_C_NCOLD] = 0;
      *n_cold_dev = 0;
    }
    return;
  }
  const uint64_t tb = (uint64_t)tile * CG_RTILE;
  if (tb >= n_lookups) return;
  const uint64_t lt = (1ull << lane) - 1ull;
  bool first[CG_RT_ITEMS];
  int32_t cd[CG_RT_ITEMS];
  uint32_t slot[CG_RT_ITEMS], g[CG_RT_ITEMS];
#pragma unroll
  for (int k = 0; k < CG_RT_ITEMS; ++k) {
    const uint64_t i = tb + (uint64_t)w * (64 * CG_RT_ITEMS) + k * 64 + lane;
    cd[k] = i < n_lookups ? codes[i] : 0;
  }
#pragma unroll
  for (int k = 0; k < CG_RT_ITEMS; ++k) {
    const uint64_t i = tb + (uint64_t)w * (64 * CG_RT_ITEMS) + k * 64 + lane;
    slot[k] = cd[k] == -1 ? ws.slotof[i] : 0xFFFFFFFFu;
    g[k] = cd[k] == -1 ? gids[i] : 0u;
  }
  uint32_t wsum = 0;
#pragma unroll
  for (int k = 0; k < CG_RT_ITEMS; ++k) {
    const uint64_t i = tb + (uint64_t)w * (64 * CG_RT_ITEMS) + k * 64 + lane;
    bool f = false;
    if (slot[k] < ws.S)  // a slot from an earlier call fails the test below
      f = ws.table[slot[k]] == (((uint64_t)(g[k] + 1) << 32) | (uint32_t)i);
    first[k] = f;
    wsum += (uint32_t)__popcll(__ballot(f));
  }
  if (lane == 0) wt[w] = wsum;
  __syncthreads();
  uint32_t before = 0, tc = 0;
  for (int j = 0; j < CG_RT_THREADS / 64; ++j) {
    if (j < w) before += wt[j];
    tc += wt[j];
  }
  if (tid == 0) {
    hl_st_store(ws.rstat + tile, hl_st_pack(epoch, tile == 0 ? HL_ST_PRE : HL_ST_AGG, tc));
    uint32_t ex = 0;
    if (tile > 0) {
      ex = hl_lookback(ws.rstat, tile, 1, epoch, err);
      hl_st_store(ws.rstat + tile, hl_st_pack(epoch, HL_ST_PRE, ex + tc));
    }
    s_excl = ex;
  }
  __syncthreads();
  uint32_t run = s_excl + before;
#pragma unroll
  for (int k = 0; k < CG_RT_ITEMS; ++k) {
    const uint64_t i = tb + (uint64_t)w * (64 * CG_RT_ITEMS) + k * 64 + lane;
    const uint64_t m = __ballot(first[k]);
    if (first[k]) {
      const uint32_t u = run + (uint32_t)__popcll(m & lt);
      ws.uidx[slot[k]] = u;
      ws.fst[u] = g[k];
    }
    run += (uint32_t)__popcll(m);
    if (i == (uint64_t)n_lookups - 1) {
      ws.ctr[CG_C_NCOLD] = run;
      *n_cold_dev = (int32_t)run;
    }
  }
}

// Every listed cold lookup points its code at its staging row; cold_ids[u] =
// id of staging row u.  Nothing but the error bit and the list reset when the
// rows do not fit.
__global__ void __launch_bounds__(256)
cg_codes(cg_ws ws, uint32_t n_max, int32_t cap, uint32_t k_cap, int32_t* __restrict__ codes,
         uint32_t* __restrict__ cold_ids, uint32_t* err) {
  const uint32_t n_list = min(ws.ctr[CG_C_SNAP], n_max), ncold = ws.ctr[CG_C_NCOLD];
  const bool fits = ncold <= (uint32_t)cap;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    ws.ctr[CG_C_LIST] = 0;  // ready for the next call
    if (!fits) hl_flag(err, HL_DEVERR_CAPACITY);
  }
  if (!fits) return;
  const uint32_t gs = gridDim.x * blockDim.x, t0 = blockIdx.x * blockDim.x + threadIdx.x;
  for (uint32_t e = t0; e < n_list; e += gs) {
    const uint32_t i = ws.list[e];
    codes[i] = (int32_t)(k_cap + ws.uidx[ws.slotof[i]]);
  }
  for (uint32_t u = t0; u < ncold; u += gs) cold_ids[u] = ws.fst[u];
}

// Row copy between host table and staging rows: TO_HOST = 0 copies
// staging[u] = host[ids[u]], TO_HOST = 1 copies host[ids[u]] = staging[u], for
// u < *n_dev.  A count above cap copies nothing and sets the capacity bit; an
// id >= n_rows is skipped and sets the range bit.  The grid is kept small (the
// host link, not the CUs, bounds it) and each thread keeps 4 units in flight.
template <typename V, bool TO_HOST>
__global__ void __launch_bounds__(256)
cg_copy(const uint32_t* __restrict__ ids, const int32_t* n_dev, int32_t cap, uint64_t n_rows, V* host, V* stg,
        uint32_t upr, uint32_t* err) {
  const int32_t nd = *n_dev;
  if (nd < 0 || nd > cap) {
    if (blockIdx.x == 0 && threadIdx.x == 0) hl_flag(err, nd < 0 ? HL_DEVERR_OUT_OF_RANGE : HL_DEVERR_CAPACITY);
    return;
  }
  const uint64_t total = (uint64_t)nd * upr, gs = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t t0 = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; t0 < total; t0 += 4 * gs) {
    V v[4];
    uint64_t dst[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint64_t t = t0 + k * gs;
      dst[k] = ~0ull;
      if (t < total) {
        const uint32_t u = (uint32_t)(t / upr), c = (uint32_t)(t - (uint64_t)u * upr);
        const uint32_t g = ids[u];
        if (g < n_rows) {
          const uint64_t hp = (uint64_t)g * upr + c, sp = (uint64_t)u * upr + c;
          v[k] = TO_HOST ? stg[sp] : host[hp];
          dst[k] = TO_HOST ? hp : sp;
        } else if (c == 0) {
          hl_flag(err, HL_DEVERR_OUT_OF_RANGE);
        }
      }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (dst[k] != ~0ull) {
        if (TO_HOST) host[dst[k]] = v[k];
        else stg[dst[k]] = v[k];
      }
    }
  }
}

static hl_status cg_launch_copy(hl_handle* h, const uint32_t* ids, const int32_t* n_dev, int32_t cap, void* host,
                                void* stg, bool to_host, hipStream_t s) {
  const uint32_t rb = h->row_bytes;
  uint64_t units = (uint64_t)(cap > 0 ? cap : 1) * (rb / 4);
  uint32_t g = (uint32_t)((units + 1023) / 1024);
  g = g < 1 ? 1 : (g > 512 ? 512 : g);
#define CG_COPY(V)                                                                                             \
  if (to_host)                                                                                                 \
    HL_KERNEL(h, s, "cg_scatter", (cg_copy<V, true>), dim3(g), dim3(256), 0, s, ids, n_dev, cap, h->n_rows,     \
              (V*)host, (V*)stg, (uint32_t)(rb / sizeof(V)), h->d_err);                                        \
  else                                                                                                         \
    HL_KERNEL(h, s, "cg_fetch", (cg_copy<V, false>), dim3(g), dim3(256), 0, s, ids, n_dev, cap, h->n_rows,      \
              (V*)host, (V*)stg, (uint32_t)(rb / sizeof(V)), h->d_err);
  if (rb % 16 == 0 && ((uintptr_t)host | (uintptr_t)stg) % 16 == 0) { CG_COPY(uint4) }
  else if (rb % 8 == 0 && ((uintptr_t)host | (uintptr_t)stg) % 8 == 0) { CG_COPY(uint2) }
  else if (rb % 4 == 0 && ((uintptr_t)host | (uintptr_t)stg) % 4 == 0) { CG_COPY(uint32_t) }
  else { CG_COPY(uint16_t) }
#undef CG_COPY
  HL_LAUNCHED();
  return HL_OK;
}

extern "C" hl_status hl_cold_plan(hl_handle* h, const uint32_t* gids, int32_t* codes, const int32_t* bag_ptr,
                                  int32_t n_samples, int32_t bps, int64_t n_lookups, const int32_t* sample_ids,
                                  const int32_t* n_sel_dev, int32_t n_sel_max, int32_t cap, uint32_t* cold_ids_out,
                                  int32_t* n_cold_dev, void* workspace, size_t ws_bytes, hl_stream stream) {
  if (!h || n_samples < 0 || bps < 1 || n_lookups < 0 || n_sel_max < 0 || cap < 0) return HL_ERR_INVALID_ARG;
  if (!n_cold_dev || !bag_ptr || !workspace) return HL_ERR_INVALID_ARG;
  if (!sample_ids && n_sel_max > n_samples) return HL_ERR_INVALID_ARG;
  if (n_lookups > 0 && (!gids || !codes || (cap > 0 && !cold_ids_out))) return HL_ERR_INVALID_ARG;
  if (n_lookups >= (1ll << 30) || (uint64_t)h->k_cap + (uint64_t)cap >= (1ull << 31)) return HL_ERR_UNSUPPORTED;
  if (ws_bytes < hl_cold_ws_bytes(h, n_lookups)) return HL_ERR_CAPACITY;
  hl_ws_note(h, workspace, HL_WSK_OTHER);
  hipStream_t s = (hipStream_t)stream;
  hl_carver c = hl_carver::after_header(workspace, ws_bytes);
  cg_ws ws;
  cg_carve(c, ws, (uint32_t)n_lookups);
  const uint32_t n_max = (uint32_t)n_lookups;
  // about 2048 lookups per insert block
  int64_t spb = n_lookups > 0 && n_samples > 0 ? (2048ll * n_samples + n_lookups - 1) / n_lookups : CG_MAX_SPB;
  spb = spb < 1 ? 1 : (spb > CG_MAX_SPB ? CG_MAX_SPB : spb);
  const uint32_t iblocks = n_sel_max > 0 ? hl_div_up(n_sel_max, spb) : 1;
  uint32_t cb = hl_div_up(ws.S, 256 * 4);
  HL_KERNEL(h, s, "cg_clear", cg_clear, dim3(cb), dim3(256), 0, s, ws);
  HL_KERNEL(h, s, "cg_insert", cg_insert, dim3(iblocks), dim3(256), 0, s, gids, codes, bag_ptr, n_samples, bps,
            sample_ids, n_sel_dev, n_sel_max, (int32_t)spb, h->n_rows, ws, n_max, h->d_err);
  const uint32_t epoch = hl_next_epoch(h);
  HL_KERNEL(h, s, "cg_rank", cg_rank, dim3(ws.rtiles), dim3(CG_RT_THREADS), 0, s, gids, codes, n_max, ws, n_cold_dev, epoch,
            h->d_err);
  uint32_t g = hl_div_up(n_max ? n_max : 1, 256);
  if (g > 1024) g = 1024;
  HL_KERNEL(h, s, "cg_codes", cg_codes, dim3(g), dim3(256), 0, s, ws, n_max, cap, h->k_cap, codes, cold_ids_out,
            h->d_err);
  HL_LAUNCHED();
  return HL_OK;
}

extern "C" hl_status hl_cold_fetch(hl_handle* h, const uint32_t* cold_ids, const int32_t* n_cold_dev, int32_t cap,
                                   const void* w_host, void* staging, hl_stream stream) {
  if (!h || cap < 0 || !n_cold_dev) return HL_ERR_INVALID_ARG;
  if (cap > 0 && (!cold_ids || !w_host || !staging)) return HL_ERR_INVALID_ARG;
  if (cap == 0) return HL_OK;
  return cg_launch_copy(h, cold_ids, n_cold_dev, cap, const_cast<void*>(w_host), staging, false, (hipStream_t)stream);
}

extern "C" hl_status hl_cold_scatter(hl_handle* h, const uint32_t* cold_ids, const int32_t* n_cold_dev, int32_t cap,
                                     const void* staging, void* w_host, hl_stream stream) {
  if (!h || cap < 0 || !n_cold_dev) return HL_ERR_INVALID_ARG;
  if (cap > 0 && (!cold_ids || !w_host || !staging)) return HL_ERR_INVALID_ARG;
  if (cap == 0) return HL_OK;
  return cg_launch_copy(h, cold_ids, n_cold_dev, cap, w_host, const_cast<void*>(staging), true, (hipStream_t)stream);
}

extern "C" hl_status hl_cold_gather(hl_handle* h, const uint32_t* gids, int32_t* codes, const int32_t* bag_ptr,
                                    int32_t n_samples, int32_t bps, int64_t n_lookups,
                                    const int32_t* sample_ids, const int32_t* n_sel_dev, int32_t n_sel_max,
                                    const void* w_host, void* staging, int32_t cap, uint32_t* cold_ids_out,
                                    int32_t* n_cold_dev, void* workspace, size_t ws_bytes,
                                    hl_stream stream) {
  if (h && n_lookups > 0 && cap > 0 && (!w_host || !staging)) return HL_ERR_INVALID_ARG;
  hl_status st = hl_cold_plan(h, gids, codes, bag_ptr, n_samples, bps, n_lookups, sample_ids, n_sel_dev, n_sel_max,
                              cap, cold_ids_out, n_cold_dev, workspace, ws_bytes, stream);
  if (st != HL_OK || n_lookups == 0) return st;
  return hl_cold_fetch(h, cold_ids_out, n_cold_dev, cap, w_host, staging, stream);
}
