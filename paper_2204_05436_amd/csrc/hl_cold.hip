// Cold-row gather of a mu-batch: the distinct non-hot rows its lookups need,
// in order of first occurrence in the mini-batch's lookup order, fetched from
// the pinned host table by the GPU over the host link, with the lookups'
// codes pointed at the staging rows.
//
//   insert : a block per 256 bags; each round a wave compacts its cold
//            lookups (code -1, sample selected) so that a lane handles about
//            one, which enters an open-addressing hash table keyed by row id
//            with one CAS (a 64-bit atomic min keeps the smallest lookup index
//            per id); the block lists its cold lookups in its own lookup range
//   rank   : a scan over all lookups in index order (tiles of 2048, decoupled
//            look-back read by the whole block) numbers the first occurrences:
//            staging row u of each id
//   codes  : capacity check, code rewrite, the cold id list, and the clearing
//            of the table slots this call used
//   copy   : the row copy between the pinned host table and the staging rows,
//            in either direction (fetch before the mu-batch runs, write-back
//            of the updated rows after it)
// The hash table belongs to the handle (cleared once, then left clean by every
// call); the rest lives in the workspace.  The copy reads only the cold id
// list and count, so it can run on a stream of its own while the popular
// mu-batch and the backward's grouping proceed (the overlap of the paper's
// pipeline, Sec. IV and Fig. "hotlinepipe").
#include "hl_internal.h"

#define CG_C_NCOLD 1
#define CG_C_RTILE 2
#define CG_BAGS 256      // bags per insert block (at most; fewer for bags of many lookups)
#define CG_BAGS_MIN 64
#define CG_IR 1024       // lookup positions per insert round (256 threads x 4)
#define CG_RT_THREADS 512
#define CG_RT (CG_RT_THREADS * 4)  // lookups per rank tile

struct cg_ws {
  uint32_t* ctr;      // header counters
  uint32_t* uidx;     // [S] staging row of the id in the slot
  uint32_t* slotof;   // [n_max] slot of a cold lookup
  uint32_t* blist;    // [n_max] cold lookups of insert block b at [bag_ptr[b * bpb], ...)
  uint32_t* bcnt;     // [iblocks] their number
  uint32_t* fst;      // [n_max] id of staging row u
  uint64_t* rstat;    // [rtiles] look-back status of the rank scan
  uint8_t* mask;      // [max_samples] selected samples (when a sample list is given)
  uint32_t S, rtiles, iblocks;
};

static uint32_t cg_table_slots(uint32_t n_max) {
  uint32_t s = 1024;
  while (s < 2u * n_max) s <<= 1;
  return s;
}

static void cg_carve(hl_carver& c, cg_ws& ws, uint32_t n_max, int64_t n_bags, int32_t n_samples) {
  ws.S = cg_table_slots(n_max);
  ws.rtiles = n_max ? hl_div_up(n_max, CG_RT) : 1;
  ws.iblocks = n_bags > 0 ? hl_div_up((uint64_t)n_bags, CG_BAGS_MIN) : 1;
  ws.ctr = c.base ? c.header() + HL_HDR_COLD : nullptr;
  ws.uidx = c.take<uint32_t>(ws.S);
  ws.slotof = c.take<uint32_t>(n_max);
  ws.blist = c.take<uint32_t>(n_max);
  ws.bcnt = c.take<uint32_t>(ws.iblocks);
  ws.fst = c.take<uint32_t>(n_max);
  ws.rstat = c.take<uint64_t>(ws.rtiles);
  ws.mask = c.take<uint8_t>((size_t)n_samples + 1);
}

size_t hl_cold_ws_bytes(const hl_handle* h, int64_t max_lookups, int64_t max_bags, int32_t max_samples) {
  (void)h;
  hl_carver c = hl_carver::after_header(nullptr, 0);
  cg_ws ws;
  cg_carve(c, ws, (uint32_t)max_lookups, max_bags, max_samples);
  return c.off;
}

// The handle's hash table, (id + 1) << 32 | smallest lookup index per slot, 0
// = empty; grown (and zeroed) when a call needs more slots.  The growth
// allocates, so a caller that captures calls into a graph reserves the largest
// size first (hl_cold_reserve).
static hl_status cg_table(hl_handle* h, uint32_t S, hipStream_t s, uint64_t** out) {
  if (h->cg_slots < S) {
    if (h->cg_table) {
      if (hipFree(h->cg_table) != hipSuccess) return HL_ERR_HIP;
      h->cg_table = nullptr;
      h->cg_slots = 0;
    }
    if (hipMalloc(&h->cg_table, (size_t)S * 8) != hipSuccess) return HL_ERR_HIP;
    h->cg_slots = S;
    hl_status st = hl_fill32((uint32_t*)h->cg_table, (uint64_t)S * 2, 0, s);
    if (st != HL_OK) return st;
  }
  *out = h->cg_table;
  return HL_OK;
}

__global__ void cg_mask(uint8_t* mask, int32_t n_samples, const int32_t* __restrict__ ids, const int32_t* n_dev,
                        int32_t n_max, int phase, uint32_t* err) {
  if (phase == 0) {
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n_samples; i += gridDim.x * blockDim.x) mask[i] = 0;
  } else {
    int32_t n = n_max;
    if (n_dev) n = min(max(*n_dev, 0), n_max);
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
      const int32_t s = ids[i];
      if (s >= 0 && s < n_samples) mask[s] = 1;
      else hl_flag(err, HL_DEVERR_OUT_OF_RANGE);
    }
  }
}

__global__ void __launch_bounds__(256)
cg_insert(const uint32_t* __restrict__ gids, const int32_t* __restrict__ codes, const int32_t* __restrict__ bag_ptr,
          int64_t n_bags, int32_t bps, int32_t bpb, const uint8_t* __restrict__ mask, uint32_t n_lookups,
          uint64_t n_rows, uint64_t* table, cg_ws ws, uint32_t* err) {
  __shared__ int32_t off[CG_BAGS + 1];
  __shared__ uint32_t cl[CG_IR], cg_[CG_IR];
  __shared__ uint32_t wn[4];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int64_t b0 = (int64_t)blockIdx.x * bpb;
  const int nb = (int)min((int64_t)bpb, n_bags - b0);
  for (int j = tid; j <= nb; j += 256) off[j] = bag_ptr[b0 + j];
  __syncthreads();
  const int32_t lo = off[0], hi = (int32_t)min((int64_t)off[nb], (int64_t)n_lookups);
  // the rank scan's status words, cleared for the kernel that follows
  for (uint32_t j = blockIdx.x * 256 + tid; j < ws.rtiles; j += gridDim.x * 256) ws.rstat[j] = 0;
  const uint64_t lt = (1ull << lane) - 1ull;
  const uint32_t smask = ws.S - 1;
  uint32_t listed = 0;  // block-wide count so far (uniform)
  for (int32_t r0 = lo; r0 < hi; r0 += CG_IR) {
    // positions r0 + k*256 + tid: cold and selected?
    bool cold[4];
    int32_t pos[4];
    uint32_t gg[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {  // codes and ids loaded together
      pos[k] = r0 + k * 256 + tid;
      const bool in = pos[k] < hi;
      cold[k] = in && codes[pos[k]] == -1;
      gg[k] = in ? gids[pos[k]] : 0u;
    }
    if (mask) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (!cold[k]) continue;
        int a = 0, b = nb;
        while (b - a > 1) {
          const int m = (a + b) >> 1;
          if (off[m] <= pos[k]) a = m; else b = m;
        }
        cold[k] = mask[(b0 + a) / bps] != 0;
      }
    }
    // compact the round's cold positions into cl (wave-major, then item, then lane)
    uint32_t c = 0;
    uint64_t m[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      m[k] = __ballot(cold[k]);
      c += (uint32_t)__popcll(m[k]);
    }
    if (lane == 0) wn[w] = c;
    __syncthreads();
    uint32_t base = 0, tot = 0;
    for (int q = 0; q < 4; ++q) {
      if (q < w) base += wn[q];
      tot += wn[q];
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (cold[k]) {
        cl[base + (uint32_t)__popcll(m[k] & lt)] = (uint32_t)pos[k];
        cg_[base + (uint32_t)__popcll(m[k] & lt)] = gg[k];
      }
      base += (uint32_t)__popcll(m[k]);
    }
    __syncthreads();
    // each thread inserts about one lookup
    for (uint32_t e = tid; e < tot; e += 256) {
      const uint32_t i = cl[e];
      const uint32_t g = cg_[e];
      if (g >= n_rows) {
        hl_flag(err, HL_DEVERR_OUT_OF_RANGE);
        ws.slotof[i] = 0xFFFFFFFFu;
        continue;
      }
      ws.slotof[i] = hl_cg_insert(table, smask, g, i);
      ws.blist[lo + listed + e] = i;
    }
    listed += tot;
    __syncthreads();  // cl and wn reused
  }
  if (tid == 0) ws.bcnt[blockIdx.x] = listed;
}

// Lookup i is a first occurrence iff it is a cold lookup of this call whose
// slot holds (its id, i); the running count of first occurrences numbers the
// staging rows.  In the fused plan (fused = 1) the ids of staging rows below
// cap go straight to the cold id list.
__global__ void __launch_bounds__(CG_RT_THREADS)
cg_rank(const uint32_t* __restrict__ gids, const int32_t* __restrict__ codes, uint32_t n_lookups,
        const uint64_t* __restrict__ table, cg_ws ws, int32_t* n_cold_dev, uint32_t epoch, uint32_t* cold_ids,
        int32_t cap, int fused, uint32_t* err) {
  __shared__ uint32_t s_tile, wt[CG_RT_THREADS / 64];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  if (tid == 0) s_tile = atomicInc(ws.ctr + CG_C_RTILE, gridDim.x - 1);
  __syncthreads();
  const uint32_t tile = s_tile;
  if (n_lookups == 0) {
    if (tile == 0 && tid == 0) {
      ws.ctr[CG_C_NCOLD] = 0;
      *n_cold_dev = 0;
    }
    return;
  }
  const uint64_t tb = (uint64_t)tile * CG_RT;
  if (tb >= n_lookups) return;
  const uint64_t lt = (1ull << lane) - 1ull;
  int32_t cd[4];
  uint32_t slot[4], g[4];
  bool first[4];
  // codes, slots and ids loaded together (the slot and id only matter for code -1)
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint64_t i = tb + w * 256 + k * 64 + lane;
    const bool in = i < n_lookups;
    cd[k] = in ? codes[i] : 0;
    slot[k] = in ? ws.slotof[i] : 0xFFFFFFFFu;
    g[k] = in ? gids[i] : 0u;
  }
#pragma unroll
  for (int k = 0; k < 4; ++k)
    if (cd[k] != -1) slot[k] = 0xFFFFFFFFu;
  uint32_t wsum = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint64_t i = tb + w * 256 + k * 64 + lane;
    bool f = false;
    if (slot[k] < ws.S)  // a slot left by an earlier call fails the test below
      f = table[slot[k]] == (((uint64_t)(g[k] + 1) << 32) | (uint32_t)i);
    first[k] = f;
    wsum += (uint32_t)__popcll(__ballot(f));
  }
  if (lane == 0) wt[w] = wsum;
  __syncthreads();
  uint32_t before = 0, tc = 0;
  for (int q = 0; q < CG_RT_THREADS / 64; ++q) {
    if (q < w) before += wt[q];
    tc += wt[q];
  }
  if (tid == 0) hl_st_store(ws.rstat + tile, hl_st_pack(epoch, tile == 0 ? HL_ST_PRE : HL_ST_AGG, tc));
  const uint32_t ex = tile > 0 ? hl_block_lookback(ws.rstat, tile, epoch, err) : 0u;
  if (tid == 0 && tile > 0) hl_st_store(ws.rstat + tile, hl_st_pack(epoch, HL_ST_PRE, ex + tc));
  uint32_t run = ex + before;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint64_t i = tb + w * 256 + k * 64 + lane;
    const uint64_t m = __ballot(first[k]);
    if (first[k]) {
      const uint32_t u = run + (uint32_t)__popcll(m & lt);
      ws.uidx[slot[k]] = u;
      if (!fused) ws.fst[u] = g[k];
      else if (u < (uint32_t)cap) cold_ids[u] = g[k];
    }
    run += (uint32_t)__popcll(m);
    if (i == (uint64_t)n_lookups - 1) {
      ws.ctr[CG_C_NCOLD] = run;
      *n_cold_dev = (int32_t)run;
    }
  }
}

// Insert block b's listed cold lookups point their codes at their staging
// rows and free their table slots; cold_ids[u] = id of staging row u.  When
// the rows do not fit: only the capacity bit and the slot clearing.
__global__ void __launch_bounds__(256)
cg_codes(const int32_t* __restrict__ bag_ptr, int32_t bpb, uint64_t* table, cg_ws ws, int32_t cap, uint32_t k_cap,
         int32_t* __restrict__ codes, uint32_t* __restrict__ cold_ids, uint32_t* err) {
  const uint32_t ncold = ws.ctr[CG_C_NCOLD];
  const bool fits = ncold <= (uint32_t)cap;
  if (blockIdx.x == 0 && threadIdx.x == 0 && !fits) hl_flag(err, HL_DEVERR_CAPACITY);
  const uint32_t cnt = ws.bcnt[blockIdx.x];
  const int32_t lo = bag_ptr[(int64_t)blockIdx.x * bpb];
  for (uint32_t e = threadIdx.x; e < cnt; e += 256) {
    const uint32_t i = ws.blist[lo + e];
    const uint32_t sl = ws.slotof[i];
    if (sl >= ws.S) continue;
    if (fits) codes[i] = (int32_t)(k_cap + ws.uidx[sl]);
    table[sl] = 0;
  }
  if (!fits) return;
  const uint32_t gs = gridDim.x * blockDim.x;
  for (uint32_t u = blockIdx.x * blockDim.x + threadIdx.x; u < ncold; u += gs) cold_ids[u] = ws.fst[u];
}

// Row copy between host table and staging rows: TO_HOST = 0 copies
// staging[u] = host[ids[u]], TO_HOST = 1 copies host[ids[u]] = staging[u], for
// u < *n_dev.  A count above cap copies nothing and sets the capacity bit; an
// id >= n_rows is skipped and sets the range bit.  Each thread keeps 4 units in
// flight.  64 blocks already hold enough reads in flight to fill the host link
// (measured: fewer blocks lose bandwidth, more gain none); more blocks only fill
// the shared memory pipeline with slow host reads, which then stall the HBM
// traffic of kernels running beside the copy on other streams (a concurrent
// streaming kernel ran 5.5x slower beside 512 copy blocks, 1.5x beside 64).
template <typename V, bool TO_HOST>
__global__ void __launch_bounds__(256)
cg_copy(const uint32_t* __restrict__ ids, const int32_t* n_dev, int32_t cap, uint64_t n_rows, V* host, V* stg,
        uint32_t upr, uint32_t* err, hl_hook hk) {
  // a handover: block 0 signals as the copy starts (the copy before it on the
  // stream is complete), and every block waits for its inputs first
  hl_hook_head(hk);
  hl_hook_gate(hk);
  if (hk.gate) __syncthreads();
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
  g = g < 1 ? 1 : (g > 64 ? 64 : g);
  const hl_hook hk = to_host ? hl_hook{} : hl_hook_take(h);  // (the fetch carries the pipeline's handover)
#define CG_COPY(V)                                                                                             \
  if (to_host)                                                                                                 \
    HL_KERNEL(h, s, "cg_scatter", (cg_copy<V, true>), dim3(g), dim3(256), 0, s, ids, n_dev, cap, h->n_rows,     \
              (V*)host, (V*)stg, (uint32_t)(rb / sizeof(V)), h->d_err, hl_hook{});                             \
  else                                                                                                         \
    HL_KERNEL(h, s, "cg_fetch", (cg_copy<V, false>), dim3(g), dim3(256), 0, s, ids, n_dev, cap, h->n_rows,      \
              (V*)host, (V*)stg, (uint32_t)(rb / sizeof(V)), h->d_err, hk);
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
  if ((int64_t)n_samples * bps >= (1ll << 31)) return HL_ERR_UNSUPPORTED;
  const int64_t n_bags = (int64_t)n_samples * bps;
  if (ws_bytes < hl_cold_ws_bytes(h, n_lookups, n_bags, n_samples)) return HL_ERR_CAPACITY;
  hl_ws_note(h, workspace, HL_WSK_OTHER);
  hipStream_t s = (hipStream_t)stream;
  hl_carver c = hl_carver::after_header(workspace, ws_bytes);
  cg_ws ws;
  cg_carve(c, ws, (uint32_t)n_lookups, n_bags, n_samples);
  uint64_t* table = nullptr;
  hl_status st = cg_table(h, ws.S, s, &table);
  if (st != HL_OK) return st;
  const uint32_t n = (uint32_t)n_lookups;
  // selection: every sample (no list) or the listed ones (a mask over samples);
  // an empty selection inserts nothing
  const uint8_t* mask = nullptr;
  if (sample_ids) {
    uint32_t gb = hl_div_up(n_samples > 0 ? n_samples : 1, 256);
    if (gb > 4096) gb = 4096;
    HL_KERNEL(h, s, "cg_mask", cg_mask, dim3(gb), dim3(256), 0, s, ws.mask, n_samples, sample_ids, n_sel_dev,
              n_sel_max, 0, h->d_err);
    HL_KERNEL(h, s, "cg_mask", cg_mask, dim3(gb), dim3(256), 0, s, ws.mask, n_samples, sample_ids, n_sel_dev,
              n_sel_max, 1, h->d_err);
    mask = ws.mask;
  }
  // without a list the first n_sel_max samples are selected: their bags come first
  const int64_t sel_bags = sample_ids ? n_bags : (int64_t)n_sel_max * bps;
  // bags per insert block: about 2048 lookups, CG_BAGS_MIN to CG_BAGS bags
  int32_t bpb = CG_BAGS;
  while (bpb > CG_BAGS_MIN && (int64_t)bpb * n > 2048 * n_bags) bpb >>= 1;
  const uint32_t ib = sel_bags > 0 ? hl_div_up((uint64_t)sel_bags, bpb) : 0;
  if (ib > 0)
    HL_KERNEL(h, s, "cg_insert", cg_insert, dim3(ib), dim3(256), 0, s, gids, codes, bag_ptr, sel_bags, bps, bpb, mask,
              n, h->n_rows, table, ws, h->d_err);
  // the insert kernel cleared the status words, so one fixed tag serves every
  // call (and every replay of a captured graph)
  const uint32_t epoch = 1;
  HL_KERNEL(h, s, "cg_rank", cg_rank, dim3(ws.rtiles), dim3(CG_RT_THREADS), 0, s, gids, codes, ib > 0 ? n : 0u, table, ws,
            n_cold_dev, epoch, nullptr, 0, 0, h->d_err);
  if (ib > 0)
    HL_KERNEL(h, s, "cg_codes", cg_codes, dim3(ib), dim3(256), 0, s, bag_ptr, bpb, table, ws, cap, h->k_cap, codes,
              cold_ids_out, h->d_err);
  HL_LAUNCHED();
  return HL_OK;
}

// The fused plan's cold state: the cold regions carved after the grouping's
// region of the workspace.
static hl_carver cg_fused_carver(const hl_handle* h, void* workspace, size_t ws_bytes, int64_t n_lookups,
                                 int64_t n_bags) {
  hl_carver c = hl_carver::after_header(workspace, ws_bytes);
  c.off = hl_bwd_ws_bytes(h, n_lookups, n_bags);
  return c;
}

size_t hl_plan_ws_bytes(const hl_handle* h, int64_t max_lookups, int64_t max_bags, int32_t max_samples) {
  hl_carver c = cg_fused_carver(h, nullptr, 0, max_lookups, max_bags);
  cg_ws ws;
  cg_carve(c, ws, (uint32_t)max_lookups, max_bags, max_samples);
  return c.off;
}

hl_status hl_cold_fused_begin(hl_handle* h, int64_t n_lookups, int64_t n_bags, int32_t n_samples, int32_t cap,
                              void* workspace, size_t ws_bytes, hipStream_t s, hl_cg_fused* out) {
  *out = hl_cg_fused{};
  if (!h || !workspace || n_lookups <= 0 || n_bags <= 0 || n_samples <= 0 || cap < 0) return HL_ERR_INVALID_ARG;
  if (n_lookups >= (1ll << 30) || (uint64_t)h->k_cap + (uint64_t)cap >= (1ull << 31)) return HL_ERR_UNSUPPORTED;
  if (ws_bytes < hl_plan_ws_bytes(h, n_lookups, n_bags, n_samples)) return HL_ERR_CAPACITY;
  hl_carver c = cg_fused_carver(h, workspace, ws_bytes, n_lookups, n_bags);
  cg_ws ws;
  cg_carve(c, ws, (uint32_t)n_lookups, n_bags, n_samples);
  // no growth here: a larger table is allocated by a plain cold plan, after
  // its waits (the table is shared with the steps still in flight)
  if (h->cg_slots < ws.S || !h->cg_table) return HL_ERR_CAPACITY;
  (void)s;
  out->table = h->cg_table;
  out->S = ws.S;
  out->slotof = ws.slotof;
  out->uidx = ws.uidx;
  out->rstat = ws.rstat;
  out->rtiles = ws.rtiles;
  out->ncold = ws.ctr + CG_C_NCOLD;
  out->cap = cap;
  return HL_OK;
}

hl_status hl_cold_rank_fused(hl_handle* h, const uint32_t* gids, const int32_t* codes, int64_t n_lookups,
                             uint32_t* cold_ids, int32_t* n_cold_dev, void* workspace, const hl_cg_fused& cf,
                             hipStream_t s) {
  if (!h || !gids || !codes || !n_cold_dev || !workspace || !cf.table || n_lookups <= 0) return HL_ERR_INVALID_ARG;
  if (cf.cap > 0 && !cold_ids) return HL_ERR_INVALID_ARG;
  cg_ws ws{};
  ws.ctr = reinterpret_cast<uint32_t*>(workspace) + HL_HDR_COLD;
  ws.S = cf.S;
  ws.uidx = cf.uidx;
  ws.slotof = cf.slotof;
  ws.rstat = cf.rstat;
  ws.rtiles = cf.rtiles;
  // the dispatch kernel cleared the status words
  const uint32_t epoch = 1;
  HL_KERNEL(h, s, "cg_rank", cg_rank, dim3(cf.rtiles), dim3(CG_RT_THREADS), 0, s, gids, codes, (uint32_t)n_lookups,
            cf.table, ws, n_cold_dev, epoch, cold_ids, cf.cap, 1, h->d_err);
  HL_LAUNCHED();
  return HL_OK;
}

extern "C" hl_status hl_cold_reserve(hl_handle* h, int64_t max_lookups, hl_stream stream) {
  if (!h || max_lookups < 0) return HL_ERR_INVALID_ARG;
  if (max_lookups >= (1ll << 30)) return HL_ERR_UNSUPPORTED;
  uint64_t* t = nullptr;
  return cg_table(h, cg_table_slots((uint32_t)max_lookups), (hipStream_t)stream, &t);
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
