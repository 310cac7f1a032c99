// Stable LSD radix sort of (key, value) uint32 pairs, 8-bit digits.
//
// One histogram kernel counts all digit positions in a single read of the keys
// (per-block counts; each pass block adds up the few it needs).  Then one
// kernel per digit: a block takes the next tile (dynamic tile ids, so every
// lower tile is already running), counts its digits and publishes them at
// once, ranks its items by digit with wave ballots, and obtains the counts of
// all earlier tiles by decoupled look-back over epoch-tagged status words (no
// clearing between calls beyond the histogram kernel's reset).  Items are
// reordered in LDS so the global writes of each digit run are contiguous.
// Item order inside a tile is wave-major, then item, then lane, which is index
// order, so the sort is stable.  Tiles are large (8192 items) so that every
// tile finds all its predecessors within one look-back window.
#include "hl_internal.h"

void hl_sort_ws_carve(hl_carver& c, hl_sort_ws& ws, uint32_t n_max) {
  ws.n_max = n_max;
  ws.tiles_max = n_max ? hl_div_up(n_max, HL_SORT_TILE) : 1;
  ws.k0 = c.take<uint32_t>(n_max);
  ws.v0 = c.take<uint32_t>(n_max);
  ws.k1 = c.take<uint32_t>(n_max);
  ws.v1 = c.take<uint32_t>(n_max);
  ws.part = c.take<uint32_t>((size_t)HL_SORT_HIST_BLOCKS * 1024);
  ws.gexcl = c.take<uint32_t>(1024);
  ws.ctr = c.base ? c.header() + HL_HDR_SORT : nullptr;
  ws.status = c.take<uint64_t>((size_t)4 * ws.tiles_max * 256);
}

__device__ __forceinline__ uint32_t srt_n(const uint32_t* n_dev, uint32_t n_host) {
  if (!n_dev) return n_host;
  const uint32_t v = *n_dev;
  return v < n_host ? v : n_host;
}

// Per-block digit counts of every pass, and a reset of the pass kernels'
// status words (n_status of them).
__global__ void __launch_bounds__(HL_SORT_HIST_THREADS)
srt_hist(const uint32_t* __restrict__ keys, const uint32_t* n_dev, uint32_t n_host, int passes,
         uint32_t* part, uint64_t* status, uint64_t n_status) {
  __shared__ uint32_t h[4][256];
  const uint32_t n = srt_n(n_dev, n_host);
  const uint32_t gs = gridDim.x * blockDim.x;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_status; i += gs) status[i] = 0;
  for (int j = threadIdx.x; j < 1024; j += blockDim.x) (&h[0][0])[j] = 0;
  __syncthreads();
  for (uint32_t b = blockIdx.x * blockDim.x + threadIdx.x; b < n; b += 8 * gs) {
    uint32_t k[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) k[u] = b + u * gs < n ? keys[b + u * gs] : 0u;
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (b + u * gs < n)
        for (int p = 0; p < passes; ++p) atomicAdd(&h[p][(k[u] >> (8 * p)) & 255u], 1u);
  }
  __syncthreads();
  for (int j = threadIdx.x; j < passes * 256; j += blockDim.x) part[blockIdx.x * 1024 + j] = (&h[0][0])[j];
}

__global__ void __launch_bounds__(HL_SORT_BLOCK)
srt_pass(const uint32_t* __restrict__ kin, const uint32_t* __restrict__ vin, uint32_t* __restrict__ kout,
         uint32_t* __restrict__ vout, const uint32_t* n_dev, uint32_t n_host, int shift,
         const uint32_t* __restrict__ part, uint32_t n_part, uint64_t* status, uint32_t* tile_ctr,
         uint32_t epoch, uint32_t* err) {
  __shared__ uint32_t s_tile;
  __shared__ uint32_t wcnt[HL_SORT_WAVES][256];
  __shared__ uint32_t thist[256], tdex[256], gbase[256], wt[4], wg[4];
  __shared__ uint32_t lk[HL_SORT_TILE], lv[HL_SORT_TILE];
  const uint32_t n = srt_n(n_dev, n_host);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  if (tid == 0) s_tile = atomicInc(tile_ctr, gridDim.x - 1);
  for (int j = tid; j < HL_SORT_WAVES * 256; j += HL_SORT_BLOCK) (&wcnt[0][0])[j] = 0;
  if (tid < 256) thist[tid] = 0;
  __syncthreads();
  const uint32_t tile = s_tile;
  const uint64_t tb = (uint64_t)tile * HL_SORT_TILE;
  if (tb >= n) return;
  uint32_t key[HL_SORT_ITEMS], val[HL_SORT_ITEMS], lr[HL_SORT_ITEMS];
#pragma unroll
  for (int k = 0; k < HL_SORT_ITEMS; ++k) {
    const uint64_t idx = tb + (uint64_t)w * (HL_SORT_ITEMS * 64) + k * 64 + lane;
    const bool ok = idx < n;
    key[k] = ok ? kin[idx] : 0xFFFFFFFFu;
    val[k] = ok ? vin[idx] : 0u;
  }
  // global count of digit tid over the histogram blocks (loads issued together)
  uint32_t dtot = 0;
  if (tid < 256) {
    uint32_t pv[HL_SORT_HIST_BLOCKS];
#pragma unroll
    for (int b = 0; b < HL_SORT_HIST_BLOCKS; ++b) pv[b] = (uint32_t)b < n_part ? part[b * 1024 + tid] : 0u;
#pragma unroll
    for (int b = 0; b < HL_SORT_HIST_BLOCKS; ++b) dtot += pv[b];
  }
  // tile digit counts first, published before the ranking so that later tiles
  // find them when they look back
#pragma unroll
  for (int k = 0; k < HL_SORT_ITEMS; ++k) {
    const uint64_t idx = tb + (uint64_t)w * (HL_SORT_ITEMS * 64) + k * 64 + lane;
    if (idx < n) atomicAdd(&thist[(key[k] >> shift) & 255u], 1u);
  }
  __syncthreads();
  uint64_t* st = status + (tid & 255);
  uint32_t tc = 0;
  if (tid < 256) {
    tc = thist[tid];
    hl_st_store(st + (size_t)tile * 256, hl_st_pack(epoch, tile == 0 ? HL_ST_PRE : HL_ST_AGG, tc));
  }
  const uint64_t lt = (1ull << lane) - 1ull;
#pragma unroll
  for (int k = 0; k < HL_SORT_ITEMS; ++k) {
    const uint64_t idx = tb + (uint64_t)w * (HL_SORT_ITEMS * 64) + k * 64 + lane;
    const bool ok = idx < n;
    const uint32_t d = (key[k] >> shift) & 255u;
    uint64_t peers = __ballot(ok);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const bool bit = (d >> b) & 1u;
      const uint64_t m = __ballot(bit);
      peers &= bit ? m : ~m;
    }
    const int leader = peers ? (__ffsll((unsigned long long)peers) - 1) : 0;
    uint32_t old = 0;
    if (ok && lane == leader) {
      old = wcnt[w][d];
      wcnt[w][d] = old + (uint32_t)__popcll(peers);
    }
    old = __shfl(old, leader);
    lr[k] = old + (uint32_t)__popcll(peers & lt);
  }
  __syncthreads();
  if (tid < 256) {
    // wave-exclusive prefixes of this digit
    uint32_t run = 0;
#pragma unroll
    for (int j = 0; j < HL_SORT_WAVES; ++j) {
      const uint32_t c = wcnt[j][tid];
      wcnt[j][tid] = run;
      run += c;
    }
    // tile-local and global exclusive scans over the digits (waves 0..3)
    uint32_t inc = tc, ginc = dtot;
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t t1 = __shfl_up(inc, o), t2 = __shfl_up(ginc, o);
      if (lane >= o) {
        inc += t1;
        ginc += t2;
      }
    }
    if (lane == 63) {
      wt[w] = inc;
      wg[w] = ginc;
    }
    tdex[tid] = inc - tc;
    gbase[tid] = ginc - dtot;
  }
  __syncthreads();
  if (tid < 256) {
    uint32_t pre = 0, gpre = 0;
    for (int j = 0; j < w; ++j) {
      pre += wt[j];
      gpre += wg[j];
    }
    tdex[tid] += pre;
    uint32_t excl = 0;
    if (tile > 0) {
      excl = hl_lookback(st, tile, 256, epoch, err);
      hl_st_store(st + (size_t)tile * 256, hl_st_pack(epoch, HL_ST_PRE, excl + tc));
    }
    gbase[tid] += gpre + excl;
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < HL_SORT_ITEMS; ++k) {
    const uint64_t idx = tb + (uint64_t)w * (HL_SORT_ITEMS * 64) + k * 64 + lane;
    if (idx < n) {
      const uint32_t d = (key[k] >> shift) & 255u;
      const uint32_t p = tdex[d] + wcnt[w][d] + lr[k];
      lk[p] = key[k];
      lv[p] = val[k];
    }
  }
  __syncthreads();
  const uint32_t nv = (uint32_t)min((uint64_t)HL_SORT_TILE, (uint64_t)n - tb);
  for (uint32_t i = tid; i < nv; i += HL_SORT_BLOCK) {
    const uint32_t kk = lk[i];
    const uint32_t d = (kk >> shift) & 255u;
    const uint32_t p = gbase[d] + (i - tdex[d]);
    kout[p] = kk;
    vout[p] = lv[i];
  }
}

hl_status hl_sort_pairs(hl_handle* h, hl_sort_ws& ws, const uint32_t* n_dev, uint32_t n_host, int bits,
                        hipStream_t s, uint32_t** out_k, uint32_t** out_v) {
  *out_k = ws.k0;
  *out_v = ws.v0;
  if (n_host == 0) return HL_OK;
  if (n_host > ws.n_max || n_host >= (1u << 30)) return HL_ERR_CAPACITY;
  if (bits < 1) bits = 1;
  const int passes = (bits + 7) / 8;
  if (passes > 4) return HL_ERR_UNSUPPORTED;
  const uint32_t epoch = hl_next_epoch(h);
  const uint32_t tiles = hl_div_up(n_host, HL_SORT_TILE);
  uint32_t hb = hl_div_up(n_host, HL_SORT_HIST_THREADS * 8);
  hb = hb < 1 ? 1 : (hb > HL_SORT_HIST_BLOCKS ? HL_SORT_HIST_BLOCKS : hb);
  HL_KERNEL(h, s, "srt_hist", srt_hist, dim3(hb), dim3(HL_SORT_HIST_THREADS), 0, s, ws.k0, n_dev, n_host, passes,
            ws.part, ws.status, (uint64_t)4 * ws.tiles_max * 256);
  uint32_t *ki = ws.k0, *vi = ws.v0, *ko = ws.k1, *vo = ws.v1;
  for (int p = 0; p < passes; ++p) {
    HL_KERNEL(h, s, "srt_pass", srt_pass, dim3(tiles), dim3(HL_SORT_BLOCK), 0, s, ki, vi, ko, vo, n_dev, n_host,
              8 * p, ws.part + p * 256, hb, ws.status + (size_t)p * ws.tiles_max * 256, ws.ctr + 1 + p, epoch,
              h->d_err);
    uint32_t* t = ki;
    ki = ko;
    ko = t;
    t = vi;
    vi = vo;
    vo = t;
  }
  HL_LAUNCHED();
  *out_k = ki;
  *out_v = vi;
  return HL_OK;
}
