// Stable LSD radix sort of (key, value) uint32 pairs.
//
// A sort of `bits` bits takes P = ceil(bits / 11) passes of b = ceil(bits / P)
// bits (two passes of 10 bits for the backward's 20-bit keys).  One histogram
// kernel counts every digit position in a single read of the keys (per-block
// counts) and clears the first pass's look-back status.  Then one kernel per
// digit: a block takes the next tile (dynamic tile ids, so every lower tile is
// already running), ranks its items by digit with per-wave LDS counters (the
// counters' totals are the tile's digit counts), publishes the counts, obtains
// those of all earlier tiles by decoupled look-back, reorders the tile in LDS
// so that each digit's run is contiguous and writes it out.  Only tile 0 adds
// up the histogram: its published prefix starts from each digit's global
// offset, so the look-back hands the offsets to every later tile.  Each pass block also
// clears its tile's status words for the next pass.  Item order inside a tile
// is wave-major, then item, then lane, which is index order, so the sort is
// stable.
#include "hl_internal.h"

void hl_sort_ws_carve(hl_carver& c, hl_sort_ws& ws, uint32_t n_max) {
  ws.n_max = n_max;
  ws.tiles_max = n_max ? hl_div_up(n_max, HL_SORT_TILE) : 1;
  ws.k0 = c.take<uint32_t>(n_max);
  ws.v0 = c.take<uint32_t>(n_max);
  ws.k1 = c.take<uint32_t>(n_max);
  ws.v1 = c.take<uint32_t>(n_max);
  ws.part = c.take<uint32_t>((size_t)HL_SORT_MAXPASS * HL_SORT_HIST_BLOCKS * HL_SORT_MAXNB);
  ws.st[0] = c.take<uint32_t>((size_t)ws.tiles_max * HL_SORT_MAXNB);
  ws.st[1] = c.take<uint32_t>((size_t)ws.tiles_max * HL_SORT_MAXNB);
  ws.ctr = c.base ? c.header() + HL_HDR_SORT : nullptr;
}

// Status word of (tile, digit): flag in the top two bits (0 = not yet
// published), count below.  Relaxed agent-scope atomics: the word carries its
// own value and no other data is published through it.
#define SRT_AGG 0x40000000u
#define SRT_PRE 0x80000000u
#define SRT_VAL 0x3FFFFFFFu
__device__ __forceinline__ void srt_st_store(uint32_t* p, uint32_t w) {
  __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t srt_st_load(const uint32_t* p) {
  return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint32_t srt_n(const uint32_t* n_dev, uint32_t n_host) {
  if (!n_dev) return n_host;
  const uint32_t v = *n_dev;
  return v < n_host ? v : n_host;
}

struct srt_plan {
  int passes, b, nb;
};
static srt_plan srt_make_plan(int bits) {
  if (bits < 1) bits = 1;
  srt_plan p;
  p.passes = (bits + 10) / 11;
  p.b = (bits + p.passes - 1) / p.passes;
  p.nb = p.b <= 8 ? 256 : (p.b <= 10 ? 1024 : 2048);
  return p;
}

// Per-block counts of every digit of every pass; clears n_zero status words.
template <int NB>
__global__ void __launch_bounds__(HL_SORT_HIST_THREADS)
srt_hist(const uint32_t* __restrict__ keys, const uint32_t* n_dev, uint32_t n_host, int passes, int b,
         uint32_t* __restrict__ part, uint32_t* __restrict__ zero, uint64_t n_zero) {
  __shared__ uint32_t h[HL_SORT_MAXPASS][NB];
  const uint32_t n = srt_n(n_dev, n_host);
  const uint32_t gs = gridDim.x * blockDim.x;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_zero; i += gs) zero[i] = 0;
  for (int j = threadIdx.x; j < HL_SORT_MAXPASS * NB; j += blockDim.x) (&h[0][0])[j] = 0;
  __syncthreads();
  const uint32_t mask = (1u << b) - 1u;
  for (uint32_t i0 = blockIdx.x * blockDim.x + threadIdx.x; i0 < n; i0 += 8 * gs) {
    uint32_t k[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) k[u] = i0 + u * gs < n ? keys[i0 + u * gs] : 0u;
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (i0 + u * gs < n)
        for (int p = 0; p < passes; ++p) atomicAdd(&h[p][(k[u] >> (b * p)) & mask], 1u);
  }
  __syncthreads();
  for (int p = 0; p < passes; ++p)
    for (int j = threadIdx.x; j < NB; j += blockDim.x)
      part[((size_t)p * HL_SORT_HIST_BLOCKS + blockIdx.x) * NB + j] = h[p][j];
}

// Block-wide exclusive scans of two values per digit (each thread owns PER
// consecutive digits).  Returns through a and c in place.
template <int NB, int PER>
__device__ __forceinline__ void srt_scan2(uint32_t (&a)[PER], uint32_t (&c)[PER], uint32_t (*ws)[2]) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  uint32_t sa = 0, sc = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    sa += a[j];
    sc += c[j];
  }
  uint32_t ia = sa, ic = sc;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t ta = __shfl_up(ia, o), tc = __shfl_up(ic, o);
    if (lane >= o) {
      ia += ta;
      ic += tc;
    }
  }
  if (lane == 63) {
    ws[w][0] = ia;
    ws[w][1] = ic;
  }
  __syncthreads();
  uint32_t ra = ia - sa, rc = ic - sc;
  for (int j = 0; j < w; ++j) {
    ra += ws[j][0];
    rc += ws[j][1];
  }
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const uint32_t ta = a[j], tc = c[j];
    a[j] = ra;
    c[j] = rc;
    ra += ta;
    rc += tc;
  }
}

template <int NB>
__global__ void __launch_bounds__(HL_SORT_THREADS)
srt_pass(const uint32_t* __restrict__ kin, const uint32_t* __restrict__ vin, uint32_t* __restrict__ kout,
         uint32_t* __restrict__ vout, const uint32_t* n_dev, uint32_t n_host, int shift, int b,
         const uint32_t* __restrict__ part, uint32_t n_part, uint32_t* st, uint32_t* st_next, uint32_t* tile_ctr,
         uint32_t* err, hl_hook hk) {
  constexpr int PER = NB >= HL_SORT_THREADS ? NB / HL_SORT_THREADS : 1;
  constexpr int OWNERS = NB / PER;         // threads that own digits
  // look-back window per digit; every predecessor read costs a load per digit
  // (NB x tiles^2 / 2 loads when no inclusive prefix is found early), so the
  // window stays short and the walk stops at the first inclusive prefix
  constexpr int WIN = PER >= 4 ? 8 : 16;
  constexpr int WIN0 = 4;
  __shared__ uint32_t s_tile;
  __shared__ uint32_t wcnt[HL_SORT_WAVES][NB];
  __shared__ uint32_t tdex[NB], gbase[NB];
  __shared__ uint32_t scan_ws[HL_SORT_WAVES][2];
  __shared__ uint32_t lk[HL_SORT_TILE], lv[HL_SORT_TILE];
  const uint32_t n = srt_n(n_dev, n_host);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  hl_hook_head(hk);
  if (tid == 0) s_tile = atomicInc(tile_ctr, gridDim.x - 1);
  for (int j = tid; j < HL_SORT_WAVES * NB; j += HL_SORT_THREADS) (&wcnt[0][0])[j] = 0;
  __syncthreads();
  const uint32_t tile = s_tile;
  if (st_next)  // this tile's status words of the next pass
    for (int j = tid; j < NB; j += HL_SORT_THREADS) st_next[(size_t)tile * NB + j] = 0;
  const uint64_t tb = (uint64_t)tile * HL_SORT_TILE;
  if (tb >= n) return;
  const uint32_t mask = (1u << b) - 1u;
  uint32_t key[HL_SORT_ITEMS], val[HL_SORT_ITEMS];
#pragma unroll
  for (int k = 0; k < HL_SORT_ITEMS; ++k) {
    const uint64_t idx = tb + (uint64_t)w * (HL_SORT_ITEMS * 64) + k * 64 + lane;
    const bool ok = idx < n;
    key[k] = ok ? kin[idx] : 0xFFFFFFFFu;
    val[k] = ok ? vin[idx] : 0u;
  }
  // global counts of the owned digits (loads issued together), read by tile 0
  // only: its published prefix carries the digits' global offsets, so every
  // later tile obtains them through the look-back
  const int d0 = tid * PER;
  const bool owner = tid < OWNERS;
  uint32_t dtot[PER];
  {
    const uint32_t np = tile == 0 ? n_part : 0u;
    uint32_t pv[PER][HL_SORT_HIST_BLOCKS];
#pragma unroll
    for (int j = 0; j < PER; ++j)
#pragma unroll
      for (int q = 0; q < HL_SORT_HIST_BLOCKS; ++q)
        pv[j][q] = (owner && (uint32_t)q < np) ? part[(size_t)q * NB + d0 + j] : 0u;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      dtot[j] = 0;
#pragma unroll
      for (int q = 0; q < HL_SORT_HIST_BLOCKS; ++q) dtot[j] += pv[j][q];
    }
  }
  // ranking: every item adds 1 to its digit's counter of the wave; the old
  // value is its rank among the wave's earlier items of that digit.  One
  // wave's LDS atomics are applied in instruction order, and the lanes of one
  // instruction that hit the same counter in lane order (a property of the LDS
  // unit, checked on this GPU over 49M random lane patterns with partial masks,
  // none out of order), so ranks follow (item, lane) order: the sort is stable.
  uint32_t dg[HL_SORT_ITEMS], lr[HL_SORT_ITEMS];
#pragma unroll
  for (int k = 0; k < HL_SORT_ITEMS; ++k) {
    const uint64_t idx = tb + (uint64_t)w * (HL_SORT_ITEMS * 64) + k * 64 + lane;
    dg[k] = (key[k] >> shift) & mask;
    lr[k] = idx < n ? atomicAdd(&wcnt[w][dg[k]], 1u) : 0u;
  }
  __syncthreads();
  // wave-exclusive offsets of each owned digit; the totals are the tile's counts
  uint32_t tc[PER], tx[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    uint32_t run = 0;
    if (owner)
#pragma unroll
      for (int q = 0; q < HL_SORT_WAVES; ++q) {
        const uint32_t c = wcnt[q][d0 + j];
        wcnt[q][d0 + j] = run;
        run += c;
      }
    tc[j] = run;
    tx[j] = run;
    if (owner && tile > 0) srt_st_store(st + (size_t)tile * NB + d0 + j, SRT_AGG | run);
  }
  uint32_t gx[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) gx[j] = dtot[j];
  srt_scan2<NB, PER>(tx, gx, scan_ws);
  // tile 0: inclusive prefix = the digit's global offset + its own count
  if (owner && tile == 0)
#pragma unroll
    for (int j = 0; j < PER; ++j) srt_st_store(st + d0 + j, SRT_PRE | (gx[j] + tc[j]));
  // decoupled look-back: counts of this digit in all earlier tiles
  uint32_t excl[PER];
  int64_t jj[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    excl[j] = 0;
    jj[j] = owner ? (int64_t)tile - 1 : -1;
  }
  uint32_t spins = 0;
  // the first window is short: the nearest tiles have most likely published
  // their inclusive prefix by then, and each word read costs bandwidth
  int win = WIN0;
  while (true) {
    uint32_t wv[PER][WIN];
#pragma unroll
    for (int j = 0; j < PER; ++j)
#pragma unroll
      for (int q = 0; q < WIN; ++q)
        wv[j][q] = q < win && jj[j] - q >= 0 ? srt_st_load(st + (size_t)(jj[j] - q) * NB + d0 + j) : SRT_PRE;
    bool any = false, stall = false;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      if (jj[j] < 0) continue;
      int used = 0;
      bool stop = false;
#pragma unroll
      for (int q = 0; q < WIN; ++q) {
        if (stop) continue;
        if (q >= win) {  // beyond this round's window
          stop = true;
          continue;
        }
        const uint32_t x = wv[j][q];
        if ((x & (SRT_AGG | SRT_PRE)) == 0) {  // not yet published
          stop = true;
          stall = true;
          continue;
        }
        if (jj[j] - q >= 0) excl[j] += x & SRT_VAL;
        if (x & SRT_PRE) {
          used = -1;
          stop = true;
          continue;
        }
        used = q + 1;
      }
      jj[j] = used < 0 ? -1 : jj[j] - used;
      any |= jj[j] >= 0;
    }
    if (!any) break;
    win = WIN;
    if (stall) {
      if (++spins > HL_SPIN_LIMIT) {
        hl_flag(err, HL_DEVERR_STALL);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  if (owner) {
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      if (tile > 0) srt_st_store(st + (size_t)tile * NB + d0 + j, SRT_PRE | (excl[j] + tc[j]));
      tdex[d0 + j] = tx[j];
      gbase[d0 + j] = tile == 0 ? gx[j] : excl[j];
    }
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < HL_SORT_ITEMS; ++k) {
    const uint64_t idx = tb + (uint64_t)w * (HL_SORT_ITEMS * 64) + k * 64 + lane;
    if (idx < n) {
      const uint32_t p = tdex[dg[k]] + wcnt[w][dg[k]] + lr[k];
      lk[p] = key[k];
      lv[p] = val[k];
    }
  }
  __syncthreads();
  const uint32_t nv = (uint32_t)min((uint64_t)HL_SORT_TILE, (uint64_t)n - tb);
#pragma unroll 4
  for (uint32_t i = tid; i < nv; i += HL_SORT_THREADS) {
    const uint32_t kk = lk[i];
    const uint32_t d = (kk >> shift) & mask;
    const uint32_t p = gbase[d] + (i - tdex[d]);
    kout[p] = kk;
    vout[p] = lv[i];
  }
}

void hl_sort_result(const hl_sort_ws& ws, int bits, uint32_t** out_k, uint32_t** out_v) {
  const bool odd = srt_make_plan(bits).passes & 1;
  *out_k = odd ? ws.k1 : ws.k0;
  *out_v = odd ? ws.v1 : ws.v0;
}

hl_sort_geom hl_sort_geometry(uint32_t n_host, int bits) {
  const srt_plan pl = srt_make_plan(bits);
  hl_sort_geom g;
  g.passes = pl.passes;
  g.b = pl.b;
  g.nb = pl.nb;
  const uint32_t hb = hl_div_up(n_host, HL_SORT_HIST_THREADS * 8);
  g.hist_blocks = hb < 1 ? 1 : (hb > HL_SORT_HIST_BLOCKS ? HL_SORT_HIST_BLOCKS : hb);
  g.n_zero = (uint64_t)hl_div_up(n_host, HL_SORT_TILE) * pl.nb;
  return g;
}

template <int NB>
static hl_status srt_hist_launch(hl_handle* h, hl_sort_ws& ws, const uint32_t* n_dev, uint32_t n_host, int bits,
                                 hipStream_t s) {
  const hl_sort_geom g = hl_sort_geometry(n_host, bits);
  HL_KERNEL(h, s, "srt_hist", srt_hist<NB>, dim3(g.hist_blocks), dim3(HL_SORT_HIST_THREADS), 0, s, ws.k0, n_dev,
            n_host, g.passes, g.b, ws.part, ws.st[0], g.n_zero);
  HL_LAUNCHED();
  return HL_OK;
}

template <int NB>
static hl_status srt_launch(hl_handle* h, hl_sort_ws& ws, const uint32_t* n_dev, uint32_t n_host, int bits,
                            hipStream_t s) {
  const uint32_t tiles = hl_div_up(n_host, HL_SORT_TILE);
  const hl_sort_geom g = hl_sort_geometry(n_host, bits);
  uint32_t *ki = ws.k0, *vi = ws.v0, *ko = ws.k1, *vo = ws.v1;
  for (int p = 0; p < g.passes; ++p) {
    HL_KERNEL(h, s, "srt_pass", srt_pass<NB>, dim3(tiles), dim3(HL_SORT_THREADS), 0, s, ki, vi, ko, vo, n_dev,
              n_host, g.b * p, g.b, ws.part + (size_t)p * HL_SORT_HIST_BLOCKS * NB, g.hist_blocks, ws.st[p & 1],
              p + 1 < g.passes ? ws.st[(p + 1) & 1] : nullptr, ws.ctr + 1 + p, h->d_err,
              p == 0 ? hl_hook_take(h) : hl_hook{});
    uint32_t* t = ki;
    ki = ko;
    ko = t;
    t = vi;
    vi = vo;
    vo = t;
  }
  HL_LAUNCHED();
  return HL_OK;
}

static hl_status srt_check(const hl_sort_ws& ws, uint32_t n_host, int bits) {
  if (n_host > ws.n_max || n_host >= (1u << 30)) return HL_ERR_CAPACITY;
  if (bits > 32) return HL_ERR_UNSUPPORTED;
  return HL_OK;
}

hl_status hl_sort_passes(hl_handle* h, hl_sort_ws& ws, const uint32_t* n_dev, uint32_t n_host, int bits,
                         hipStream_t s, uint32_t** out_k, uint32_t** out_v) {
  *out_k = ws.k0;
  *out_v = ws.v0;
  if (n_host == 0) return HL_OK;
  hl_status st = srt_check(ws, n_host, bits);
  if (st != HL_OK) return st;
  const srt_plan pl = srt_make_plan(bits);
  if (pl.nb == 256) st = srt_launch<256>(h, ws, n_dev, n_host, bits, s);
  else if (pl.nb == 1024) st = srt_launch<1024>(h, ws, n_dev, n_host, bits, s);
  else st = srt_launch<2048>(h, ws, n_dev, n_host, bits, s);
  if (st != HL_OK) return st;
  hl_sort_result(ws, bits, out_k, out_v);
  return HL_OK;
}

hl_status hl_sort_pairs(hl_handle* h, hl_sort_ws& ws, const uint32_t* n_dev, uint32_t n_host, int bits,
                        hipStream_t s, uint32_t** out_k, uint32_t** out_v) {
  *out_k = ws.k0;
  *out_v = ws.v0;
  if (n_host == 0) return HL_OK;
  hl_status st = srt_check(ws, n_host, bits);
  if (st != HL_OK) return st;
  const srt_plan pl = srt_make_plan(bits);
  if (pl.nb == 256) st = srt_hist_launch<256>(h, ws, n_dev, n_host, bits, s);
  else if (pl.nb == 1024) st = srt_hist_launch<1024>(h, ws, n_dev, n_host, bits, s);
  else st = srt_hist_launch<2048>(h, ws, n_dev, n_host, bits, s);
  if (st != HL_OK) return st;
  return hl_sort_passes(h, ws, n_dev, n_host, bits, s, out_k, out_v);
}
