// Stable LSD radix sort of (key, value) uint32 pairs.
//
// A sort of `bits` bits takes P = ceil(bits / 11) passes of b = ceil(bits / P)
// bits (two passes of 10 bits for the backward's 20-bit keys).  One histogram
// kernel counts every digit position in a single read of the keys (per-block
// counts) and clears the first pass's status words.  Then one kernel per
// digit: a block takes the next tile (dynamic tile ids, so every lower tile is
// already running), ranks its items by digit with per-wave LDS counters that
// the lanes of one digit advance together (their peer mask found by ballots;
// the counters' totals are the tile's digit counts), publishes the counts, adds up
// the counts of all earlier tiles (read together, 64 words in flight per
// thread: at these sizes every tile runs at once, so one round of loads
// replaces a chain of inclusive prefixes), adds each digit's global offset
// (the histogram's exclusive scan, which every tile forms), and writes out the
// tile, which it has reordered in LDS (before reading the earlier tiles'
// counts) so that each digit's run is contiguous.  Each pass
// block also clears its tile's status words for the next pass.  Item order inside a tile
// is wave-major, then item, then lane, which is index order, so the sort is
// stable.
#include "hl_internal.h"

void hl_sort_ws_carve(hl_carver& c, hl_sort_ws& ws, uint32_t n_max) {
  ws.n_max = n_max;
  ws.tiles_max = n_max ? hl_div_up(n_max, HL_SORT_TILE_MIN) : 1;
  ws.k0 = c.take<uint32_t>(n_max);
  ws.v0 = c.take<uint32_t>(n_max);
  ws.k1 = c.take<uint32_t>(n_max);
  ws.v1 = c.take<uint32_t>(n_max);
  ws.part = c.take<uint32_t>((size_t)HL_SORT_MAXPASS * HL_SORT_HIST_BLOCKS * HL_SORT_MAXNB);
  ws.st[0] = c.take<uint32_t>((size_t)ws.tiles_max * HL_SORT_MAXNB);
  ws.st[1] = c.take<uint32_t>((size_t)ws.tiles_max * HL_SORT_MAXNB);
  ws.ctr = c.base ? c.header() + HL_HDR_SORT : nullptr;
}

// Status of (tile, digit): a flag bit (0 = not yet published) over the
// tile's count of the digit.  With one digit per owning thread a 32-bit word
// per digit (SRT_AGG); with two or more, two digits share a word, 16 bits
// each (SRT_AGG2 per half: a tile's count stays below 2^15), so a thread
// reads its digits' counts of a tile in one load.  Relaxed agent-scope
// atomics: a word carries its own value and no other data is published
// through it.
#define SRT_AGG 0x40000000u
#define SRT_VAL 0x3FFFFFFFu
#define SRT_AGG2 0x80008000u
static_assert(HL_SORT_TILE_MAX < 0x8000, "a tile's digit count must fit 15 bits");
__device__ __forceinline__ void srt_st_store(uint32_t* p, uint32_t w) {
  __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t srt_st_load(const uint32_t* p) {
  return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t srt_st_load2(const uint32_t* p) {  // two words (8-byte aligned)
  return __hip_atomic_load(reinterpret_cast<uint64_t*>(const_cast<uint32_t*>(p)), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
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

template <int NB, int ITEMS>
__global__ void __launch_bounds__(HL_SORT_THREADS)
srt_pass(const uint32_t* __restrict__ kin, const uint32_t* __restrict__ vin, uint32_t* __restrict__ kout,
         uint32_t* __restrict__ vout, const uint32_t* n_dev, uint32_t n_host, int shift, int b,
         const uint32_t* __restrict__ part, uint32_t n_part, uint32_t* st, uint32_t* st_next, uint32_t* tile_ctr,
         uint32_t* err, hl_hook hk) {
  constexpr uint32_t TILE = HL_SORT_THREADS * ITEMS;
  constexpr int PER = NB >= HL_SORT_THREADS ? NB / HL_SORT_THREADS : 1;
  constexpr int OWNERS = NB / PER;         // threads that own digits
  // status words of a tile per digit owner, and the earlier tiles whose
  // counts one round reads (48 words in flight per thread)
  constexpr int PW = PER >= 2 ? PER / 2 : 1;
  constexpr int CHUNK = 48 / PW;
  constexpr size_t TW = PER >= 2 ? NB / 2 : NB;  // words per tile
  __shared__ uint32_t s_tile;
  __shared__ uint32_t wcnt[HL_SORT_WAVES][NB];
  __shared__ uint32_t tdex[NB], gbase[NB];
  __shared__ uint32_t scan_ws[HL_SORT_WAVES][2];
  __shared__ uint32_t lk[TILE], lv[TILE];
  const uint32_t n = srt_n(n_dev, n_host);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  hl_hook_head(hk);
  if (tid == 0) s_tile = atomicInc(tile_ctr, gridDim.x - 1);
  for (int j = tid; j < HL_SORT_WAVES * NB; j += HL_SORT_THREADS) (&wcnt[0][0])[j] = 0;
  __syncthreads();
  const uint32_t tile = s_tile;
  if (st_next)  // this tile's status words of the next pass
    for (int j = tid; j < (int)TW; j += HL_SORT_THREADS) st_next[(size_t)tile * TW + j] = 0;
  const uint64_t tb = (uint64_t)tile * TILE;
  if (tb >= n) return;
  const uint32_t mask = (1u << b) - 1u;
  uint32_t key[ITEMS], val[ITEMS];
#pragma unroll
  for (int k = 0; k < ITEMS; ++k) {
    const uint64_t idx = tb + (uint64_t)w * (ITEMS * 64) + k * 64 + lane;
    const bool ok = idx < n;
    key[k] = ok ? kin[idx] : 0xFFFFFFFFu;
    val[k] = ok ? vin[idx] : 0u;
  }
  // global counts of the owned digits: loads issued with the keys', summed
  // after the ranking (which waits only for the keys)
  const int d0 = tid * PER;
  const bool owner = tid < OWNERS;
  uint32_t pv[PER][HL_SORT_HIST_BLOCKS];
#pragma unroll
  for (int q = 0; q < HL_SORT_HIST_BLOCKS; ++q) {
    const bool in = owner && (uint32_t)q < n_part;
    if constexpr (PER >= 2) {  // two digits per load
#pragma unroll
      for (int j = 0; j < PER; j += 2) {
        const uint2 x = in ? *reinterpret_cast<const uint2*>(part + (size_t)q * NB + d0 + j) : make_uint2(0u, 0u);
        pv[j][q] = x.x;
        pv[j + 1][q] = x.y;
      }
    } else {
      pv[0][q] = in ? part[(size_t)q * NB + d0] : 0u;
    }
  }
  // ranking, stable by construction: for each item slot the lanes holding the
  // same digit find one another with one ballot per digit bit (their peer
  // mask); the lowest peer adds the group's size to the wave's counter of that
  // digit (one atomic per distinct digit, so no two lanes of an instruction
  // touch one counter) and the others take its old value by a lane shuffle;
  // a lane's rank is that value plus its peers on lower lanes.  A wave's LDS
  // instructions execute in issue order, so the counters advance in item
  // order: ranks follow (item, lane) order, which is index order.
  uint32_t dg[ITEMS], lr[ITEMS];
  const uint64_t lt = (1ull << lane) - 1ull;
#pragma unroll
  for (int k = 0; k < ITEMS; ++k) {
    const uint64_t idx = tb + (uint64_t)w * (ITEMS * 64) + k * 64 + lane;
    const bool valid = idx < n;
    dg[k] = (key[k] >> shift) & mask;
    const uint64_t peers = hl_match_digit(dg[k], b, valid);
    const int leader = __ffsll((unsigned long long)peers) - 1;
    uint32_t base = 0;
    if (valid && lane == leader) base = atomicAdd(&wcnt[w][dg[k]], (uint32_t)__popcll(peers));
    base = __shfl(base, leader < 0 ? 0 : leader);
    lr[k] = valid ? base + (uint32_t)__popcll(peers & lt) : 0u;
  }
  uint32_t dtot[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    dtot[j] = 0;
#pragma unroll
    for (int q = 0; q < HL_SORT_HIST_BLOCKS; ++q) dtot[j] += pv[j][q];
  }
  __syncthreads();
  // wave-exclusive offsets of each owned digit; the totals are the tile's
  // counts, published at once for the later tiles
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
  }
  if (owner) {
    if constexpr (PER >= 2) {
#pragma unroll
      for (int j = 0; j < PER; j += 2)
        srt_st_store(st + (size_t)tile * TW + (d0 + j) / 2, SRT_AGG2 | tc[j] | (tc[j + 1] << 16));
    } else {
      srt_st_store(st + (size_t)tile * TW + d0, SRT_AGG | tc[0]);
    }
  }
  uint32_t gx[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) gx[j] = dtot[j];
  srt_scan2<NB, PER>(tx, gx, scan_ws);
  if (owner)
#pragma unroll
    for (int j = 0; j < PER; ++j) tdex[d0 + j] = tx[j];
  __syncthreads();
  // the tile in digit order in LDS (its own offsets are known now; the
  // earlier tiles' counts are read below)
#pragma unroll
  for (int k = 0; k < ITEMS; ++k) {
    const uint64_t idx = tb + (uint64_t)w * (ITEMS * 64) + k * 64 + lane;
    if (idx < n) {
      const uint32_t p = tdex[dg[k]] + wcnt[w][dg[k]] + lr[k];
      lk[p] = key[k];
      lv[p] = val[k];
    }
  }
  // counts of each owned digit in all earlier tiles: their published counts,
  // read CHUNK tiles at a time with every load in flight (no chain through
  // inclusive prefixes); a round with an unpublished word is read again
  uint32_t excl[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) excl[j] = 0;
  uint32_t spins = 0;
  for (uint32_t q0 = 0; owner && q0 < tile; q0 += CHUNK) {
    for (;;) {
      uint32_t wv[CHUNK][PW];
#pragma unroll
      for (int q = 0; q < CHUNK; ++q) {
        const bool in = q0 + q < tile;
        const uint32_t* a = st + (size_t)(q0 + q) * TW + (PER >= 2 ? d0 / 2 : d0);
        if constexpr (PW == 2) {
          const uint64_t x = in ? srt_st_load2(a) : ((uint64_t)SRT_AGG2 << 32 | SRT_AGG2);
          wv[q][0] = (uint32_t)x;
          wv[q][1] = (uint32_t)(x >> 32);
        } else {
          wv[q][0] = in ? srt_st_load(a) : (PER >= 2 ? SRT_AGG2 : SRT_AGG);
        }
      }
      bool ready = true;
      uint32_t sum[PER];
#pragma unroll
      for (int j = 0; j < PER; ++j) sum[j] = 0;
#pragma unroll
      for (int q = 0; q < CHUNK; ++q)
#pragma unroll
        for (int x = 0; x < PW; ++x) {
          const uint32_t v = wv[q][x];
          if constexpr (PER >= 2) {
            ready = ready && (v & SRT_AGG2) == SRT_AGG2;
            sum[2 * x] += v & 0x7FFFu;
            sum[2 * x + 1] += (v >> 16) & 0x7FFFu;
          } else {
            ready = ready && (v & SRT_AGG) != 0;
            sum[0] += v & SRT_VAL;
          }
        }
      if (ready) {
#pragma unroll
        for (int j = 0; j < PER; ++j) excl[j] += sum[j];
        break;
      }
      if (++spins > HL_SPIN_LIMIT) {
        hl_flag(err, HL_DEVERR_STALL);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  if (owner)
#pragma unroll
    for (int j = 0; j < PER; ++j) gbase[d0 + j] = gx[j] + excl[j];
  __syncthreads();
  const uint32_t nv = (uint32_t)min((uint64_t)TILE, (uint64_t)n - tb);
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

int hl_stream_cus(hipStream_t s) {
  uint32_t m[16] = {0};
  if (hipExtStreamGetCUMask(s, 16, m) != hipSuccess) return 0;
  int c = 0;
  for (uint32_t w : m) c += __builtin_popcount(w);
  return c;
}

hl_sort_geom hl_sort_geometry(uint32_t n_host, int bits, int cus) {
  const srt_plan pl = srt_make_plan(bits);
  hl_sort_geom g;
  g.passes = pl.passes;
  g.b = pl.b;
  g.nb = pl.nb;
  const uint32_t hb = hl_div_up(n_host, HL_SORT_HIST_THREADS * 8);
  g.hist_blocks = hb < 1 ? 1 : (hb > HL_SORT_HIST_BLOCKS ? HL_SORT_HIST_BLOCKS : hb);
  const uint32_t aim = cus > 0 && cus < HL_SORT_TILES_AIM ? (uint32_t)cus : HL_SORT_TILES_AIM;
  g.items = 12;
  for (int it : {4, 6})
    if (hl_div_up(n_host, HL_SORT_THREADS * it) <= aim) {
      g.items = it;
      break;
    }
  g.tile = HL_SORT_THREADS * g.items;
  g.n_zero = (uint64_t)hl_div_up(n_host, g.tile) * pl.nb;
  return g;
}

template <int NB>
static hl_status srt_hist_launch(hl_handle* h, hl_sort_ws& ws, const uint32_t* n_dev, uint32_t n_host, int bits,
                                 hipStream_t s) {
  const hl_sort_geom g = hl_sort_geometry(n_host, bits, hl_stream_cus(s));
  HL_KERNEL(h, s, "srt_hist", srt_hist<NB>, dim3(g.hist_blocks), dim3(HL_SORT_HIST_THREADS), 0, s, ws.k0, n_dev,
            n_host, g.passes, g.b, ws.part, ws.st[0], g.n_zero);
  HL_LAUNCHED();
  return HL_OK;
}

template <int NB, int ITEMS>
static hl_status srt_launch(hl_handle* h, hl_sort_ws& ws, const uint32_t* n_dev, uint32_t n_host, int bits,
                            hipStream_t s) {
  const hl_sort_geom g = hl_sort_geometry(n_host, bits, hl_stream_cus(s));
  const uint32_t tiles = hl_div_up(n_host, g.tile);
  uint32_t *ki = ws.k0, *vi = ws.v0, *ko = ws.k1, *vo = ws.v1;
  for (int p = 0; p < g.passes; ++p) {
    HL_KERNEL(h, s, "srt_pass", (srt_pass<NB, ITEMS>), dim3(tiles), dim3(HL_SORT_THREADS), 0, s, ki, vi, ko, vo, n_dev,
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
  const hl_sort_geom g = hl_sort_geometry(n_host, bits, hl_stream_cus(s));
#define SRT(NB)                                                                       \
  (g.items == 4 ? srt_launch<NB, 4>(h, ws, n_dev, n_host, bits, s)                    \
                : g.items == 6 ? srt_launch<NB, 6>(h, ws, n_dev, n_host, bits, s)     \
                               : srt_launch<NB, 12>(h, ws, n_dev, n_host, bits, s))
  if (g.nb == 256) st = SRT(256);
  else if (g.nb == 1024) st = SRT(1024);
  else st = SRT(2048);
#undef SRT
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
