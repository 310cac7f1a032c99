// Popularity classification, mu-batch partition (stable compaction), the
// gid -> hot-slot remap, and the dispatch kernel that does all of them (with
// the address generation) in one pass.
#include "hl_internal.h"

// ----------------------------------------------------------------------------- classify
// A block owns `spb` consecutive samples; their lookups are contiguous.  Threads
// probe one lookup each (coalesced ids, one bitmap word per probe); a non-hot
// lookup clears its sample's flag in LDS, the sample found by binary search
// over the block's sample offsets.
#define CL_MAX_SPB 1024
#define CL_U 4
__global__ void __launch_bounds__(256)
cl_kernel(const uint32_t* __restrict__ gids, const int32_t* __restrict__ bag_ptr, int32_t n_samples,
          int32_t bps, int32_t spb, const uint64_t* __restrict__ bitmap, uint64_t n_rows,
          uint8_t* __restrict__ flags, int64_t n_lookups, uint32_t* err) {
  __shared__ int32_t off[CL_MAX_SPB + 1];
  __shared__ uint8_t fl[CL_MAX_SPB];
  const int64_t s0 = (int64_t)blockIdx.x * spb;
  const int ns = (int)min((int64_t)spb, (int64_t)n_samples - s0);
  for (int j = threadIdx.x; j <= ns; j += blockDim.x) off[j] = bag_ptr[(s0 + j) * bps];
  for (int j = threadIdx.x; j < ns; j += blockDim.x) fl[j] = 1;
  if (blockIdx.x == 0 && threadIdx.x == 0 && bag_ptr[(int64_t)n_samples * bps] != n_lookups)
    hl_flag(err, HL_DEVERR_SHAPE);
  __syncthreads();
  // a bag_ptr that overruns n_lookups is flagged above; no id past n_lookups is read
  const int32_t lo = (int32_t)min((int64_t)off[0], n_lookups), hi = (int32_t)min((int64_t)off[ns], n_lookups);
  // CL_U lookups per thread at a time: their ids, then their bitmap words, in flight together
  for (int32_t i0 = lo + threadIdx.x; i0 < hi; i0 += CL_U * blockDim.x) {
    uint32_t g[CL_U];
#pragma unroll
    for (int u = 0; u < CL_U; ++u) {
      const int32_t i = i0 + u * (int32_t)blockDim.x;
      g[u] = i < hi ? gids[i] : 0u;
    }
    bool hot[CL_U];
#pragma unroll
    for (int u = 0; u < CL_U; ++u) hot[u] = g[u] < n_rows && hl_is_hot(bitmap, g[u]);
#pragma unroll
    for (int u = 0; u < CL_U; ++u) {
      const int32_t i = i0 + u * (int32_t)blockDim.x;
      if (i >= hi || hot[u]) continue;
      if (g[u] >= n_rows) hl_flag(err, HL_DEVERR_OUT_OF_RANGE);
      int a = 0, b = ns;
      while (b - a > 1) {
        int m = (a + b) >> 1;
        if (off[m] <= i) a = m; else b = m;
      }
      fl[a] = 0;
    }
  }
  __syncthreads();
  for (int j = threadIdx.x; j < ns; j += blockDim.x) flags[s0 + j] = fl[j];
}

// samples per classify block: about 512 lookups
static int64_t cl_spb(int32_t n_samples, int64_t n_lookups) {
  int64_t spb = n_lookups > 0 ? (512ll * n_samples + n_lookups - 1) / n_lookups : CL_MAX_SPB;
  return spb < 1 ? 1 : (spb > CL_MAX_SPB ? CL_MAX_SPB : spb);
}

extern "C" hl_status hl_classify(const hl_handle* h, const uint32_t* gids, const int32_t* bag_ptr,
                                 int32_t n_samples, int32_t bps, int64_t n_lookups, uint8_t* flags,
                                 hl_stream stream) {
  if (!h || n_samples < 0 || bps < 1 || n_lookups < 0) return HL_ERR_INVALID_ARG;
  if (n_samples == 0) return HL_OK;
  if (!bag_ptr || !flags || (n_lookups > 0 && !gids)) return HL_ERR_INVALID_ARG;
  if ((int64_t)n_samples * bps >= (1ll << 31)) return HL_ERR_UNSUPPORTED;
  const int64_t spb = cl_spb(n_samples, n_lookups);
  hipStream_t s = (hipStream_t)stream;
  HL_KERNEL(h, s, "cl_kernel", cl_kernel, dim3(hl_div_up(n_samples, spb)), dim3(256), 0, s, gids,
                     bag_ptr, n_samples, bps, (int32_t)spb, h->d_bitmap, h->n_rows, flags, n_lookups,
                     h->d_err);
  HL_LAUNCHED();
  return HL_OK;
}

// ----------------------------------------------------------------------------- partition
// Stable compaction of sample ids by flag.  A block of 1024 threads handles a
// tile of `tile` samples in chunks of 1024: a wave ballot gives each lane's
// rank among the wave's popular samples, the 16 wave totals are scanned in
// LDS, and a running carry links the chunks.  A popular sample goes to
// pop[p], a non-popular one to nonpop[i - p], p = popular samples before i.
// Tile prefixes: up to 1024 tiles of 1024 samples, every block adds up the
// counts of the tiles before it; beyond that, 64K-sample tiles and a serial
// scan of their counts.
#define PT_SMALL 1024
#define PT_BIG 65536
__global__ void __launch_bounds__(1024)
pt_count(const uint8_t* __restrict__ flags, int32_t n, int32_t tile, uint32_t* tile_cnt) {
  __shared__ uint32_t red[1024];
  const int64_t base = (int64_t)blockIdx.x * tile;
  uint32_t c = 0;
  for (int k = 0; k < tile / 1024; ++k) {
    const int64_t i = base + k * 1024 + threadIdx.x;
    if (i < n) c += flags[i] != 0;
  }
  red[threadIdx.x] = c;
  __syncthreads();
  for (int o = 512; o > 0; o >>= 1) {
    if (threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) tile_cnt[blockIdx.x] = red[0];
}

__global__ void __launch_bounds__(1024)
pt_scan(uint32_t* tile_cnt, int32_t n_tiles) {
  if (threadIdx.x == 0) {
    uint32_t acc = 0;
    for (int32_t t = 0; t < n_tiles; ++t) {
      uint32_t v = tile_cnt[t];
      tile_cnt[t] = acc;
      acc += v;
    }
  }
}

// prefix_mode 0: no other tiles; 1: tile_cnt holds raw counts (sum those before
// this tile); 2: tile_cnt holds exclusive prefixes.
__global__ void __launch_bounds__(1024)
pt_emit(const uint8_t* __restrict__ flags, int32_t n, int32_t tile, const uint32_t* tile_cnt, int prefix_mode,
        int32_t* __restrict__ pop, int32_t* __restrict__ nonpop, int32_t* counts) {
  __shared__ uint32_t wtot[16];
  __shared__ uint32_t carry;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t base = (int64_t)blockIdx.x * tile;
  if (prefix_mode == 1) {
    uint32_t c = 0;
    for (uint32_t t = threadIdx.x; t < blockIdx.x; t += blockDim.x) c += tile_cnt[t];
    for (int o = 32; o > 0; o >>= 1) c += __shfl_down(c, o);
    if (lane == 0) wtot[w] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t t = 0;
      for (int j = 0; j < 16; ++j) t += wtot[j];
      carry = t;
    }
  } else if (threadIdx.x == 0) {
    carry = prefix_mode == 2 ? tile_cnt[blockIdx.x] : 0u;
  }
  __syncthreads();
  const uint64_t lt = (1ull << lane) - 1ull;
  for (int k = 0; k < tile / 1024; ++k) {
    const int64_t c0 = base + k * 1024;
    if (c0 >= n) break;
    const int64_t i = c0 + threadIdx.x;
    const bool valid = i < n;
    const bool p = valid && flags[i] != 0;
    const uint64_t b = __ballot(p);
    if (lane == 0) wtot[w] = __popcll(b);
    __syncthreads();
    uint32_t before = carry;
    for (int j = 0; j < w; ++j) before += wtot[j];
    before += __popcll(b & lt);
    if (valid) {
      if (p) pop[before] = (int32_t)i;
      else nonpop[i - before] = (int32_t)i;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t t = 0;
      for (int j = 0; j < 16; ++j) t += wtot[j];
      carry += t;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0 && (blockIdx.x == gridDim.x - 1)) {
    counts[0] = (int32_t)carry;
    counts[1] = n - (int32_t)carry;
  }
}

// Up to PT_ONE samples: one block; a thread holds 4 consecutive flags of each
// chunk of 4096 (one 4-byte load when the flags are 4-byte aligned), a wave
// scan gives each thread the popular samples before its 4 within the wave,
// the totals of every (chunk, wave) go to LDS, one wave scans them in (chunk,
// wave) order, which is index order, and every sample is then placed: one
// launch, two barriers.
#define PT_ONE 16384
template <int C>  // chunks of 4096 samples (1, 2 or 4): each thread holds 4 consecutive samples of a chunk
__global__ void __launch_bounds__(1024)
pt_one(const uint8_t* __restrict__ flags, int32_t n, int aligned, int32_t* __restrict__ pop,
       int32_t* __restrict__ nonpop, int32_t* counts) {
  __shared__ uint32_t wt[C * 16];
  __shared__ uint32_t s_total;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint32_t f[C], ex[C];  // f: the 4 samples' flags as bits 0..3; ex: popular samples before them in the wave
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int32_t b = c * 4096 + 4 * (int32_t)threadIdx.x;
    uint32_t v = 0;
    if (aligned && b + 3 < n) {
      const uint32_t x = *reinterpret_cast<const uint32_t*>(flags + b);
#pragma unroll
      for (int q = 0; q < 4; ++q) v |= (((x >> (8 * q)) & 0xFFu) != 0u ? 1u : 0u) << q;
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) v |= (b + q < n && flags[b + q] != 0 ? 1u : 0u) << q;
    }
    f[c] = v;
  }
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const uint32_t cnt = (uint32_t)__popc(f[c]);
    uint32_t x = cnt;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = __shfl_up(x, o);
      if (lane >= o) x += y;
    }
    ex[c] = x - cnt;
    if (lane == 63) wt[c * 16 + w] = x;
  }
  __syncthreads();
  if (w == 0) {  // the C*16 wave totals (at most 64, one per lane), scanned in order
    const uint32_t v = lane < C * 16 ? wt[lane] : 0u;
    uint32_t x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = __shfl_up(x, o);
      if (lane >= o) x += y;
    }
    if (lane < C * 16) wt[lane] = x - v;
    if (lane == 63) s_total = x;
  }
  __syncthreads();
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int32_t b = c * 4096 + 4 * (int32_t)threadIdx.x;
    uint32_t before = wt[c * 16 + w] + ex[c];  // popular samples before sample b
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int32_t i = b + q;
      if (i >= n) break;
      if ((f[c] >> q) & 1u) pop[before++] = i;
      else nonpop[i - (int32_t)before] = i;
    }
  }
  if (threadIdx.x == 0) {
    counts[0] = (int32_t)s_total;
    counts[1] = n - (int32_t)s_total;
  }
}

size_t hl_partition_ws_bytes(int32_t max_samples) {
  return HL_WS_HEADER + 4 * ((size_t)(max_samples + PT_SMALL - 1) / PT_SMALL + 64);
}

extern "C" hl_status hl_partition(hl_handle* h, const uint8_t* flags, int32_t n, int32_t* pop,
                                  int32_t* nonpop, int32_t* counts, void* ws, size_t ws_bytes,
                                  hl_stream stream) {
  if (!h || n < 0 || !counts || (n > 0 && (!flags || !pop || !nonpop))) return HL_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  if (n <= PT_ONE) {
    const int al = ((uintptr_t)flags & 3u) == 0;
    if (n <= 4096) HL_KERNEL(h, s, "pt_one", pt_one<1>, dim3(1), dim3(1024), 0, s, flags, n, al, pop, nonpop, counts);
    else if (n <= 8192) HL_KERNEL(h, s, "pt_one", pt_one<2>, dim3(1), dim3(1024), 0, s, flags, n, al, pop, nonpop, counts);
    else HL_KERNEL(h, s, "pt_one", pt_one<4>, dim3(1), dim3(1024), 0, s, flags, n, al, pop, nonpop, counts);
    HL_LAUNCHED();
    return HL_OK;
  }
  const bool small = n <= PT_SMALL * 1024;
  const int32_t tile = small ? PT_SMALL : PT_BIG;
  const int32_t tiles = n == 0 ? 1 : (int32_t)hl_div_up(n, tile);
  uint32_t* tc = nullptr;
  int mode = 0;
  if (tiles > 1) {
    if (!ws || ws_bytes < hl_partition_ws_bytes(n)) return HL_ERR_CAPACITY;
    hl_ws_note(h, ws, HL_WSK_OTHER);
    tc = (uint32_t*)((char*)ws + HL_WS_HEADER);
    HL_KERNEL(h, s, "pt_count", pt_count, dim3(tiles), dim3(1024), 0, s, flags, n, tile, tc);
    if (small) {
      mode = 1;
    } else {
      HL_KERNEL(h, s, "pt_scan", pt_scan, dim3(1), dim3(1024), 0, s, tc, tiles);
      mode = 2;
    }
  }
  HL_KERNEL(h, s, "pt_emit", pt_emit, dim3(tiles), dim3(1024), 0, s, flags, n, tile, tc, mode, pop, nonpop, counts);
  HL_LAUNCHED();
  return HL_OK;
}

// ----------------------------------------------------------------------------- remap
__global__ void __launch_bounds__(256)
rm_kernel(const uint32_t* __restrict__ gids, int64_t n, const uint64_t* __restrict__ bitmap,
          const uint32_t* __restrict__ rank, uint64_t n_rows, int32_t* __restrict__ codes, uint32_t* err) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t g = gids[i];
    int32_t c = -1;
    if (g < n_rows) c = hl_hot_slot(bitmap, rank, g);
    else hl_flag(err, HL_DEVERR_OUT_OF_RANGE);
    codes[i] = c;
  }
}

extern "C" hl_status hl_remap(const hl_handle* h, const uint32_t* gids, int64_t n, int32_t* codes,
                              hl_stream stream) {
  if (!h || n < 0 || (n > 0 && (!gids || !codes))) return HL_ERR_INVALID_ARG;
  if (n == 0) return HL_OK;
  uint32_t g = hl_div_up(n, 256);
  if (g > 65535) g = 65535;
  hipStream_t s = (hipStream_t)stream;
  HL_KERNEL(h, s, "rm_kernel", rm_kernel, dim3(g), dim3(256), 0, s, gids, n, h->d_bitmap, h->d_rank,
                     h->n_rows, codes, h->d_err);
  HL_LAUNCHED();
  return HL_OK;
}

// ----------------------------------------------------------------------------- dispatch
// The Data Dispatcher of Sec. V-A in one kernel: a block owns `spb` consecutive
// samples (their bag offsets in LDS); per lookup it forms the gid from the
// table base (address generation), probes the hot-set bitmap (input
// classifier), writes the hot slot or -1 (remap) and clears its sample's flag
// when the row is not hot; then the popular samples of all earlier blocks,
// obtained by decoupled look-back, place each sample in the popular or the
// non-popular list (fragmentation, Eq. 3).  The look-back status words live in
// the workspace header, tagged with an epoch kept on the device: the last block
// to finish advances it, so no clearing is needed between calls (nor between
// replays of a captured graph).
#define DS_THREADS 512
#define DS_MAX_TABLES 1024  // table bases and sizes in LDS up to this many tables
#define DS_MAX_BAGS 4096
#define DS_MAX_SPB 2048
#define DS_LOOKUPS_MIN 512  // lookups per block: n_lookups / DS_BLOCKS_AIM within these bounds
#define DS_LOOKUPS_MAX 2048
#define DS_BLOCKS_AIM 64
#define DS_MAP 8192         // lookups per block mapped to their bag in LDS
#define DS_EPOCH 0
#define DS_DONE 1
#define DS_TILE 2
__global__ void __launch_bounds__(DS_THREADS)
ds_kernel(const uint32_t* __restrict__ rows, const int32_t* __restrict__ bag_ptr, int32_t n_samples, int32_t bps,
          int32_t spb, const uint32_t* __restrict__ base, const uint32_t* __restrict__ nrow, int32_t n_tables,
          const uint64_t* __restrict__ bitmap, const uint32_t* __restrict__ rank, uint64_t n_rows,
          uint32_t* __restrict__ gids, int32_t* __restrict__ codes, uint8_t* __restrict__ flags, int32_t* pop,
          int32_t* nonpop, int32_t* counts, int64_t n_lookups, uint32_t* hdr, uint64_t* st, uint32_t* err,
          hl_hook hk, hl_cg_fused cf) {
  __shared__ int32_t off[DS_MAX_BAGS + 1];
  __shared__ uint32_t tb_base[DS_MAX_TABLES], tb_rows[DS_MAX_TABLES];
  __shared__ uint8_t fl[DS_MAX_SPB];
  __shared__ uint16_t bmap[DS_MAP];  // lookup - lo -> bag within the block
  __shared__ uint32_t s_tile, s_epoch, wsum[DS_THREADS / 64];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  hl_hook_head(hk);
  hl_hook_gate(hk);
  if (tid == 0) {
    s_tile = atomicInc(hdr + DS_TILE, gridDim.x - 1);
    // status words of earlier calls carry older epochs; zeroed words carry no flag
    s_epoch = __hip_atomic_load(hdr + DS_EPOCH, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  const uint32_t tile = s_tile, epoch = s_epoch;
  const int64_t s0 = (int64_t)tile * spb;
  const int ns = (int)min((int64_t)spb, (int64_t)n_samples - s0);
  const int64_t bg0 = s0 * bps;
  const int nbg = ns * bps;
  for (int j = tid; j <= nbg; j += DS_THREADS) off[j] = bag_ptr[bg0 + j];
  // the first round's rows, loaded before the offsets reach LDS (their range
  // needs only the block's first and last offsets)
  const int32_t lo0 = bag_ptr[bg0], hi0 = (int32_t)min((int64_t)bag_ptr[bg0 + nbg], n_lookups);
  uint32_t r0[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int32_t i = lo0 + tid + k * DS_THREADS;
    r0[k] = i < hi0 ? rows[i] : 0u;
  }
  for (int j = tid; j < ns; j += DS_THREADS) fl[j] = 1;
  for (int j = tid; j < n_tables; j += DS_THREADS) {
    tb_base[j] = base[j];
    tb_rows[j] = nrow[j];
  }
  if (tile == 0 && tid == 0 && bag_ptr[(int64_t)n_samples * bps] != n_lookups) hl_flag(err, HL_DEVERR_SHAPE);
  if (cf.table)  // the fused plan's rank scan status, cleared for the scan that follows
    for (uint32_t j = blockIdx.x * DS_THREADS + tid; j < cf.rtiles; j += gridDim.x * DS_THREADS) cf.rstat[j] = 0;
  __syncthreads();
  const int32_t lo = off[0], hi = (int32_t)min((int64_t)off[nbg], n_lookups);
  // each lookup's bag from an LDS map built bag by bag (a binary search over the
  // offsets when the block holds more lookups than the map)
  const bool mapped = hi - lo <= DS_MAP;
  if (mapped) {
    for (int j = tid; j < nbg; j += DS_THREADS) {
      const int32_t e = min(off[j + 1], hi);
      for (int32_t q = max(off[j], lo); q < e; ++q) bmap[q - lo] = (uint16_t)j;
    }
    __syncthreads();
  }
  // the table of bag j is (t0 + j) % n_tables, its sample j / bps
  const uint32_t t0 = (uint32_t)(bg0 % n_tables);
  const float inv_t = 1.0f / (float)n_tables, inv_b = 1.0f / (float)bps;
  // 4 lookups per thread per round, their loads issued together
  for (int32_t i0 = lo + tid; i0 < hi; i0 += 4 * DS_THREADS) {
    const bool first = i0 == lo + tid;
    int a[4];
    uint32_t r[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int32_t i = i0 + k * DS_THREADS;
      int x = 0, y = nbg;  // off[x] <= i < off[y]
      if (i < hi) {
        if (mapped) x = bmap[i - lo];
        else
          while (y - x > 1) {
            const int m = (x + y) >> 1;
            if (off[m] <= i) x = m; else y = m;
          }
      }
      a[k] = x;
      r[k] = first ? r0[k] : (i < hi ? rows[i] : 0u);
    }
    uint32_t g[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      uint32_t t;
      (void)hl_fdiv(t0 + (uint32_t)a[k], (uint32_t)n_tables, inv_t, &t);
      const bool in = i0 + k * DS_THREADS < hi;
      g[k] = 0xFFFFFFFFu;
      if (in) {
        if (r[k] < tb_rows[t]) g[k] = tb_base[t] + r[k];
        else hl_flag(err, HL_DEVERR_OUT_OF_RANGE);
      }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int32_t i = i0 + k * DS_THREADS;
      if (i >= hi) continue;
      const int32_t c = g[k] < n_rows ? hl_hot_slot(bitmap, rank, g[k]) : -1;
      gids[i] = g[k];
      codes[i] = c;
      uint32_t rm;
      if (c < 0) {
        fl[hl_fdiv((uint32_t)a[k], (uint32_t)bps, inv_b, &rm)] = 0;
        // the fused plan: the cold plan's insert (an id out of range takes no slot)
        if (cf.table) cf.slotof[i] = g[k] < n_rows ? hl_cg_insert(cf.table, cf.S - 1, g[k], (uint32_t)i) : 0xFFFFFFFFu;
      }
    }
  }
  __syncthreads();
  // popular samples of this block: exclusive ranks over its samples (4 per thread)
  uint32_t f4[4], loc = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int j = tid * 4 + k;
    f4[k] = j < ns ? fl[j] : 0u;
    loc += f4[k];
  }
  uint32_t inc = loc;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t t2 = __shfl_up(inc, o);
    if (lane >= o) inc += t2;
  }
  if (lane == 63) wsum[w] = inc;
  __syncthreads();
  uint32_t before = inc - loc, tc = 0;
  for (int q = 0; q < DS_THREADS / 64; ++q) {
    if (q < w) before += wsum[q];
    tc += wsum[q];
  }
  if (tid == 0) hl_st_store(st + tile, hl_st_pack(epoch, tile == 0 ? HL_ST_PRE : HL_ST_AGG, tc));
  const uint32_t ex = tile > 0 ? hl_block_lookback(st, tile, epoch, err) : 0u;
  if (tid == 0 && tile > 0) hl_st_store(st + tile, hl_st_pack(epoch, HL_ST_PRE, ex + tc));
  uint32_t pp = ex + before;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int j = tid * 4 + k;
    if (j >= ns) continue;
    const int32_t sid = (int32_t)(s0 + j);
    flags[sid] = (uint8_t)f4[k];
    if (f4[k]) pop[pp++] = sid;
    else nonpop[sid - (int32_t)pp] = sid;
  }
  if (tile == gridDim.x - 1 && tid == 0) {
    counts[0] = (int32_t)(ex + tc);
    counts[1] = n_samples - (int32_t)(ex + tc);
  }
  // the last block to finish advances the epoch for the next call
  if (tid == 0 && atomicInc(hdr + DS_DONE, gridDim.x - 1) == gridDim.x - 1)
    __hip_atomic_store(hdr + DS_EPOCH, epoch + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// the samples per block of the fused dispatch, or 0 when it takes the step by
// step calls
static int64_t ds_spb(const hl_handle* h, int32_t n_samples, int32_t bps, int64_t n_lookups, const void* workspace,
                      size_t ws_bytes) {
  // About 64 blocks: fewer leave a small mini-batch's dependent loads to a few
  // CUs, more lengthen the look-back chain and the cold inserts' contention.
  int64_t lpb = n_lookups / DS_BLOCKS_AIM;
  lpb = lpb < DS_LOOKUPS_MIN ? DS_LOOKUPS_MIN : (lpb > DS_LOOKUPS_MAX ? DS_LOOKUPS_MAX : lpb);
  int64_t spb = n_lookups > 0 ? (lpb * n_samples + n_lookups - 1) / n_lookups : DS_MAX_SPB;
  const int64_t bag_cap = DS_MAX_BAGS / bps;
  if (spb > bag_cap) spb = bag_cap;
  if (spb > DS_MAX_SPB) spb = DS_MAX_SPB;
  if (spb < 1) spb = 1;
  const int64_t tiles = n_samples > 0 ? (n_samples + spb - 1) / spb : 0;
  if (tiles == 0 || bps > DS_MAX_BAGS || tiles > HL_DISP_MAX_TILES || h->n_tables > DS_MAX_TABLES || !workspace ||
      ws_bytes < HL_WS_HEADER)
    return 0;
  return spb;
}

bool hl_dispatch_fused(const hl_handle* h, int32_t n_samples, int32_t bps, int64_t n_lookups, const void* workspace,
                       size_t ws_bytes) {
  return h && bps >= 1 && n_samples >= 0 && ds_spb(h, n_samples, bps, n_lookups, workspace, ws_bytes) > 0;
}

extern "C" hl_status hl_dispatch(hl_handle* h, const uint32_t* rows, const int32_t* bag_ptr, int32_t n_samples,
                                 int32_t bps, int64_t n_lookups, uint32_t* gids, int32_t* codes, uint8_t* flags,
                                 int32_t* pop_ids, int32_t* nonpop_ids, int32_t* counts_dev, void* workspace,
                                 size_t ws_bytes, hl_stream stream) {
  return hl_dispatch_ex(h, rows, bag_ptr, n_samples, bps, n_lookups, gids, codes, flags, pop_ids, nonpop_ids,
                        counts_dev, workspace, ws_bytes, stream, nullptr);
}

hl_status hl_dispatch_ex(hl_handle* h, const uint32_t* rows, const int32_t* bag_ptr, int32_t n_samples, int32_t bps,
                         int64_t n_lookups, uint32_t* gids, int32_t* codes, uint8_t* flags, int32_t* pop_ids,
                         int32_t* nonpop_ids, int32_t* counts_dev, void* workspace, size_t ws_bytes,
                         hl_stream stream, const hl_cg_fused* cf) {
  if (!h || n_samples < 0 || bps < 1 || n_lookups < 0 || !counts_dev || !bag_ptr) return HL_ERR_INVALID_ARG;
  if (n_samples > 0 && (!flags || !pop_ids || !nonpop_ids)) return HL_ERR_INVALID_ARG;
  if (n_lookups > 0 && (!rows || !gids || !codes)) return HL_ERR_INVALID_ARG;
  if ((int64_t)n_samples * bps >= (1ll << 31) || n_lookups >= (1ll << 31)) return HL_ERR_UNSUPPORTED;
  hipStream_t s = (hipStream_t)stream;
  const int64_t spb = ds_spb(h, n_samples, bps, n_lookups, workspace, ws_bytes);
  const int64_t tiles = spb ? (n_samples + spb - 1) / spb : 0;
  if (!spb && cf && cf->table) return HL_ERR_INVALID_ARG;  // the fused plan needs the fused dispatch
  if (!spb) {
    // the step by step calls (also for an empty batch)
    hl_status st = hl_lookup_gids(h, rows, bag_ptr, (int64_t)n_samples * bps, gids, stream);
    if (st == HL_OK) st = hl_classify(h, gids, bag_ptr, n_samples, bps, n_lookups, flags, stream);
    if (st == HL_OK) st = hl_partition(h, flags, n_samples, pop_ids, nonpop_ids, counts_dev, workspace, ws_bytes, stream);
    if (st == HL_OK) st = hl_remap(h, gids, n_lookups, codes, stream);
    return st;
  }
  uint32_t* hdr = (uint32_t*)workspace + HL_HDR_DISP;
  uint64_t* stw = (uint64_t*)((uint32_t*)workspace + HL_HDR_DSTAT);
  HL_KERNEL(h, s, "ds_kernel", ds_kernel, dim3((uint32_t)tiles), dim3(DS_THREADS), 0, s, rows, bag_ptr, n_samples, bps,
            (int32_t)spb, h->d_base, h->d_rows, h->n_tables, h->d_bitmap, h->d_rank, h->n_rows, gids, codes, flags,
            pop_ids, nonpop_ids, counts_dev, n_lookups, hdr, stw, h->d_err, hl_hook_take(h), cf ? *cf : hl_cg_fused{});
  HL_LAUNCHED();
  return HL_OK;
}
