// Hot-set selection from access counts: exact top-K by (count desc, id asc)
// among rows accessed at least once, and installation of an explicit hot set.
//
// Selection is a most-significant-digit radix select on the 32-bit counts
// (four 8-bit levels) that finds the K-th largest count tau and how many rows
// with count == tau still fit (need_tau).  A row is hot iff count > tau, or
// count == tau and fewer than need_tau rows with count == tau have a smaller
// id.  The output pass then streams ids in ascending order, so hot slots are
// ascending-id ranks by construction, and writes hot ids, the membership
// bitmap and the rank directory in one pass.
#include "hl_internal.h"

#define HL_TRY_ST(x)                  \
  do {                                \
    const hl_status _st = (x);        \
    if (_st != HL_OK) return _st;     \
  } while (0)

#define TK_BLOCKS 1024
#define TK_STATE 16
// state words
#define S_PREFIX 0
#define S_NEED 1
#define S_NGT 2
#define S_DONE 3
#define S_TAU 4
#define S_NEEDTAU 5
#define S_NONZERO 6
#define S_NHOT 7
#define S_CTR 8

size_t hl_topk_scratch_bytes(uint64_t n_rows) {
  uint64_t tiles = (n_rows + 4095) / 4096;
  return 4 * (TK_STATE + (size_t)TK_BLOCKS * 257 + 2 * tiles + 64);
}

__global__ void tk_init(uint32_t* st, uint32_t k) {
  st[S_PREFIX] = 0;
  st[S_NEED] = k;
  st[S_NGT] = 0;
  st[S_DONE] = (k == 0);
  st[S_TAU] = k == 0 ? 0xFFFFFFFFu : 0u;
  st[S_NEEDTAU] = 0;
  st[S_NONZERO] = 0;
  st[S_NHOT] = 0;
}

// One radix-select level over counts >= 1 whose higher digits match the prefix
// found so far.  The last block to finish merges the per-block histograms and
// picks the digit where the running count from the top reaches `need`.
__global__ void __launch_bounds__(256)
tk_level(const uint32_t* __restrict__ counts, uint64_t n, uint32_t* st, int level, uint32_t k) {
  if (st[S_DONE]) return;
  __shared__ uint32_t hist[256];
  __shared__ uint32_t nzs;
  __shared__ bool last;
  uint32_t* part = st + TK_STATE;
  hist[threadIdx.x] = 0;
  if (threadIdx.x == 0) nzs = 0;
  __syncthreads();
  const int shift = 24 - 8 * level;
  const uint32_t prefix = st[S_PREFIX];
  uint32_t nz = 0;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (uint64_t)gridDim.x * blockDim.x) {
    const uint32_t c = counts[i];
    if (c == 0) continue;
    ++nz;
    if (level == 0 || (c >> (shift + 8)) == (prefix >> (shift + 8)))
      atomicAdd(&hist[(c >> shift) & 255u], 1u);
  }
  if (level == 0) atomicAdd(&nzs, nz);
  __syncthreads();
  part[blockIdx.x * 257 + threadIdx.x] = hist[threadIdx.x];
  if (threadIdx.x == 0) part[blockIdx.x * 257 + 256] = nzs;
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) last = atomicInc(st + S_CTR, gridDim.x - 1) == gridDim.x - 1;
  __syncthreads();
  if (!last) return;
  __threadfence();
  uint32_t tot = 0;
  for (uint32_t b = 0; b < gridDim.x; ++b) tot += part[b * 257 + threadIdx.x];
  hist[threadIdx.x] = tot;
  __syncthreads();
  if (threadIdx.x != 0) return;
  if (level == 0) {
    uint32_t nonzero = 0;
    for (uint32_t b = 0; b < gridDim.x; ++b) nonzero += part[b * 257 + 256];
    st[S_NONZERO] = nonzero;
    if (nonzero <= k) {  // every accessed row fits: select count >= 1
      st[S_TAU] = 1;
      st[S_NEEDTAU] = 0xFFFFFFFFu;
      st[S_DONE] = 1;
      return;
    }
  }
  uint32_t need = st[S_NEED], cum = 0;
  int d = 255;
  for (; d > 0; --d) {
    if (cum + hist[d] >= need) break;
    cum += hist[d];
  }
  st[S_PREFIX] = prefix | ((uint32_t)d << shift);
  st[S_NGT] += cum;
  st[S_NEED] = need - cum;
  if (level == 3) {
    st[S_TAU] = prefix | (uint32_t)d;
    st[S_NEEDTAU] = need - cum;
    st[S_DONE] = 1;
  }
}

// Per 4096-id tile: rows with count > tau and rows with count == tau.
__global__ void __launch_bounds__(256)
tk_tiles(const uint32_t* __restrict__ counts, uint64_t n, uint32_t* st, uint64_t n_tiles) {
  const uint32_t tau = st[S_TAU];
  uint32_t* ts = st + TK_STATE + TK_BLOCKS * 257;
  uint32_t* te = ts + n_tiles;
  const uint64_t base = (uint64_t)blockIdx.x * 4096;
  uint32_t s = 0, e = 0;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const uint64_t g = base + k * 256 + threadIdx.x;
    const uint32_t c = g < n ? counts[g] : 0u;
    s += (c > tau) & (c != 0);
    e += (c == tau) & (c != 0);
  }
  __shared__ uint32_t rs[256], re[256];
  rs[threadIdx.x] = s;
  re[threadIdx.x] = e;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) {
      rs[threadIdx.x] += rs[threadIdx.x + o];
      re[threadIdx.x] += re[threadIdx.x + o];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    ts[blockIdx.x] = rs[0];
    te[blockIdx.x] = re[0];
  }
}

// Exclusive scan (in place) of both tile-count arrays by one block; totals give
// n_hot = strict + min(need_tau, equal).
__global__ void __launch_bounds__(1024)
tk_scan(uint32_t* st, uint64_t n_tiles, uint32_t* rank_last) {
  uint32_t* ts = st + TK_STATE + TK_BLOCKS * 257;
  uint32_t* te = ts + n_tiles;
  __shared__ uint32_t ws[16], we[16];
  __shared__ uint32_t carry_s, carry_e;
  if (threadIdx.x == 0) carry_s = carry_e = 0;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  for (uint64_t c0 = 0; c0 < n_tiles; c0 += 1024) {
    const uint64_t i = c0 + threadIdx.x;
    uint32_t vs = i < n_tiles ? ts[i] : 0, ve = i < n_tiles ? te[i] : 0;
    uint32_t is = vs, ie = ve;
    for (int o = 1; o < 64; o <<= 1) {
      uint32_t a = __shfl_up(is, o), b = __shfl_up(ie, o);
      if (lane >= o) { is += a; ie += b; }
    }
    if (lane == 63) { ws[w] = is; we[w] = ie; }
    __syncthreads();
    uint32_t ps = carry_s, pe = carry_e;
    for (int j = 0; j < w; ++j) { ps += ws[j]; pe += we[j]; }
    if (i < n_tiles) { ts[i] = ps + is - vs; te[i] = pe + ie - ve; }
    __syncthreads();
    if (threadIdx.x == 1023) { carry_s = ps + is; carry_e = pe + ie; }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const uint32_t need = st[S_NEEDTAU];
    const uint32_t nh = carry_s + (carry_e < need ? carry_e : need);
    st[S_NHOT] = nh;
    *rank_last = nh;
  }
}

// Output pass: wave w of the block streams ids [tile*4096 + w*1024, +1024) in
// ascending order, 64 at a time.
__global__ void __launch_bounds__(256)
tk_emit(uint32_t* __restrict__ counts, uint64_t n, const uint32_t* st, uint64_t n_tiles,
        uint32_t* __restrict__ hot_ids, uint64_t* __restrict__ bitmap, uint32_t* __restrict__ rank,
        int reset) {
  const uint32_t tau = st[S_TAU], need = st[S_NEEDTAU];
  const uint32_t* ts = st + TK_STATE + TK_BLOCKS * 257;
  const uint32_t* te = ts + n_tiles;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const uint64_t base = (uint64_t)blockIdx.x * 4096 + (uint64_t)w * 1024;
  uint32_t c[16];
  uint32_t ns = 0, ne = 0;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const uint64_t g = base + k * 64 + lane;
    c[k] = g < n ? counts[g] : 0u;
    ns += __popcll(__ballot((c[k] > tau) & (c[k] != 0)));
    ne += __popcll(__ballot((c[k] == tau) & (c[k] != 0)));
  }
  __shared__ uint32_t wsum[4], wequ[4];
  if (lane == 0) { wsum[w] = ns; wequ[w] = ne; }
  __syncthreads();
  uint32_t sb = ts[blockIdx.x], eb = te[blockIdx.x];
  for (int j = 0; j < w; ++j) { sb += wsum[j]; eb += wequ[j]; }
  const uint64_t lt = (1ull << lane) - 1ull;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const uint64_t g = base + k * 64 + lane;
    const bool s = (c[k] > tau) & (c[k] != 0), e = (c[k] == tau) & (c[k] != 0);
    const uint64_t bs = __ballot(s), be = __ballot(e);
    const uint32_t sbef = sb + __popcll(bs & lt), ebef = eb + __popcll(be & lt);
    const uint32_t pos = sbef + (ebef < need ? ebef : need);
    const bool sel = s || (e && ebef < need);
    if (sel) hot_ids[pos] = (uint32_t)g;
    const uint64_t bsel = __ballot(sel);
    if (lane == 0) bitmap[g >> 6] = bsel;
    if ((g & 255) == 0) rank[g >> 8] = pos;
    if (reset && g < n) counts[g] = 0;
    sb += __popcll(bs);
    eb += __popcll(be);
  }
}

extern "C" hl_status hl_profile_topk(hl_handle* h, uint32_t k, uint32_t* hot_ids_out, uint32_t* n_hot_out,
                                     int reset_counts, hl_stream stream) {
  if (!h || !hot_ids_out) return HL_ERR_INVALID_ARG;
  if (k > h->k_cap) return HL_ERR_OUT_OF_RANGE;
  hipStream_t s = (hipStream_t)stream;
  const uint64_t n = h->n_rows, tiles = h->n_tiles4k;
  uint32_t nb = hl_div_up(n, 256 * 16);
  if (nb > TK_BLOCKS) nb = TK_BLOCKS;
  HL_KERNEL(h, s, "tk_init", tk_init, dim3(1), dim3(1), 0, s, h->d_tk, k);
  for (int lvl = 0; lvl < 4; ++lvl)
    HL_KERNEL(h, s, "tk_level", tk_level, dim3(nb), dim3(256), 0, s, h->d_counts, n, h->d_tk, lvl, k);
  HL_KERNEL(h, s, "tk_tiles", tk_tiles, dim3((uint32_t)tiles), dim3(256), 0, s, h->d_counts, n, h->d_tk, tiles);
  HL_KERNEL(h, s, "tk_scan", tk_scan, dim3(1), dim3(1024), 0, s, h->d_tk, tiles, h->d_rank + tiles * 16);
  HL_KERNEL(h, s, "tk_emit", tk_emit, dim3((uint32_t)tiles), dim3(256), 0, s, h->d_counts, n, h->d_tk, tiles,
                     hot_ids_out, h->d_bitmap, h->d_rank, reset_counts);
  HL_LAUNCHED();
  HL_TRY_ST(hl_table_bounds(h, s));
  uint32_t nh = 0;
  HL_HIP(hipMemcpyAsync(&nh, h->d_tk + S_NHOT, 4, hipMemcpyDeviceToHost, s));
  HL_HIP(hipStreamSynchronize(s));
  h->n_hot = nh;
  if (n_hot_out) *n_hot_out = nh;
  return HL_OK;
}

// ----------------------------------------------------------------------------- explicit hot set
__global__ void __launch_bounds__(256)
sh_bits(const uint32_t* __restrict__ ids, uint32_t n_hot, uint64_t n_rows, uint64_t* bitmap, uint32_t* err) {
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n_hot; i += gridDim.x * blockDim.x) {
    const uint32_t g = ids[i];
    const bool ok = g < n_rows && (i == 0 || ids[i - 1] < g);
    if (!ok) { hl_flag(err, HL_DEVERR_BAD_HOTSET); continue; }
    atomicOr((unsigned long long*)(bitmap + (g >> 6)), 1ull << (g & 63));
  }
}

__global__ void __launch_bounds__(256)
sh_rank(const uint32_t* __restrict__ ids, uint32_t n_hot, uint64_t n_entries, uint32_t* rank) {
  for (uint64_t j = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n_entries;
       j += (uint64_t)gridDim.x * blockDim.x) {
    const uint64_t key = j * 256;
    uint32_t a = 0, b = n_hot;  // first index with ids[idx] >= key
    while (a < b) {
      uint32_t m = (a + b) >> 1;
      if ((uint64_t)ids[m] < key) a = m + 1; else b = m;
    }
    rank[j] = a;
  }
}

extern "C" hl_status hl_set_hot(hl_handle* h, const uint32_t* hot_ids, uint32_t n_hot, hl_stream stream) {
  if (!h || (n_hot && !hot_ids)) return HL_ERR_INVALID_ARG;
  if (n_hot > h->k_cap || n_hot > h->n_rows) return HL_ERR_OUT_OF_RANGE;
  hipStream_t s = (hipStream_t)stream;
  const uint64_t tiles = h->n_tiles4k;
  hl_status st = hl_fill32((uint32_t*)h->d_bitmap, tiles * 128, 0, s);
  if (st != HL_OK) return st;
  if (n_hot) {
    uint32_t g = hl_div_up(n_hot, 256);
    if (g > 4096) g = 4096;
    HL_KERNEL(h, s, "sh_bits", sh_bits, dim3(g), dim3(256), 0, s, hot_ids, n_hot, h->n_rows, h->d_bitmap, h->d_err);
  }
  const uint64_t ne = tiles * 16 + 1;
  uint32_t g2 = hl_div_up(ne, 256);
  if (g2 > 4096) g2 = 4096;
  HL_KERNEL(h, s, "sh_rank", sh_rank, dim3(g2), dim3(256), 0, s, hot_ids, n_hot, ne, h->d_rank);
  HL_LAUNCHED();
  HL_TRY_ST(hl_table_bounds(h, s));
  h->n_hot = n_hot;
  return HL_OK;
}
