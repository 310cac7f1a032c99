// Internal declarations shared by the HIP sources of libhotline (not installed).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/hotline.h"

#define HL_WAVE 64

// ----------------------------------------------------------------------------- tracing
struct hl_trace_rec {
  const char* name;
  hipEvent_t a, b;
};
struct hl_trace {
  int32_t cap = 0, n = 0;
  hl_trace_rec* rec = nullptr;
  char only[256] = {0};  // record only kernels of these comma-separated names (empty: all)
};
// A record for kernel `name` (its two events in *a, *b), or -1 when none is
// taken (tracing off, full, or another name selected).
int hl_trace_take(const struct hl_handle* h, const char* name, hipEvent_t* a, hipEvent_t* b);
// A kernel launch; when traced, through the launch that has the dispatch
// itself record its start and end in the record's events (the kernel's own
// duration: no marker packets before and after it on the stream).
template <typename F, typename... A>
static inline void hl_launch(const struct hl_handle* h, const char* name, F kernel, dim3 grid, dim3 block,
                             uint32_t shmem, hipStream_t s, A... args) {
  hipEvent_t a, b;
  if (hl_trace_take(h, name, &a, &b) >= 0)
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, a, b, 0u, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, shmem, s, args...);
}
#define HL_KERNEL(h, s, name, ...) hl_launch((h), (name), __VA_ARGS__)

// ----------------------------------------------------------------------------- handle
// A workspace holding a backward plan (grouping) for a later apply step.
struct hl_ws_rec {
  const void* ws;      // NULL: free
  int64_t n, bags;     // the plan's lookups and bags
  int32_t stg;         // its staging rows
  int part1;           // the first half of the apply ran on it (3: without its spanning segments)
  int vec;             // the row vector width that half used (its tile layout depends on it)
  int compact;         // the plan used the layout without the staging-row sums (whole applies only)
};
struct hl_handle {
  int device;
  int32_t n_tables;
  uint64_t n_rows;
  int32_t dim;
  hl_dtype dtype;
  uint32_t k_cap;
  uint32_t row_bytes;
  uint32_t n_hot;
  uint64_t n_tiles4k;    // ceil(n_rows / 4096): the bitmap and rank directory cover n_tiles4k*4096 ids
  uint32_t* d_base;      // [n_tables] first gid of each table
  uint32_t* d_rows;      // [n_tables] rows of each table
  uint32_t* d_counts;    // [n_rows] access counts
  uint64_t* d_bitmap;    // [n_tiles4k*64] hot-set membership, bit g of word g/64
  uint32_t* d_rank;      // [n_tiles4k*16 + 1] hot ids below 256*j
  uint32_t* d_tb;        // [n_tables + 1] hot ids below each table's first row (the last: n_hot)
  uint32_t* d_err;       // device error word
  uint32_t* d_tk;        // top-K scratch (state, histograms, tile counts)
  size_t tk_bytes;
  hl_trace* trace;       // per-kernel event records (owned)
  // Workspaces that hold a backward plan (grouping) for a later apply step;
  // any other call on a workspace clears its record.
  int ballot_ranks;      // the sorts rank every pass by ballots (hl_debug_ballot_ranks)
  hl_ws_rec ws_rec[4];
  int ws_next;           // next record to reuse when all are taken
  uint64_t* cg_table;    // cold-gather hash table (kept clean between calls)
  uint32_t cg_slots;     // its slots
  mutable struct hl_hook {  // a handover for the next kernel that takes one (hl_hook_take)
    uint32_t* sflag;
    uint32_t sv;
    const uint32_t* wflag;   // waits: wflag >= wv, then w2flag >= w2v
    uint32_t wv;
    const uint32_t* w2flag;
    uint32_t w2v;
    uint32_t gate;           // the waits are every block's, at the kernel's start (hl_hook_gate)
    uint32_t* err;
  } hook;
};
typedef hl_handle::hl_hook hl_hook;
// The pending handover, cleared: the kernel about to launch carries it.
static inline hl_hook hl_hook_take(const hl_handle* h) {
  const hl_hook k = h->hook;
  h->hook = hl_hook{};
  return k;
}
#define HL_WSK_OTHER 1
#define HL_WSK_BWD_PLAN 2
static inline void hl_ws_note(hl_handle* h, const void* ws, int kind, int64_t n = 0, int64_t bags = 0,
                              int32_t stg = 0) {
  for (auto& r : h->ws_rec)
    if (r.ws == ws) r.ws = nullptr;
  if (kind != HL_WSK_BWD_PLAN) return;
  hl_ws_rec* r = nullptr;
  for (auto& c : h->ws_rec)
    if (!c.ws && !r) r = &c;
  if (!r) {  // more plans than records: the oldest is forgotten
    r = &h->ws_rec[h->ws_next];
    h->ws_next = (h->ws_next + 1) % 4;
  }
  *r = {ws, n, bags, stg, 0};
}
static inline hl_ws_rec* hl_ws_find(hl_handle* h, const void* ws) {
  for (auto& r : h->ws_rec)
    if (ws && r.ws == ws) return &r;
  return nullptr;
}

// n / d and n % d for 0 <= n < 2^22, d >= 1, with inv = 1.0f / d: the float
// quotient is off by at most one, and the remainder check corrects it (no
// integer division, which takes tens of instructions).
__device__ __forceinline__ uint32_t hl_fdiv(uint32_t n, uint32_t d, float inv, uint32_t* rem) {
  uint32_t q = (uint32_t)((float)n * inv);
  int32_t r = (int32_t)(n - q * d);
  if (r < 0) {
    --q;
    r += (int32_t)d;
  } else if (r >= (int32_t)d) {
    ++q;
    r -= (int32_t)d;
  }
  *rem = (uint32_t)r;
  return q;
}

// ----------------------------------------------------------------------------- errors
#define HL_HIP(call)                                   \
  do {                                                 \
    hipError_t _e = (call);                            \
    if (_e != hipSuccess) return HL_ERR_HIP;           \
  } while (0)

#define HL_LAUNCHED()                                  \
  do {                                                 \
    if (hipGetLastError() != hipSuccess) return HL_ERR_HIP; \
  } while (0)

__device__ __forceinline__ void hl_flag(uint32_t* err, uint32_t bit) { atomicOr(err, bit); }

// The lanes of the wave whose `bits`-bit digit equals this lane's, among the
// lanes where `valid` holds (0 on a lane where it does not): one ballot per
// digit bit, each keeping the lanes that agree on that bit.
__device__ __forceinline__ uint64_t hl_match_digit(uint32_t digit, int bits, bool valid) {
  uint64_t m = __ballot(valid);
  for (int b = 0; b < bits; ++b) {
    const bool one = (digit >> b) & 1u;
    const uint64_t ones = __ballot(one);
    m &= one ? ones : ~ones;
  }
  return valid ? m : 0ull;
}

// ----------------------------------------------------------------------------- hot set probes
// Membership: bit (g & 63) of word g >> 6.  Rank: rank[g >> 8] counts hot ids
// below the 256-id block; the block's 4 words before g's word and the bits of
// g's word below g add the rest.
__device__ __forceinline__ bool hl_is_hot(const uint64_t* __restrict__ bm, uint32_t g) {
  return (bm[g >> 6] >> (g & 63)) & 1ull;
}

__device__ __forceinline__ int32_t hl_hot_slot(const uint64_t* __restrict__ bm,
                                               const uint32_t* __restrict__ rank, uint32_t g) {
  const uint32_t blk = g >> 8;
  const ulonglong2* p = reinterpret_cast<const ulonglong2*>(bm + (size_t)blk * 4);
  // the rank word is loaded with the bitmap words, not after the membership test
  ulonglong2 a = p[0], b = p[1];
  uint32_t r = rank[blk];
  uint64_t w[4] = {a.x, a.y, b.x, b.y};
  const uint32_t wi = (g >> 6) & 3, bit = g & 63;
  uint64_t word = w[wi];
  if (!((word >> bit) & 1ull)) return -1;
#pragma unroll
  for (uint32_t k = 0; k < 3; ++k)
    if (k < wi) r += __popcll(w[k]);
  r += __popcll(word & ((1ull << bit) - 1ull));
  return (int32_t)r;
}

// ----------------------------------------------------------------------------- workspace
// Every workspace starts with a fixed header of self-resetting counters (their
// place must not depend on the sizes of a call); buffers are carved after it
// with 256-byte alignment.
#define HL_WS_HEADER 16384
#define HL_HDR_SORT 0    // 8 words: per-pass tile counters
#define HL_HDR_COLD 16   // 16 words: cold-gather counters
#define HL_HDR_DISP 64   // 8 words: dispatch epoch, done counter, tile counter
#define HL_HDR_DSTAT 128 // dispatch look-back status words (64-bit), to the header's end
#define HL_DISP_MAX_TILES ((HL_WS_HEADER - 4 * HL_HDR_DSTAT) / 8)
// Workspace carving with 256-byte alignment.
struct hl_carver {
  char* base;
  size_t off, cap;
  static hl_carver after_header(void* ws, size_t bytes) { return hl_carver{(char*)ws, HL_WS_HEADER, bytes}; }
  uint32_t* header() const { return reinterpret_cast<uint32_t*>(base); }
  template <class T>
  T* take(size_t count) {
    off = (off + 255) & ~(size_t)255;
    T* p = reinterpret_cast<T*>(base ? base + off : nullptr);
    off += count * sizeof(T);
    return p;
  }
};

// The cold half of the forward (hl_embbag_fwd_part 2 over the non-popular
// mu-batch) read from the backward's grouping held in `workspace`: the same
// sums, over the cold lookups only.  Needs a plan over every sample and the
// first apply half (which marks where the cold keys start) on that workspace.
hl_status hl_embbag_fwd_cold_sorted(hl_handle* h, const void* staging, int32_t stg_rows, const int32_t* codes,
                                    const int32_t* bag_ptr, int32_t n_samples, int32_t bps, int64_t n_lookups,
                                    float* out, void* workspace, size_t ws_bytes, hl_stream stream);

// hl_embbag_bwd_apply_part with one more part: 3, the first half without the
// segments that span tiles, which hl_embbag_finish_cold then completes.
hl_status hl_embbag_bwd_apply_any(hl_handle* h, void* w_hot, void* staging, int32_t stg_rows, int32_t n_samples,
                                  int32_t bps, int64_t n_lookups, const float* dY, float lr, int32_t part,
                                  void* workspace, size_t ws_bytes, hl_stream stream);
// After part 3, once the staging rows are fetched: the cold half of the
// forward (as hl_embbag_fwd_cold_sorted) with part 3's spanning segments in one
// launch, then the staging-row updates (as part 2).
hl_status hl_embbag_finish_cold(hl_handle* h, void* w_hot, void* staging, int32_t stg_rows, const int32_t* codes,
                                const int32_t* bag_ptr, int32_t n_samples, int32_t bps, int64_t n_lookups, float lr,
                                float* out, void* workspace, size_t ws_bytes, hl_stream stream);
// hl_dispatch takes the fused single-kernel path (its kernel takes a hook)
bool hl_dispatch_fused(const hl_handle* h, int32_t n_samples, int32_t bps, int64_t n_lookups, const void* workspace,
                       size_t ws_bytes);

// ---------------------------------------------------------- the fused plan
// A look-ahead plan over every sample in five launches instead of seven: the
// dispatch kernel also enters its cold lookups into the cold-gather hash table
// (the cold plan's insert), the rank scan writes the cold id list itself, and
// the grouping's first kernel also points the cold lookups' codes at their
// staging rows and frees their table slots (the cold plan's last kernel).  The
// cold plan's state lies after the grouping's region of the workspace, so the
// grouping can read it.
struct hl_cg_fused {
  uint64_t* table;        // the handle's hash table (NULL: no fused cold plan)
  uint32_t S;             // its slots (a power of two)
  uint32_t* slotof;       // [n] slot of a cold lookup
  uint32_t* uidx;         // [S] staging row of the id in a slot
  uint64_t* rstat;        // [rtiles] the rank scan's look-back status (cleared by the dispatch)
  uint32_t rtiles;
  const uint32_t* ncold;  // distinct cold ids (written by the rank scan)
  int32_t cap;            // staging rows
};
// The backward's sort key of a slot code: the hot slot, or n_hot + staging
// row; any other code (an invalid one, or -1) gets EB_SENT, which the
// reduction skips.
#define EB_SENT 0xFFFFFFFFu
__device__ __forceinline__ uint32_t bw_key(uint32_t c, uint32_t n_hot, uint32_t k_cap, int32_t stg_rows) {
  if (c < n_hot) return c;
  if (c >= k_cap && c - k_cap < (uint32_t)stg_rows) return n_hot + (c - k_cap);
  return EB_SENT;
}
// The fused plan: a cold lookup's code (-1) points at its staging row once the
// rank scan numbered the rows, if they fit; any other code is returned as is.
__device__ __forceinline__ int32_t bw_fused_code(int32_t c, uint32_t i, const hl_cg_fused& cf, uint32_t k_cap,
                                                 bool fits) {
  if (c != -1 || !cf.table) return c;
  const uint32_t sl = cf.slotof[i];
  return sl < cf.S && fits ? (int32_t)(k_cap + cf.uidx[sl]) : -1;
}
// A kernel starts only once the kernels before it on its stream are complete
// and their writes visible: a store at its start is a handover signal for
// them (block 0 makes it, with release order at agent scope).
__device__ __forceinline__ void bw_start_signal(uint32_t* sflag, uint32_t sv) {
  if (sflag && blockIdx.x == 0 && threadIdx.x == 0)
    __hip_atomic_store(sflag, sv, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}
// d_tb of the current hot set (after the bitmap and the rank directory)
hl_status hl_table_bounds(hl_handle* h, hipStream_t s);
// Hot ids below row id g (g < n_rows): the rank directory's count for g's
// 256-id block plus the bitmap bits of that block below g.
__device__ __forceinline__ uint32_t hl_hot_below(const uint64_t* __restrict__ bm, const uint32_t* __restrict__ rank,
                                                 uint32_t g) {
  const uint32_t blk = g >> 8, wi = (g >> 6) & 3, bit = g & 63;
  uint32_t r = rank[blk];
  for (uint32_t k = 0; k < wi; ++k) r += __popcll(bm[(size_t)blk * 4 + k]);
  return r + __popcll(bm[(size_t)blk * 4 + wi] & ((1ull << bit) - 1ull));
}

// workspace bytes of the backward's plan and apply
size_t hl_bwd_ws_bytes(const hl_handle* h, int64_t max_lookups, int64_t max_bags);
// the same without the staging-row sums that the applies in halves keep
// (enough for a plan followed by a whole apply)
size_t hl_bwd_ws_bytes_compact(const hl_handle* h, int64_t max_lookups, int64_t max_bags);
// the allocation-free backward's static workspace: its device address on
// `device` is looked up (and the array zero-filled) once, with that device
// current; hl_create does it for the handle's device
hl_status hl_scratch_setup(int device);
// workspace bytes of the fused plan (hl_workspace_bytes covers them)
size_t hl_plan_ws_bytes(const hl_handle* h, int64_t max_lookups, int64_t max_bags, int32_t max_samples);
// carves the fused plan's cold state; HL_ERR_CAPACITY if the workspace or the
// handle's hash table is too small (a plain cold plan grows the table)
hl_status hl_cold_fused_begin(hl_handle* h, int64_t n_lookups, int64_t n_bags, int32_t n_samples, int32_t cap,
                              void* workspace, size_t ws_bytes, hipStream_t s, hl_cg_fused* out);
// hl_dispatch whose kernel also inserts the cold lookups (cf: from hl_cold_fused_begin)
hl_status hl_dispatch_ex(hl_handle* h, const uint32_t* rows, const int32_t* bag_ptr, int32_t n_samples, int32_t bps,
                         int64_t n_lookups, uint32_t* gids, int32_t* codes, uint8_t* flags, int32_t* pop_ids,
                         int32_t* nonpop_ids, int32_t* counts_dev, void* workspace, size_t ws_bytes,
                         hl_stream stream, const hl_cg_fused* cf);
// the rank scan of the fused plan: staging rows by first occurrence, the cold
// id list (ids of staging rows below cap) and its count
hl_status hl_cold_rank_fused(hl_handle* h, const uint32_t* gids, const int32_t* codes, int64_t n_lookups,
                             uint32_t* cold_ids, int32_t* n_cold_dev, void* workspace, const hl_cg_fused& cf,
                             hipStream_t s);

// the cold-gather hash table: open addressing keyed by row id, a slot holds
// (id + 1) << 32 | the smallest lookup index of that id (0 = empty)
__device__ __forceinline__ uint32_t hl_cg_hash(uint32_t x) {  // 32-bit finalising mix
  x ^= x >> 16;
  x *= 0x85EBCA6Bu;
  x ^= x >> 13;
  x *= 0xC2B2AE35u;
  x ^= x >> 16;
  return x;
}
// enters id g of lookup i; returns its slot
__device__ __forceinline__ uint32_t hl_cg_insert(uint64_t* table, uint32_t smask, uint32_t g, uint32_t i) {
  const uint64_t want = ((uint64_t)(g + 1) << 32) | i;
  uint32_t slot = hl_cg_hash(g) & smask;
  for (uint32_t probe = 0; probe <= smask; ++probe) {
    const uint64_t prev = atomicCAS((unsigned long long*)(table + slot), 0ull, (unsigned long long)want);
    if (prev == 0) break;
    if ((uint32_t)(prev >> 32) == g + 1) {
      atomicMin((unsigned long long*)(table + slot), (unsigned long long)want);
      break;
    }
    slot = (slot + 1) & smask;
  }
  return slot;
}
// hl_embbag_bwd_plan whose first kernel, when it launches one (*sent), also
// stores sv into *sflag as it starts: a handover signal for the kernels
// enqueued before it on the stream.
hl_status hl_embbag_bwd_plan_signal(hl_handle* h, int32_t stg_rows, int32_t* codes, const int32_t* bag_ptr,
                                    int32_t n_samples, int32_t bps, int64_t n_lookups, const int32_t* sample_ids,
                                    const int32_t* n_sel_dev, int32_t n_sel_max, void* workspace, size_t ws_bytes,
                                    hl_stream stream, uint32_t* sflag, uint32_t sv, bool* sent,
                                    const hl_cg_fused* cf, bool compact = false);

// ----------------------------------------------------------------------------- grouping by table
// The backward's grouping of a one-hot mini-batch table by table (hl_group.hip):
// taken when every bag holds one lookup (n_lookups = n_bags, checked per bag
// on the device: HL_DEVERR_SHAPE otherwise), the bags split evenly over at
// most 64 tables and a table has at most 8192 bags.  k_tm: scratch of n_bags
// keys; cum: scratch of n_bags words (the prep blocks' hot counts, at most
// ceil(E / 32) (T + 1) of them); kout/vout: the grouping.
bool hl_group_by_table_ok(const hl_handle* h, int64_t n_lookups, int64_t n_bags);
// The grouping's first launch alone (gt_prep); returns its block count, which
// the sort takes (hl_group_sort.h: gt_sort_body).
uint32_t hl_group_prep(hl_handle* h, int32_t* codes, const int32_t* bag_ptr, int64_t n_bags, int32_t stg_rows,
                       uint32_t* k_tm, uint32_t* cum, uint32_t* sflag, uint32_t sv, const hl_cg_fused* cf,
                       hipStream_t s);
hl_status hl_group_by_table(hl_handle* h, int32_t* codes, const int32_t* bag_ptr, int64_t n_bags, int32_t stg_rows,
                            uint32_t* k_tm, uint32_t* cum, uint32_t* kout, uint32_t* vout, uint32_t* sflag,
                            uint32_t sv, const hl_cg_fused* cf, hipStream_t s);

// ----------------------------------------------------------------------------- sort
// Stable LSD radix sort of (key, value) uint32 pairs with digits of up to 11
// bits: one histogram kernel plus one kernel per digit with decoupled look-back
// for the cross-tile digit offsets.  See hl_sort.hip.
#define HL_SORT_THREADS 512
#define HL_SORT_WAVES (HL_SORT_THREADS / 64)
// items per thread of a pass block: 4, 6 or 12 (the fewest that keep the
// tiles to HL_SORT_TILES_AIM and to the stream's compute units, so a small
// sort still spreads over the units it has, in one round of blocks)
#define HL_SORT_TILE_MIN (HL_SORT_THREADS * 4)
#define HL_SORT_TILE_MAX (HL_SORT_THREADS * 12)
#define HL_SORT_TILES_AIM 128
#define HL_SORT_MAXNB 2048        // bins of an 11-bit digit
#define HL_SORT_MAXPASS 3
#define HL_SORT_HIST_BLOCKS 16
#define HL_SORT_HIST_THREADS 1024
struct hl_sort_ws {
  uint32_t *k0, *v0, *k1, *v1;  // ping-pong buffers, n_max each; input in k0/v0
  uint32_t* part;               // [HL_SORT_MAXPASS][HL_SORT_HIST_BLOCKS][HL_SORT_MAXNB] per-block digit counts
  uint32_t* st[2];              // [tiles_max][HL_SORT_MAXNB] look-back status, alternating between passes
  uint32_t* ctr;                // [8] self-resetting tile counters (in the workspace header)
  uint32_t tiles_max;
  uint32_t n_max;
};

void hl_sort_ws_carve(hl_carver& c, hl_sort_ws& ws, uint32_t n_max);
// Sorts ws.k0/ws.v0 (first *n_dev items if n_dev != NULL, else n_host) by the
// low `bits` bits of the key; returns in *out_k/*out_v the buffers holding the
// result.  Keys must be < 2^bits - 1 except the all-ones sentinel, which sorts
// last.
hl_status hl_sort_pairs(hl_handle* h, hl_sort_ws& ws, const uint32_t* n_dev, uint32_t n_host,
                        int bits, hipStream_t s, uint32_t** out_k, uint32_t** out_v);
// The buffers hl_sort_pairs leaves its result in for a sort of `bits` bits
// with n_host > 0.
void hl_sort_result(const hl_sort_ws& ws, int bits, uint32_t** out_k, uint32_t** out_v);
// A producer of the keys may count their digits itself (in the same launch
// that writes them) and then run only the digit passes.  Geometry of a sort
// of n_host items and `bits` bits: `passes` digits of `b` bits, nb bins,
// hist_blocks partial counts per pass (ws.part[(p * HL_SORT_HIST_BLOCKS +
// block) * nb + digit], digit p = (key >> (b * p)) & ((1 << b) - 1)), and the
// first pass's status words ws.st[0][0 .. n_zero) to clear.
struct hl_sort_geom {
  int passes, b, nb;
  int items;      // per thread of a pass block
  uint32_t tile;  // items per pass block
  uint32_t hist_blocks;
  uint64_t n_zero;
};
// cus: compute units of the stream the sort runs on (its mask; 0: unknown),
// which cap the tiles (one pass block per unit)
hl_sort_geom hl_sort_geometry(uint32_t n_host, int bits, int cus);
// Compute units in a stream's mask (0 if it cannot be read).
int hl_stream_cus(hipStream_t s);
// The digit passes of hl_sort_pairs, once the counts and the cleared status
// words are in place (hl_sort_geometry); same contract otherwise.
hl_status hl_sort_passes(hl_handle* h, hl_sort_ws& ws, const uint32_t* n_dev, uint32_t n_host, int bits,
                         hipStream_t s, uint32_t** out_k, uint32_t** out_v);

// Decoupled look-back helpers (epoch-tagged 64-bit status words).  A status
// word carries its own value, so relaxed agent-scope atomics suffice: no other
// data is published through it.
#define HL_ST_AGG 1ull
#define HL_ST_PRE 2ull
#define HL_SPIN_LIMIT (1u << 24)

// A handover between streams carried by a kernel of the path instead of a
// launch of its own.  Block 0 stores sv into *sflag as the kernel starts: the
// kernels before it on its stream are complete, and their writes were made
// visible when they ended, so a relaxed store publishes them.  Block 0 waits
// at its end until *wflag reaches wv: the kernel, and so its stream, ends only
// then, and the next kernel's start orders its reads after the wait (the
// relaxed loads need no acquire).  Bounded: past the limit the wait sets
// HL_DEVERR_STALL and returns.
__device__ __forceinline__ void hl_hook_head(const hl_hook& k) {
  if (k.sflag && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0)
    __hip_atomic_store(k.sflag, k.sv, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void hl_hook_spin(const uint32_t* f, uint32_t v, uint32_t* err) {
  if (!f) return;
  uint32_t spins = 0;
  // (int32_t)(x - v) >= 0: x has reached v (sequence numbers wrap)
  while ((int32_t)(__hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) - v) < 0) {
    if (++spins > HL_SPIN_LIMIT) {
      hl_flag(err, HL_DEVERR_STALL);
      return;
    }
    __builtin_amdgcn_s_sleep(8);
  }
}
__device__ __forceinline__ void hl_hook_tail(const hl_hook& k) {
  if (k.gate || blockIdx.x != 0 || blockIdx.y != 0 || threadIdx.x != 0) return;
  hl_hook_spin(k.wflag, k.wv, k.err);
  hl_hook_spin(k.w2flag, k.w2v, k.err);
}
// A gate: thread 0 of every block waits before the block starts (the caller
// synchronizes the block after it).  Only for handovers that order this
// kernel's writes after other kernels' reads and writes (nothing this kernel
// reads comes through them): the waits end inside the kernel, after its start
// made earlier writes visible.
__device__ __forceinline__ void hl_hook_gate(const hl_hook& k) {
  if (!k.gate || threadIdx.x != 0) return;
  hl_hook_spin(k.wflag, k.wv, k.err);
  hl_hook_spin(k.w2flag, k.w2v, k.err);
}
#ifndef HL_LB_WIN
#define HL_LB_WIN 32
#endif

__device__ __forceinline__ uint64_t hl_st_pack(uint32_t epoch, uint64_t flag, uint32_t v) {
  return ((uint64_t)epoch << 32) | (flag << 30) | (uint64_t)(v & 0x3FFFFFFFu);
}
__device__ __forceinline__ void hl_st_store(uint64_t* p, uint64_t w) {
  __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t hl_st_load(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Exclusive prefix of tile `tile`'s value over tiles [0, tile) for one lane of
// status words laid out with stride `stride` between tiles.  Reads a window of
// HL_LB_WIN predecessors per round trip.
__device__ __forceinline__ uint32_t hl_lookback(const uint64_t* st, uint32_t tile, size_t stride,
                                                uint32_t epoch, uint32_t* err) {
  uint32_t excl = 0;
  int64_t j = (int64_t)tile - 1;
  uint32_t spins = 0;
  while (j >= 0) {
    uint64_t w[HL_LB_WIN];
#pragma unroll
    for (int k = 0; k < HL_LB_WIN; ++k) w[k] = (j - k >= 0) ? hl_st_load(st + (size_t)(j - k) * stride) : 0ull;
    int k = 0;
    bool stall = false;
#pragma unroll
    for (int q = 0; q < HL_LB_WIN; ++q) {
      if (stall || j - q < 0) continue;
      const uint32_t e = (uint32_t)(w[q] >> 32);
      const uint64_t f = (w[q] >> 30) & 3ull;
      if (e != epoch || f == 0) {
        stall = true;
        continue;
      }
      excl += (uint32_t)(w[q] & 0x3FFFFFFFu);
      if (f == HL_ST_PRE) return excl;
      k = q + 1;
    }
    j -= k;
    if (stall) {
      if (++spins > HL_SPIN_LIMIT) {
        hl_flag(err, HL_DEVERR_STALL);
        return excl;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  return excl;
}

// Exclusive prefix of `tile` over tiles [0, tile) from single-value status
// words (hl_st_pack), read by the whole block: thread t looks at tile j - t of
// the current window, so one round trip covers blockDim.x predecessors, and the
// walk stops at the nearest inclusive prefix.  Every thread of the block calls
// it (uniform control flow) and receives the result.
__device__ __forceinline__ uint32_t hl_block_lookback(const uint64_t* st, uint32_t tile, uint32_t epoch,
                                                      uint32_t* err) {
  __shared__ int s_first, s_first_pre;
  __shared__ uint32_t s_part[16];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, nw = (int)(blockDim.x >> 6);
  uint32_t excl = 0, spins = 0;
  int64_t j = (int64_t)tile - 1;
  while (j >= 0) {
    const int64_t p = j - tid;
    const uint64_t wd = p >= 0 ? hl_st_load(st + p) : hl_st_pack(epoch, HL_ST_PRE, 0);
    const uint32_t f = (uint32_t)((wd >> 30) & 3ull);
    const bool ok = (uint32_t)(wd >> 32) == epoch && f != 0;
    const bool stop = !ok || f == HL_ST_PRE;
    if (tid == 0) s_first = 0x7FFFFFFF;
    __syncthreads();
    const uint64_t sm = __ballot(stop);
    if (lane == 0 && sm) atomicMin(&s_first, w * 64 + __ffsll((unsigned long long)sm) - 1);
    __syncthreads();
    const int first = s_first;
    if (tid == first) s_first_pre = ok ? 1 : 0;
    __syncthreads();
    const bool none = first == 0x7FFFFFFF;
    const bool pre = !none && s_first_pre;
    const int use = none ? (int)blockDim.x : (pre ? first + 1 : first);  // words [0, use) are summed
    uint32_t v = tid < use ? (uint32_t)(wd & 0x3FFFFFFFu) : 0u;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    if (lane == 0) s_part[w] = v;
    __syncthreads();
    uint32_t tot = 0;
    for (int q = 0; q < nw; ++q) tot += s_part[q];
    __syncthreads();  // s_first, s_first_pre and s_part are reused
    excl += tot;
    if (pre) break;
    j -= use;
    if (!none) {  // an unpublished predecessor: wait for it
      if (++spins > HL_SPIN_LIMIT) {
        if (tid == 0) hl_flag(err, HL_DEVERR_STALL);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  return excl;
}

// ----------------------------------------------------------------------------- misc
static inline uint32_t hl_div_up(uint64_t a, uint64_t b) { return (uint32_t)((a + b - 1) / b); }
static inline int hl_bit_width(uint64_t x) {
  int b = 0;
  while (x) { ++b; x >>= 1; }
  return b;
}

// Row copy (bitwise) of n rows: dst[r] = src[ids[r]], rows of row_bytes; n is
// *n_dev (clamped to n_host) when n_dev is given.  Ids >= n_src_rows are
// skipped and flag HL_DEVERR_OUT_OF_RANGE.
hl_status hl_launch_gather(const hl_handle* h, const uint32_t* ids, const int32_t* n_dev, uint32_t n_host,
                           const void* src, uint64_t n_src_rows, void* dst, uint32_t row_bytes,
                           uint32_t* err, hipStream_t s);
hl_status hl_fill32(uint32_t* p, uint64_t n, uint32_t v, hipStream_t s);
