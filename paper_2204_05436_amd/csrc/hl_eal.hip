// The Embedding Access Logger with SRRIP replacement (Sec. V-B): instead of a
// counter per row, a set-associative cache of row ids with a 2-bit
// re-reference prediction value (RRPV) per way.  Id g lives in set
// mix(g) % n_sets (mix: the 32-bit finalizer of MurmurHash3); a hit sets its
// RRPV to 0; a miss takes the first way whose RRPV is 3, ageing the set by one
// until one is, and enters with RRPV 2.  Empty ways hold 0xFFFFFFFF and RRPV 3.
// The hot set the logger yields is every id it holds, ascending.
//
// Sets are independent, so the stream-order semantics hold per set: a batch's
// (set, id) pairs are sorted by set with the library's stable radix sort
// (ties keep lookup order), and the first thread of each set's run replays
// the run in order on the set's ways held in registers.
#include "hl_internal.h"

#define EAL_MAX_WAYS 16
#define EAL_EMPTY 0xFFFFFFFFu

struct hl_eal {
  hl_handle* h;
  uint32_t n_sets;
  int32_t ways;
  int64_t max_n;    // lookups per call
  uint32_t* tag;    // [n_sets * ways]
  uint8_t* rrpv;    // [n_sets * ways]
  uint32_t* cnt;    // [1] held ids (extraction)
  void* ws;         // sort workspace, zero-filled once
  size_t ws_bytes;
  uint32_t sort_n;  // the sort's capacity: max(max_n, n_sets * ways)
};

__device__ __forceinline__ uint32_t eal_mix(uint32_t x) {
  x ^= x >> 16;
  x *= 0x85EBCA6Bu;
  x ^= x >> 13;
  x *= 0xC2B2AE35u;
  x ^= x >> 16;
  return x;
}

__global__ void eal_init(uint32_t* tag, uint8_t* rrpv, uint64_t m) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m; i += (uint64_t)gridDim.x * blockDim.x) {
    tag[i] = EAL_EMPTY;
    rrpv[i] = 3;
  }
}

// (set, id) of every lookup; an invalid id (0xFFFFFFFF) gets the key n_sets,
// which sorts after every set and is skipped
__global__ void eal_keys(const uint32_t* __restrict__ gids, uint32_t n, uint32_t n_sets, uint32_t* __restrict__ keys,
                         uint32_t* __restrict__ vals) {
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    const uint32_t g = gids[i];
    keys[i] = g == EAL_EMPTY ? n_sets : eal_mix(g) % n_sets;
    vals[i] = g;
  }
}

// The head of each run of one set replays the run: ways in registers, every
// index into them a compile-time constant (no per-lane scratch).
__global__ void __launch_bounds__(256)
eal_runs(const uint32_t* __restrict__ keys, const uint32_t* __restrict__ vals, uint32_t n, uint32_t n_sets,
         int32_t ways, uint32_t* __restrict__ tag, uint8_t* __restrict__ rrpv) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint32_t s = keys[i];
  if (s >= n_sets || (i > 0 && keys[i - 1] == s)) return;
  uint32_t t[EAL_MAX_WAYS], r[EAL_MAX_WAYS];
#pragma unroll
  for (int w = 0; w < EAL_MAX_WAYS; ++w) {
    t[w] = w < ways ? tag[(uint64_t)s * ways + w] : EAL_EMPTY;
    r[w] = w < ways ? rrpv[(uint64_t)s * ways + w] : 0u;  // ways beyond the set never match nor reach 3 first
  }
  for (uint32_t p = i; p < n && keys[p] == s; ++p) {
    const uint32_t g = vals[p];
    bool hit = false;
#pragma unroll
    for (int w = 0; w < EAL_MAX_WAYS; ++w)
      if (w < ways && t[w] == g) {
        r[w] = 0;
        hit = true;
      }
    if (hit) continue;
    for (int age = 0; age < 4; ++age) {  // at most three ageings make some way 3
      int v = -1;
#pragma unroll
      for (int w = EAL_MAX_WAYS - 1; w >= 0; --w)
        if (w < ways && r[w] == 3) v = w;
      if (v >= 0) {
#pragma unroll
        for (int w = 0; w < EAL_MAX_WAYS; ++w)
          if (w == v) {
            t[w] = g;
            r[w] = 2;
          }
        break;
      }
#pragma unroll
      for (int w = 0; w < EAL_MAX_WAYS; ++w)
        if (w < ways) ++r[w];
    }
  }
#pragma unroll
  for (int w = 0; w < EAL_MAX_WAYS; ++w)
    if (w < ways) {
      tag[(uint64_t)s * ways + w] = t[w];
      rrpv[(uint64_t)s * ways + w] = (uint8_t)r[w];
    }
}

__global__ void eal_compact(const uint32_t* __restrict__ tag, uint64_t m, uint32_t* __restrict__ out,
                            uint32_t* __restrict__ vals, uint32_t* cnt) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m; i += (uint64_t)gridDim.x * blockDim.x) {
    const uint32_t g = tag[i];
    if (g != EAL_EMPTY) {
      const uint32_t k = atomicAdd(cnt, 1u);
      out[k] = g;
      vals[k] = g;
    }
  }
}

static uint32_t eal_grid(uint64_t n) {
  uint64_t b = (n + 255) / 256;
  return (uint32_t)(b < 1 ? 1 : (b > 4096 ? 4096 : b));
}

extern "C" hl_status hl_eal_destroy(hl_eal* e) {
  if (!e) return HL_ERR_INVALID_ARG;
  hl_status st = HL_OK;
  for (void* p : {(void*)e->tag, (void*)e->rrpv, (void*)e->cnt, e->ws})
    if (p && hipFree(p) != hipSuccess) st = HL_ERR_HIP;
  delete e;
  return st;
}

extern "C" hl_status hl_eal_reset(hl_eal* e, hl_stream stream) {
  if (!e) return HL_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  const uint64_t m = (uint64_t)e->n_sets * e->ways;
  HL_KERNEL(e->h, s, "eal_init", eal_init, dim3(eal_grid(m)), dim3(256), 0, s, e->tag, e->rrpv, m);
  HL_LAUNCHED();
  return HL_OK;
}

extern "C" hl_status hl_eal_create(hl_handle* h, uint32_t n_sets, int32_t ways, int64_t max_lookups, hl_eal** out) {
  if (!h || !out || n_sets < 1 || ways < 1 || ways > EAL_MAX_WAYS || max_lookups < 0) return HL_ERR_INVALID_ARG;
  const uint64_t m = (uint64_t)n_sets * ways;
  if (m >= (1ull << 30) || max_lookups >= (1ll << 30)) return HL_ERR_UNSUPPORTED;
  hl_eal* e = new hl_eal();
  e->h = h;
  e->n_sets = n_sets;
  e->ways = ways;
  e->max_n = max_lookups;
  e->sort_n = (uint32_t)((uint64_t)max_lookups > m ? (uint64_t)max_lookups : m);
  hl_carver c = hl_carver::after_header(nullptr, 0);
  hl_sort_ws sw;
  hl_sort_ws_carve(c, sw, e->sort_n);
  e->ws_bytes = c.off;
  hl_status st = HL_OK;
  if (hipMalloc(&e->tag, m * 4) != hipSuccess || hipMalloc(&e->rrpv, m) != hipSuccess ||
      hipMalloc(&e->cnt, 4) != hipSuccess || hipMalloc(&e->ws, e->ws_bytes) != hipSuccess ||
      hipMemset(e->ws, 0, e->ws_bytes) != hipSuccess)
    st = HL_ERR_HIP;
  if (st == HL_OK) st = hl_eal_reset(e, nullptr);
  if (st == HL_OK && hipDeviceSynchronize() != hipSuccess) st = HL_ERR_HIP;
  if (st != HL_OK) {
    hl_eal_destroy(e);
    return st;
  }
  *out = e;
  return HL_OK;
}

extern "C" hl_status hl_eal_access(hl_eal* e, const uint32_t* gids, int64_t n, hl_stream stream) {
  if (!e || n < 0 || (n > 0 && !gids)) return HL_ERR_INVALID_ARG;
  if (n > e->max_n) return HL_ERR_CAPACITY;
  if (n == 0) return HL_OK;
  hipStream_t s = (hipStream_t)stream;
  hl_carver c = hl_carver::after_header(e->ws, e->ws_bytes);
  hl_sort_ws sw;
  hl_sort_ws_carve(c, sw, e->sort_n);
  const uint32_t nn = (uint32_t)n;
  HL_KERNEL(e->h, s, "eal_keys", eal_keys, dim3(eal_grid(nn)), dim3(256), 0, s, gids, nn, e->n_sets, sw.k0, sw.v0);
  HL_LAUNCHED();
  uint32_t *sk, *sv;
  hl_status st = hl_sort_pairs(e->h, sw, nullptr, nn, hl_bit_width(e->n_sets), s, &sk, &sv);
  if (st != HL_OK) return st;
  HL_KERNEL(e->h, s, "eal_runs", eal_runs, dim3(hl_div_up(nn, 256)), dim3(256), 0, s, sk, sv, nn, e->n_sets, e->ways,
            e->tag, e->rrpv);
  HL_LAUNCHED();
  return HL_OK;
}

extern "C" hl_status hl_eal_hot(hl_eal* e, uint32_t* hot_ids_out, uint32_t* n_hot_out, hl_stream stream) {
  if (!e || !hot_ids_out || !n_hot_out) return HL_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  const uint64_t m = (uint64_t)e->n_sets * e->ways;
  hl_carver c = hl_carver::after_header(e->ws, e->ws_bytes);
  hl_sort_ws sw;
  hl_sort_ws_carve(c, sw, e->sort_n);
  HL_HIP(hipMemsetAsync(e->cnt, 0, 4, s));
  HL_KERNEL(e->h, s, "eal_compact", eal_compact, dim3(eal_grid(m)), dim3(256), 0, s, e->tag, m, sw.k0, sw.v0, e->cnt);
  HL_LAUNCHED();
  uint32_t *sk, *sv;
  hl_status st = hl_sort_pairs(e->h, sw, e->cnt, (uint32_t)m, hl_bit_width(e->h->n_rows), s, &sk, &sv);
  if (st != HL_OK) return st;
  uint32_t n = 0;
  HL_HIP(hipMemcpyAsync(&n, e->cnt, 4, hipMemcpyDeviceToHost, s));
  HL_HIP(hipStreamSynchronize(s));
  if (n) HL_HIP(hipMemcpy(hot_ids_out, sk, (size_t)n * 4, hipMemcpyDeviceToDevice));
  *n_hot_out = n;
  return HL_OK;
}

extern "C" hl_status hl_eal_state(const hl_eal* e, uint32_t* tags_out, uint8_t* rrpv_out, hl_stream stream) {
  if (!e || !tags_out || !rrpv_out) return HL_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  const uint64_t m = (uint64_t)e->n_sets * e->ways;
  HL_HIP(hipMemcpyAsync(tags_out, e->tag, m * 4, hipMemcpyDeviceToDevice, s));
  HL_HIP(hipMemcpyAsync(rrpv_out, e->rrpv, m, hipMemcpyDeviceToDevice, s));
  return HL_OK;
}
