// Handle, workspace, errors, pinned host memory, address generation, access
// counting and the bitwise row gather.
#include <stdlib.h>
#include <string.h>

#include <vector>

#include <cstring>

#include "hl_internal.h"

size_t hl_topk_scratch_bytes(uint64_t n_rows);
size_t hl_partition_ws_bytes(int32_t max_samples);
size_t hl_cold_ws_bytes(const hl_handle* h, int64_t max_lookups, int64_t max_bags, int32_t max_samples);
size_t hl_bwd_ws_bytes(const hl_handle* h, int64_t max_lookups, int64_t max_bags);
size_t hl_plan_ws_bytes(const hl_handle* h, int64_t max_lookups, int64_t max_bags, int32_t max_samples);

extern "C" const char* hl_status_string(int32_t s) {
  switch (s) {
    case HL_OK: return "ok";
    case HL_ERR_INVALID_ARG: return "invalid argument";
    case HL_ERR_OUT_OF_RANGE: return "out of range";
    case HL_ERR_CAPACITY: return "capacity exceeded";
    case HL_ERR_HIP: return "HIP runtime error";
    case HL_ERR_UNSUPPORTED: return "unsupported";
    case HL_ERR_DEVICE: return "device error word set";
  }
  return "unknown status";
}

// ----------------------------------------------------------------------------- fill
__global__ void hl_k_fill32(uint32_t* p, uint64_t n, uint32_t v) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (uint64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

static hl_status fill32(uint32_t* p, uint64_t n, uint32_t v, hipStream_t s) {
  if (n == 0) return HL_OK;
  uint32_t g = hl_div_up(n, 256);
  if (g > 8192) g = 8192;
  hipLaunchKernelGGL(hl_k_fill32, dim3(g), dim3(256), 0, s, p, n, v);
  HL_LAUNCHED();
  return HL_OK;
}

hl_status hl_fill32(uint32_t* p, uint64_t n, uint32_t v, hipStream_t s) { return fill32(p, n, v, s); }

// ----------------------------------------------------------------------------- tracing
// name is one of the comma-separated names of list
static bool trace_listed(const char* list, const char* name) {
  const size_t n = strlen(name);
  for (const char* p = list; *p;) {
    const char* e = strchr(p, ',');
    const size_t m = e ? (size_t)(e - p) : strlen(p);
    if (m == n && strncmp(p, name, n) == 0) return true;
    if (!e) break;
    p = e + 1;
  }
  return false;
}

int hl_trace_take(const hl_handle* h, const char* name, hipEvent_t* a, hipEvent_t* b) {
  hl_trace* t = h ? h->trace : nullptr;
  if (!t || t->n >= t->cap) return -1;
  if (t->only[0] && !trace_listed(t->only, name)) return -1;
  const int i = t->n++;
  t->rec[i].name = name;
  *a = t->rec[i].a;
  *b = t->rec[i].b;
  return i;
}

static void trace_free(hl_trace* t) {
  for (int i = 0; i < t->cap; ++i) {
    (void)hipEventDestroy(t->rec[i].a);
    (void)hipEventDestroy(t->rec[i].b);
  }
  free(t->rec);
  t->rec = nullptr;
  t->cap = t->n = 0;
}

extern "C" hl_status hl_trace_enable(hl_handle* h, int32_t cap) {
  if (!h || cap < 0) return HL_ERR_INVALID_ARG;
  HL_HIP(hipDeviceSynchronize());
  trace_free(h->trace);
  if (cap == 0) return HL_OK;
  h->trace->rec = (hl_trace_rec*)calloc((size_t)cap, sizeof(hl_trace_rec));
  if (!h->trace->rec) return HL_ERR_CAPACITY;
  for (int i = 0; i < cap; ++i) {
    // timing only: no system-scope fence (cache write-back and invalidate) at
    // each record, which would lengthen and perturb what is measured
    if (hipEventCreateWithFlags(&h->trace->rec[i].a, hipEventDisableSystemFence) != hipSuccess ||
        hipEventCreateWithFlags(&h->trace->rec[i].b, hipEventDisableSystemFence) != hipSuccess) {
      h->trace->cap = i + 1;
      trace_free(h->trace);
      return HL_ERR_HIP;
    }
  }
  h->trace->cap = cap;
  return HL_OK;
}

extern "C" hl_status hl_trace_only(hl_handle* h, const char* name) {
  if (!h || (name && strlen(name) >= sizeof(h->trace->only))) return HL_ERR_INVALID_ARG;
  strcpy(h->trace->only, name ? name : "");
  return HL_OK;
}

extern "C" int32_t hl_trace_count(const hl_handle* h) { return h ? h->trace->n : 0; }

extern "C" hl_status hl_trace_read(const hl_handle* h, int32_t i, const char** name, float* ms) {
  if (!h || i < 0 || i >= h->trace->n || !name || !ms) return HL_ERR_INVALID_ARG;
  HL_HIP(hipEventSynchronize(h->trace->rec[i].b));
  HL_HIP(hipEventElapsedTime(ms, h->trace->rec[i].a, h->trace->rec[i].b));
  *name = h->trace->rec[i].name;
  return HL_OK;
}

extern "C" hl_status hl_trace_read_at(const hl_handle* h, int32_t i, const char** name, float* start_ms,
                                      float* ms) {
  if (!h || i < 0 || i >= h->trace->n || !name || !start_ms || !ms) return HL_ERR_INVALID_ARG;
  const hl_status st = hl_trace_read(h, i, name, ms);
  if (st != HL_OK) return st;
  HL_HIP(hipEventSynchronize(h->trace->rec[0].a));
  HL_HIP(hipEventElapsedTime(start_ms, h->trace->rec[0].a, h->trace->rec[i].a));
  return HL_OK;
}

extern "C" hl_status hl_trace_reset(hl_handle* h) {
  if (!h) return HL_ERR_INVALID_ARG;
  HL_HIP(hipDeviceSynchronize());
  h->trace->n = 0;
  return HL_OK;
}

// ----------------------------------------------------------------------------- handle
// ----------------------------------------------------------------------------- table bounds
__global__ void hl_k_tbounds(const uint32_t* __restrict__ base, int32_t n_tables, const uint64_t* __restrict__ bm,
                             const uint32_t* __restrict__ rank, uint64_t n_entries, uint32_t* __restrict__ tb) {
  for (int32_t t = threadIdx.x; t <= n_tables; t += blockDim.x)
    tb[t] = t < n_tables ? hl_hot_below(bm, rank, base[t]) : rank[n_entries - 1];
}

hl_status hl_table_bounds(hl_handle* h, hipStream_t s) {
  HL_KERNEL(h, s, "hl_k_tbounds", hl_k_tbounds, dim3(1), dim3(256), 0, s, h->d_base, h->n_tables, h->d_bitmap,
            h->d_rank, h->n_tiles4k * 16 + 1, h->d_tb);
  HL_LAUNCHED();
  return HL_OK;
}

extern "C" hl_status hl_create(hl_handle** out, int32_t n_tables, const uint32_t* rows_per_table,
                               int32_t dim, int32_t dtype, uint32_t k_cap) {
  if (!out || n_tables < 1 || !rows_per_table || dim < 1 || dim > 8192 || k_cap < 1)
    return HL_ERR_INVALID_ARG;
  if (dtype != HL_F32 && dtype != HL_BF16) return HL_ERR_INVALID_ARG;
  uint64_t total = 0;
  std::vector<uint32_t> base(n_tables);
  for (int32_t t = 0; t < n_tables; ++t) {
    if (rows_per_table[t] == 0) return HL_ERR_INVALID_ARG;
    base[t] = (uint32_t)total;
    total += rows_per_table[t];
    if (total >= 0xFFFFFFFFull) return HL_ERR_OUT_OF_RANGE;
  }
  hl_handle* h = (hl_handle*)calloc(1, sizeof(hl_handle));
  if (!h) return HL_ERR_CAPACITY;
  h->n_tables = n_tables;
  h->n_rows = total;
  h->dim = dim;
  h->dtype = (hl_dtype)dtype;
  h->k_cap = k_cap;
  h->row_bytes = (uint32_t)dim * (dtype == HL_F32 ? 4u : 2u);
  h->n_tiles4k = (total + 4095) / 4096;
  h->tk_bytes = hl_topk_scratch_bytes(total);
  h->trace = new hl_trace();
  hl_status st = HL_OK;
  if (hipGetDevice(&h->device) != hipSuccess) st = HL_ERR_HIP;
  // the allocation-free backward's static workspace on this device
  if (st == HL_OK) st = hl_scratch_setup(h->device);
  auto dm = [&](void** p, size_t bytes) {
    if (st == HL_OK && hipMalloc(p, bytes) != hipSuccess) st = HL_ERR_HIP;
  };
  dm((void**)&h->d_base, sizeof(uint32_t) * n_tables);
  dm((void**)&h->d_rows, sizeof(uint32_t) * n_tables);
  dm((void**)&h->d_counts, sizeof(uint32_t) * total);
  dm((void**)&h->d_bitmap, sizeof(uint64_t) * h->n_tiles4k * 64);
  dm((void**)&h->d_rank, sizeof(uint32_t) * (h->n_tiles4k * 16 + 1));
  dm((void**)&h->d_tb, sizeof(uint32_t) * (n_tables + 1));
  dm((void**)&h->d_err, sizeof(uint32_t));
  dm((void**)&h->d_tk, h->tk_bytes);
  if (st == HL_OK) {
    if (hipMemcpy(h->d_base, base.data(), sizeof(uint32_t) * n_tables, hipMemcpyHostToDevice) != hipSuccess ||
        hipMemcpy(h->d_rows, rows_per_table, sizeof(uint32_t) * n_tables, hipMemcpyHostToDevice) != hipSuccess)
      st = HL_ERR_HIP;
  }
  if (st == HL_OK) st = fill32(h->d_counts, total, 0, 0);
  if (st == HL_OK) st = fill32((uint32_t*)h->d_bitmap, h->n_tiles4k * 128, 0, 0);
  if (st == HL_OK) st = fill32(h->d_rank, h->n_tiles4k * 16 + 1, 0, 0);
  if (st == HL_OK) st = fill32(h->d_tb, n_tables + 1, 0, 0);
  if (st == HL_OK) st = fill32(h->d_err, 1, 0, 0);
  if (st == HL_OK) st = fill32(h->d_tk, h->tk_bytes / 4, 0, 0);
  if (st == HL_OK && hipDeviceSynchronize() != hipSuccess) st = HL_ERR_HIP;
  if (st != HL_OK) {
    hl_destroy(h);
    return st;
  }
  *out = h;
  return HL_OK;
}

extern "C" hl_status hl_destroy(hl_handle* h) {
  if (!h) return HL_ERR_INVALID_ARG;
  void* ps[] = {h->d_base, h->d_rows, h->d_counts, h->d_bitmap, h->d_rank, h->d_tb, h->d_err, h->d_tk, h->cg_table};
  hl_status st = HL_OK;
  if (h->trace) {
    trace_free(h->trace);
    delete h->trace;
  }
  for (void* p : ps)
    if (p && hipFree(p) != hipSuccess) st = HL_ERR_HIP;
  free(h);
  return st;
}

extern "C" hl_status hl_debug_ballot_ranks(hl_handle* h, int32_t on) {
  if (!h) return HL_ERR_INVALID_ARG;
  h->ballot_ranks = on != 0;
  return HL_OK;
}

extern "C" uint64_t hl_n_rows(const hl_handle* h) { return h ? h->n_rows : 0; }
extern "C" uint32_t hl_n_hot(const hl_handle* h) { return h ? h->n_hot : 0; }
extern "C" uint32_t hl_k_cap(const hl_handle* h) { return h ? h->k_cap : 0; }

extern "C" size_t hl_workspace_bytes(const hl_handle* h, int64_t max_lookups, int64_t max_bags,
                                     int32_t max_samples) {
  if (!h || max_lookups < 0 || max_bags < 0 || max_samples < 0) return 0;
  size_t a = hl_partition_ws_bytes(max_samples);
  size_t b = hl_cold_ws_bytes(h, max_lookups, max_bags, max_samples);
  size_t c = hl_bwd_ws_bytes(h, max_lookups, max_bags);
  size_t d = hl_plan_ws_bytes(h, max_lookups, max_bags, max_samples);
  size_t m = a > b ? a : b;
  m = m > c ? m : c;
  m = m > d ? m : d;
  return (m + 4095) & ~(size_t)4095;
}

extern "C" hl_status hl_workspace_init(void* ws, size_t bytes, hl_stream stream) {
  if (!ws || (bytes & 3)) return HL_ERR_INVALID_ARG;
  return fill32((uint32_t*)ws, bytes / 4, 0, (hipStream_t)stream);
}

extern "C" hl_status hl_last_device_error(hl_handle* h, uint32_t* err_out) {
  if (!h || !err_out) return HL_ERR_INVALID_ARG;
  HL_HIP(hipDeviceSynchronize());
  uint32_t e = 0;
  HL_HIP(hipMemcpy(&e, h->d_err, 4, hipMemcpyDeviceToHost));
  uint32_t z = 0;
  HL_HIP(hipMemcpy(h->d_err, &z, 4, hipMemcpyHostToDevice));
  *err_out = e;
  return e ? HL_ERR_DEVICE : HL_OK;
}

extern "C" hl_status hl_host_alloc(size_t bytes, void** host, void** dev) {
  if (!host || bytes == 0) return HL_ERR_INVALID_ARG;
  void* p = nullptr;
  HL_HIP(hipHostMalloc(&p, bytes, hipHostMallocMapped | hipHostMallocPortable));
  if (dev) {
    void* d = nullptr;
    if (hipHostGetDevicePointer(&d, p, 0) != hipSuccess) {
      (void)hipHostFree(p);
      return HL_ERR_HIP;
    }
    *dev = d;
  }
  *host = p;
  return HL_OK;
}

extern "C" hl_status hl_host_free(void* host) {
  if (!host) return HL_ERR_INVALID_ARG;
  HL_HIP(hipHostFree(host));
  return HL_OK;
}

// ----------------------------------------------------------------------------- gids
// Block = GIDS_BAGS bags; their lookups are contiguous.  Threads walk the
// lookups, four at a time with their row loads issued together, and find each
// one's bag by binary search over the block's bag offsets in LDS.  (The call
// knows bags, not lookups: 64 bags keep multi-hot blocks at ~1300 lookups.)
#define GIDS_BAGS 64
__global__ void __launch_bounds__(256)
hl_k_gids(const uint32_t* __restrict__ rows, const int32_t* __restrict__ bag_ptr, int64_t n_bags,
          const uint32_t* __restrict__ base, const uint32_t* __restrict__ nrow, int32_t n_tables,
          uint32_t* __restrict__ gids, uint32_t* err) {
  __shared__ int32_t off[GIDS_BAGS + 1];
  const int64_t b0 = (int64_t)blockIdx.x * GIDS_BAGS;
  const int nb = (int)min((int64_t)GIDS_BAGS, n_bags - b0);
  for (int j = threadIdx.x; j <= nb; j += blockDim.x) off[j] = bag_ptr[b0 + j];
  __syncthreads();
  const int32_t lo = off[0], hi = off[nb];
  // 4 lookups per thread at a time, their row loads issued together
  for (int32_t i0 = lo + threadIdx.x; i0 < hi; i0 += 4 * (int32_t)blockDim.x) {
    uint32_t r[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int32_t i = i0 + k * (int32_t)blockDim.x;
      r[k] = i < hi ? rows[i] : 0u;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int32_t i = i0 + k * (int32_t)blockDim.x;
      if (i >= hi) continue;
      int a = 0, b = nb;  // off[a] <= i < off[b]
      while (b - a > 1) {
        int m = (a + b) >> 1;
        if (off[m] <= i) a = m; else b = m;
      }
      const int32_t t = (int32_t)((b0 + a) % n_tables);
      if (r[k] < nrow[t]) {
        gids[i] = base[t] + r[k];
      } else {
        gids[i] = 0xFFFFFFFFu;
        hl_flag(err, HL_DEVERR_OUT_OF_RANGE);
      }
    }
  }
}

extern "C" hl_status hl_lookup_gids(const hl_handle* h, const uint32_t* rows, const int32_t* bag_ptr,
                                    int64_t n_bags, uint32_t* gids, hl_stream stream) {
  if (!h || n_bags < 0 || (n_bags > 0 && (!rows || !bag_ptr || !gids))) return HL_ERR_INVALID_ARG;
  if (n_bags == 0) return HL_OK;
  if (n_bags >= (1ll << 31)) return HL_ERR_UNSUPPORTED;
  hipStream_t s = (hipStream_t)stream;
  HL_KERNEL(h, s, "hl_k_gids", hl_k_gids, dim3(hl_div_up(n_bags, GIDS_BAGS)), dim3(256), 0, s,
                     rows, bag_ptr, n_bags, h->d_base, h->d_rows, h->n_tables, gids, h->d_err);
  HL_LAUNCHED();
  return HL_OK;
}

// ----------------------------------------------------------------------------- counting
__global__ void __launch_bounds__(256)
hl_k_count(const uint32_t* __restrict__ gids, int64_t n, uint32_t* __restrict__ counts,
           uint64_t n_rows, uint32_t* err) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t g = gids[i];
    if (g < n_rows) atomicAdd(counts + g, 1u);
    else hl_flag(err, HL_DEVERR_OUT_OF_RANGE);
  }
}

extern "C" hl_status hl_profile_count(hl_handle* h, const uint32_t* gids, int64_t n, hl_stream stream) {
  if (!h || n < 0 || (n > 0 && !gids)) return HL_ERR_INVALID_ARG;
  if (n == 0) return HL_OK;
  uint32_t g = hl_div_up(n, 256);
  if (g > 16384) g = 16384;
  hipStream_t s = (hipStream_t)stream;
  HL_KERNEL(h, s, "hl_k_count", hl_k_count, dim3(g), dim3(256), 0, s, gids, n, h->d_counts,
                     h->n_rows, h->d_err);
  HL_LAUNCHED();
  return HL_OK;
}

extern "C" hl_status hl_profile_counts(const hl_handle* h, uint32_t* counts_out, hl_stream stream) {
  if (!h || !counts_out) return HL_ERR_INVALID_ARG;
  HL_HIP(hipMemcpyAsync(counts_out, h->d_counts, sizeof(uint32_t) * h->n_rows, hipMemcpyDeviceToDevice,
                        (hipStream_t)stream));
  return HL_OK;
}

// ----------------------------------------------------------------------------- gather
// dst[r] = src[ids[r]], bit for bit.  Lanes copy U-byte units of a row; for a
// 256-byte row and U = 16, 16 lanes cover a row and a wave moves 4 rows.
// Ids >= n_src_rows are skipped and flagged (the source is never read out of
// bounds).
template <typename V>
__global__ void __launch_bounds__(256)
hl_k_gather(const uint32_t* __restrict__ ids, const int32_t* n_dev, uint32_t n_host,
            const V* __restrict__ src, uint64_t n_src_rows, V* __restrict__ dst, uint32_t upr,
            uint32_t* err) {
  const uint32_t n = n_dev ? (uint32_t)max((int64_t)0, min((int64_t)*n_dev, (int64_t)n_host)) : n_host;
  const uint64_t total = (uint64_t)n * upr;
  for (uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
       t += (uint64_t)gridDim.x * blockDim.x) {
    const uint32_t r = (uint32_t)(t / upr), c = (uint32_t)(t - (uint64_t)r * upr);
    const uint32_t id = ids[r];
    if (id < n_src_rows) dst[(uint64_t)r * upr + c] = src[(uint64_t)id * upr + c];
    else if (c == 0) hl_flag(err, HL_DEVERR_OUT_OF_RANGE);
  }
}

hl_status hl_launch_gather(const hl_handle* h, const uint32_t* ids, const int32_t* n_dev, uint32_t n_host,
                           const void* src, uint64_t n_src_rows, void* dst, uint32_t row_bytes, uint32_t* err,
                           hipStream_t s) {
  if (n_host == 0) return HL_OK;
  uint64_t total;
  uint32_t g;
#define HL_GATHER_LAUNCH(V)                                                                       \
  total = (uint64_t)n_host * (row_bytes / sizeof(V));                                             \
  g = hl_div_up(total, 256);                                                                      \
  if (g > 16384) g = 16384;                                                                       \
  HL_KERNEL(h, s, "hl_k_gather", hl_k_gather<V>, dim3(g), dim3(256), 0, s, ids, n_dev, n_host, (const V*)src, \
                     n_src_rows, (V*)dst, (uint32_t)(row_bytes / sizeof(V)), err);
  if (row_bytes % 16 == 0) { HL_GATHER_LAUNCH(uint4) }
  else if (row_bytes % 8 == 0) { HL_GATHER_LAUNCH(uint2) }
  else if (row_bytes % 4 == 0) { HL_GATHER_LAUNCH(uint32_t) }
  else { HL_GATHER_LAUNCH(uint16_t) }
#undef HL_GATHER_LAUNCH
  HL_LAUNCHED();
  return HL_OK;
}

extern "C" hl_status hl_hot_fill(const hl_handle* h, const uint32_t* hot_ids, const void* w_host,
                                 void* w_hot, hl_stream stream) {
  if (!h || (h->n_hot && (!hot_ids || !w_host || !w_hot))) return HL_ERR_INVALID_ARG;
  return hl_launch_gather(h, hot_ids, nullptr, h->n_hot, w_host, h->n_rows, w_hot, h->row_bytes, h->d_err,
                          (hipStream_t)stream);
}

// ----------------------------------------------------------------------------- streams
extern "C" hl_status hl_stream_create(int32_t first_cu, int32_t n_cu, int32_t complement, hl_stream* out) {
  if (!out || first_cu < 0 || n_cu < 0) return HL_ERR_INVALID_ARG;
  int dev = 0, ncu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return HL_ERR_HIP;
  if (n_cu == 0) {  // no mask
    hipStream_t s;
    if (hipStreamCreateWithFlags(&s, hipStreamNonBlocking) != hipSuccess) return HL_ERR_HIP;
    *out = (hl_stream)s;
    return HL_OK;
  }
  if (first_cu + n_cu > ncu || (complement && n_cu >= ncu)) return HL_ERR_INVALID_ARG;
  const int words = (ncu + 31) / 32;
  std::vector<uint32_t> mask((size_t)words, 0u);
  for (int c = 0; c < ncu; ++c) {
    const bool in = c >= first_cu && c < first_cu + n_cu;
    if (in != (complement != 0)) mask[(size_t)c / 32] |= 1u << (c % 32);
  }
  hipStream_t s;
  if (hipExtStreamCreateWithCUMask(&s, (uint32_t)words, mask.data()) != hipSuccess) return HL_ERR_HIP;
  *out = (hl_stream)s;
  return HL_OK;
}

extern "C" hl_status hl_stream_destroy(hl_stream s) {
  if (!s) return HL_ERR_INVALID_ARG;
  return hipStreamDestroy((hipStream_t)s) == hipSuccess ? HL_OK : HL_ERR_HIP;
}
