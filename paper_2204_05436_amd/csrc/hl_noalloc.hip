// The backward of sum pooling with one coalesced SGD step (hl_embbag_bwd_sgd)
// without a workspace argument and without allocating: its workspace is a
// file-scope device array of fixed size, one copy per GPU, for callers that
// cannot allocate device memory (code under graph capture, serving loops,
// harnesses that forbid allocation).  Every call on a GPU uses that GPU's copy
// and leaves its last contents there; the kernels keep the state that must
// start at zero (tile counters, look-back words) reset themselves, and the
// copy is zero-filled once when its address is looked up.  Calls that overlap
// on one GPU race on the array.
#include <mutex>

#include "hl_internal.h"

#define HL_SCRATCH_BYTES ((size_t)32 << 20)
#define HL_SCRATCH_DEVICES 64

static __device__ __align__(256) uint8_t scratch[HL_SCRATCH_BYTES];

static std::mutex g_scratch_mu;
static void* g_scratch[HL_SCRATCH_DEVICES];  // device address of each GPU's copy

hl_status hl_fill32(uint32_t* p, uint64_t n, uint32_t v, hipStream_t s);

// Once per device, with that device current: the address of its copy of the
// array (in host code the array's name is no device address), then a zero fill.
hl_status hl_scratch_setup(int device) {
  if (device < 0 || device >= HL_SCRATCH_DEVICES) return HL_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch[device]) return HL_OK;
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return HL_ERR_HIP;
  if (cur != device && hipSetDevice(device) != hipSuccess) return HL_ERR_HIP;
  void* ptr = nullptr;
  hl_status st = HL_OK;
  if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) st = HL_ERR_HIP;
  if (st == HL_OK) st = hl_fill32((uint32_t*)ptr, HL_SCRATCH_BYTES / 4, 0, nullptr);
  if (st == HL_OK && hipStreamSynchronize(nullptr) != hipSuccess) st = HL_ERR_HIP;
  if (st == HL_OK) g_scratch[device] = ptr;
  if (cur != device && hipSetDevice(cur) != hipSuccess) st = HL_ERR_HIP;
  return st;
}

extern "C" size_t hl_noalloc_scratch_bytes(void) { return HL_SCRATCH_BYTES; }

extern "C" hl_status hl_embbag_bwd_sgd_noalloc(hl_handle* h, void* w_hot, void* staging, int32_t stg_rows,
                                               const int32_t* codes, const int32_t* bag_ptr, int32_t n_samples,
                                               int32_t bps, int64_t n_lookups, const int32_t* sample_ids,
                                               const int32_t* n_sel_dev, int32_t n_sel_max, const float* dY,
                                               float lr, hl_stream stream) {
  if (!h || n_samples < 0 || bps < 1 || n_lookups < 0 || n_sel_max < 0 || stg_rows < 0) return HL_ERR_INVALID_ARG;
  if (!bag_ptr || (n_lookups > 0 && !codes)) return HL_ERR_INVALID_ARG;
  if (n_samples == 0 || n_lookups == 0 || n_sel_max == 0) return HL_OK;
  if (!dY || (h->n_hot && !w_hot) || (stg_rows && !staging)) return HL_ERR_INVALID_ARG;
  if ((int64_t)n_samples * bps >= (1ll << 31) || n_lookups >= (1ll << 30)) return HL_ERR_UNSUPPORTED;
  const int64_t n_bags = (int64_t)n_samples * bps;
  if (hl_bwd_ws_bytes_compact(h, n_lookups, n_bags) > HL_SCRATCH_BYTES) return HL_ERR_CAPACITY;
  void* ws = (h->device >= 0 && h->device < HL_SCRATCH_DEVICES) ? g_scratch[h->device] : nullptr;
  if (!ws) return HL_ERR_HIP;  // the handle's set-up found no address for the array
  bool sent = false;
  hl_status st = hl_embbag_bwd_plan_signal(h, stg_rows, const_cast<int32_t*>(codes), bag_ptr, n_samples, bps,
                                           n_lookups, sample_ids, n_sel_dev, n_sel_max, ws, HL_SCRATCH_BYTES, stream,
                                           nullptr, 0, &sent, nullptr, true);
  if (st != HL_OK) return st;
  return hl_embbag_bwd_apply_any(h, w_hot, staging, stg_rows, n_samples, bps, n_lookups, dY, lr, 0, ws,
                                 HL_SCRATCH_BYTES, stream);
}
