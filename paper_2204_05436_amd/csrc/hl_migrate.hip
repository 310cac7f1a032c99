// Hot-set migration of the recurring learning phase (Sec. V-B: the EAL
// switches back to learning from time to time; Sec. IV: hot rows are trained
// on the GPU, the others in CPU memory).  Once a new hot set has replaced the
// old one in the handle (hl_profile_topk or hl_set_hot), the hot cache is
// rebuilt in the new slot order: a row that stays moves from its old slot
// with its trained value, a row that enters is read from the host table, and
// a row that leaves is written back to the host table.  The table the path
// reads (a hot row from the cache, any other from the host) is the same
// before and after.
//
// One launch, two roles that touch disjoint rows: blocks [0, fill_blocks)
// take the new slots (a binary search of the old ids gives a staying row's
// old slot), the others the old slots (the new set's bitmap tells the rows
// that leave).  Per round a block resolves up to 256 / units-per-row rows
// and then copies them with one 16-byte (or narrower) unit per thread.
#include "hl_internal.h"

#define HM_SKIP INT64_MIN

// first position in ascending v[0..n) holding a value >= key
__device__ __forceinline__ uint32_t hm_lower_bound(const uint32_t* __restrict__ v, uint32_t n, uint32_t key) {
  uint32_t lo = 0, hi = n;
  while (lo < hi) {
    const uint32_t m = lo + ((hi - lo) >> 1);
    if (v[m] < key) lo = m + 1;
    else hi = m;
  }
  return lo;
}

template <typename V>
__global__ void __launch_bounds__(256)
hm_migrate(const uint32_t* __restrict__ old_ids, uint32_t n_old, const uint32_t* __restrict__ new_ids,
           uint32_t n_new, const uint64_t* __restrict__ bitmap, uint64_t n_rows, const V* __restrict__ w_old,
           V* __restrict__ w_new, V* host, uint32_t upr, uint32_t fill_blocks, uint32_t* err) {
  __shared__ int64_t src[256];
  const uint32_t rpi = upr >= 256 ? 1u : 256u / upr;  // rows per round
  const bool fill = blockIdx.x < fill_blocks;
  const uint32_t nb = fill ? fill_blocks : gridDim.x - fill_blocks;
  const uint32_t b = fill ? blockIdx.x : blockIdx.x - fill_blocks;
  const uint32_t n = fill ? n_new : n_old;
  for (uint64_t r0 = (uint64_t)b * rpi; r0 < n; r0 += (uint64_t)nb * rpi) {
    if (threadIdx.x < rpi) {
      const uint64_t r = r0 + threadIdx.x;
      int64_t v = HM_SKIP;
      if (r < n) {
        const uint32_t g = fill ? new_ids[r] : old_ids[r];
        if (g >= n_rows) {
          hl_flag(err, HL_DEVERR_BAD_HOTSET);
        } else if (fill) {
          // >= 0: the old slot of a staying row; < 0: -(id + 1) of a row read from the host
          const uint32_t o = hm_lower_bound(old_ids, n_old, g);
          v = o < n_old && old_ids[o] == g ? (int64_t)o : -(int64_t)g - 1;
        } else if (!hl_is_hot(bitmap, g)) {
          v = (int64_t)g;  // leaves the cache: back to the host table
        }
      }
      src[threadIdx.x] = v;
    }
    __syncthreads();
    for (uint32_t t = threadIdx.x; t < rpi * upr; t += 256) {
      const uint32_t j = t / upr, c = t - j * upr;
      const uint64_t r = r0 + j;
      const int64_t v = src[j];
      if (r >= n || v == HM_SKIP) continue;
      if (fill) w_new[r * upr + c] = v >= 0 ? w_old[(uint64_t)v * upr + c] : host[(uint64_t)(-v - 1) * upr + c];
      else host[(uint64_t)v * upr + c] = w_old[r * upr + c];
    }
    __syncthreads();
  }
}

extern "C" hl_status hl_hot_migrate(const hl_handle* h, const uint32_t* old_ids, uint32_t n_old,
                                    const uint32_t* new_ids, const void* w_hot_old, void* w_hot_new, void* w_host,
                                    hl_stream stream) {
  if (!h) return HL_ERR_INVALID_ARG;
  const uint32_t n_new = h->n_hot;
  if (n_old > h->k_cap) return HL_ERR_CAPACITY;
  if ((n_old && (!old_ids || !w_hot_old)) || (n_new && (!new_ids || !w_hot_new)) || ((n_old || n_new) && !w_host))
    return HL_ERR_INVALID_ARG;
  if (n_old == 0 && n_new == 0) return HL_OK;
  const uint64_t rb = (uint64_t)h->dim * (h->dtype == HL_F32 ? 4 : 2);
  // the old and new caches must not overlap (rows move between slots)
  const char *a0 = (const char*)w_hot_old, *b0 = (const char*)w_hot_new;
  if (n_old && n_new && a0 < b0 + n_new * rb && b0 < a0 + n_old * rb) return HL_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  const uintptr_t al = (uintptr_t)w_hot_old | (uintptr_t)w_hot_new | (uintptr_t)w_host;
#define HM_LAUNCH(V)                                                                                             \
  do {                                                                                                           \
    const uint32_t upr = (uint32_t)(rb / sizeof(V));                                                             \
    const uint32_t rpi = upr >= 256 ? 1u : 256u / upr;                                                           \
    uint32_t fb = hl_div_up(n_new, rpi), ob = hl_div_up(n_old, rpi);                                           \
    fb = fb > 1024 ? 1024 : fb;                                                                                  \
    ob = ob > 1024 ? 1024 : ob;                                                                                  \
    HL_KERNEL(h, s, "hm_migrate", hm_migrate<V>, dim3(fb + ob), dim3(256), 0, s, old_ids, n_old, new_ids, n_new, \
              h->d_bitmap, h->n_rows, (const V*)w_hot_old, (V*)w_hot_new, (V*)w_host, upr, fb, h->d_err);      \
  } while (0)
  if (rb % 16 == 0 && al % 16 == 0) HM_LAUNCH(uint4);
  else if (rb % 8 == 0 && al % 8 == 0) HM_LAUNCH(uint2);
  else if (rb % 4 == 0 && al % 4 == 0) HM_LAUNCH(uint32_t);
  else HM_LAUNCH(uint16_t);
#undef HM_LAUNCH
  HL_LAUNCHED();
  return HL_OK;
}
