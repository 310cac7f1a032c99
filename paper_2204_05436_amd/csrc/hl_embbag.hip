// EmbeddingBag sum-pooling forward and the coalesced sparse-SGD backward over
// the hot cache (HBM) and the staging buffer of gathered cold rows.
//
// Lane layout: a row is covered by G lanes holding VEC consecutive elements
// each (fp32: 16-byte loads for VEC = 4; bf16: 16-byte loads for VEC = 8,
// widened to fp32),
// G = min(dim/VEC, 64); a wave holds NG = 64/G row groups; rows wider than 64
// vectors are split into column chunks over blockIdx.y.
//
// Backward: the lookups of the mini-batch are sorted by compressed row key
// (hot slot, or n_hot + staging row) with their bag as payload; then tiles of
// the sorted list are reduced by groups of E consecutive entries: a run of
// equal keys entirely inside a group is a complete segment and its row is
// updated at once; pieces of runs that cross group boundaries are combined in
// LDS in group order, and pieces that cross tile boundaries are combined by a
// second kernel in tile order.  Every row is read and written once and the
// summation order depends only on the sorted order, so results are
// deterministic.
#include <algorithm>
#include <initializer_list>

#include "hl_group_sort.h"
#include "hl_internal.h"

// sorted entries per row group of the reduction: 6 for rows of 4 or more
// elements per lane (the register budget of 7 waves per SIMD), else 8
#define RB_EN(V) ((V) >= 4 ? 6 : 8)
#ifndef RB_WAVES
#define RB_WAVES 2  // waves per reduction block (2 measured fastest: a block waits for its slowest wave)
#endif
#define RB_BLOCK (RB_WAVES * 64)

// ----------------------------------------------------------------------------- row I/O
template <int VEC, bool BF>
struct RowIO;

// A row slice of VEC elements: load() gives it as floats; load_raw() keeps the
// loaded bytes (Raw) and unpack() converts them when they are used, so a row
// in flight holds only its bytes' registers (bf16: half of the floats').
template <>
struct RowIO<4, false> {
  typedef float T;
  typedef float4 Raw;
  static __device__ __forceinline__ Raw load_raw(const T* p) { return *reinterpret_cast<const float4*>(p); }
  static __device__ __forceinline__ void unpack(const Raw& x, float* v) {
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
  }
  static __device__ __forceinline__ void load(const T* p, float* v) { unpack(load_raw(p), v); }
  static __device__ __forceinline__ void store(T* p, const float* v) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  }
};
template <>
struct RowIO<2, false> {
  typedef float T;
  typedef float2 Raw;
  static __device__ __forceinline__ Raw load_raw(const T* p) { return *reinterpret_cast<const float2*>(p); }
  static __device__ __forceinline__ void unpack(const Raw& x, float* v) {
    v[0] = x.x; v[1] = x.y;
  }
  static __device__ __forceinline__ void load(const T* p, float* v) { unpack(load_raw(p), v); }
  static __device__ __forceinline__ void store(T* p, const float* v) {
    *reinterpret_cast<float2*>(p) = make_float2(v[0], v[1]);
  }
};
template <>
struct RowIO<8, false> {
  typedef float T;
  struct Raw {
    float4 a, b;
  };
  static __device__ __forceinline__ Raw load_raw(const T* p) {
    return Raw{*reinterpret_cast<const float4*>(p), *reinterpret_cast<const float4*>(p + 4)};
  }
  static __device__ __forceinline__ void unpack(const Raw& x, float* v) {
    RowIO<4, false>::unpack(x.a, v);
    RowIO<4, false>::unpack(x.b, v + 4);
  }
  static __device__ __forceinline__ void load(const T* p, float* v) { unpack(load_raw(p), v); }
  static __device__ __forceinline__ void store(T* p, const float* v) {
    RowIO<4, false>::store(p, v);
    RowIO<4, false>::store(p + 4, v + 4);
  }
};
template <>
struct RowIO<1, false> {
  typedef float T;
  typedef float Raw;
  static __device__ __forceinline__ Raw load_raw(const T* p) { return *p; }
  static __device__ __forceinline__ void unpack(const Raw& x, float* v) { v[0] = x; }
  static __device__ __forceinline__ void load(const T* p, float* v) { v[0] = *p; }
  static __device__ __forceinline__ void store(T* p, const float* v) { *p = v[0]; }
};

__device__ __forceinline__ float bf2f(uint32_t b) { return __uint_as_float(b << 16); }
__device__ __forceinline__ uint32_t f2bf(float f) {  // round to nearest even (finite values)
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

template <>
struct RowIO<4, true> {
  typedef uint16_t T;
  typedef uint2 Raw;
  static __device__ __forceinline__ Raw load_raw(const T* p) { return *reinterpret_cast<const uint2*>(p); }
  static __device__ __forceinline__ void unpack(const Raw& x, float* v) {
    v[0] = bf2f(x.x & 0xFFFFu); v[1] = bf2f(x.x >> 16); v[2] = bf2f(x.y & 0xFFFFu); v[3] = bf2f(x.y >> 16);
  }
  static __device__ __forceinline__ void load(const T* p, float* v) { unpack(load_raw(p), v); }
  static __device__ __forceinline__ void store(T* p, const float* v) {
    *reinterpret_cast<uint2*>(p) = make_uint2(f2bf(v[0]) | (f2bf(v[1]) << 16), f2bf(v[2]) | (f2bf(v[3]) << 16));
  }
};
template <>
struct RowIO<8, true> {
  typedef uint16_t T;
  typedef uint4 Raw;
  static __device__ __forceinline__ Raw load_raw(const T* p) { return *reinterpret_cast<const uint4*>(p); }
  static __device__ __forceinline__ void unpack(const Raw& x, float* v) {
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = bf2f(w[i] & 0xFFFFu);
      v[2 * i + 1] = bf2f(w[i] >> 16);
    }
  }
  static __device__ __forceinline__ void load(const T* p, float* v) { unpack(load_raw(p), v); }
  static __device__ __forceinline__ void store(T* p, const float* v) {
    *reinterpret_cast<uint4*>(p) = make_uint4(f2bf(v[0]) | (f2bf(v[1]) << 16), f2bf(v[2]) | (f2bf(v[3]) << 16),
                                              f2bf(v[4]) | (f2bf(v[5]) << 16), f2bf(v[6]) | (f2bf(v[7]) << 16));
  }
};
template <>
struct RowIO<2, true> {
  typedef uint16_t T;
  typedef uint32_t Raw;
  static __device__ __forceinline__ Raw load_raw(const T* p) { return *reinterpret_cast<const uint32_t*>(p); }
  static __device__ __forceinline__ void unpack(const Raw& x, float* v) {
    v[0] = bf2f(x & 0xFFFFu); v[1] = bf2f(x >> 16);
  }
  static __device__ __forceinline__ void load(const T* p, float* v) { unpack(load_raw(p), v); }
  static __device__ __forceinline__ void store(T* p, const float* v) {
    *reinterpret_cast<uint32_t*>(p) = f2bf(v[0]) | (f2bf(v[1]) << 16);
  }
};
template <>
struct RowIO<1, true> {
  typedef uint16_t T;
  typedef uint16_t Raw;
  static __device__ __forceinline__ Raw load_raw(const T* p) { return *p; }
  static __device__ __forceinline__ void unpack(const Raw& x, float* v) { v[0] = bf2f(x); }
  static __device__ __forceinline__ void load(const T* p, float* v) { v[0] = bf2f(*p); }
  static __device__ __forceinline__ void store(T* p, const float* v) { *p = (uint16_t)f2bf(v[0]); }
};

template <int VEC>
__device__ __forceinline__ void ld_f32(const float* p, float* v) { RowIO<VEC, false>::load(p, v); }
template <int VEC>
__device__ __forceinline__ void st_f32(float* p, const float* v) { RowIO<VEC, false>::store(p, v); }

// Pooled outputs are written once per launch and not read again by it: the
// non-temporal hint marks their lines for early eviction, so they do not push
// the hot rows out of the caches (the forward's hot half measured ~20% faster
// alone on the GPU; the same hint on the backward's gradient-row loads was
// slower, and they keep plain loads).
typedef float hl_f4 __attribute__((ext_vector_type(4)));
template <int VEC>
__device__ __forceinline__ void st_f32_nt(float* p, const float* v) {
  if constexpr (VEC == 4 || VEC == 8) {
#pragma unroll
    for (int i = 0; i < VEC; i += 4) {
      const hl_f4 x = {v[i], v[i + 1], v[i + 2], v[i + 3]};
      __builtin_nontemporal_store(x, reinterpret_cast<hl_f4*>(p + i));
    }
  } else {
    RowIO<VEC, false>::store(p, v);
  }
}

struct eb_geom {
  int32_t D, vpr, G, NG, cchunks, VEC;
};

static eb_geom eb_make_geom(int32_t D, int vec) {
  eb_geom g;
  g.D = D;
  g.VEC = vec;
  g.vpr = D / vec;
  g.G = g.vpr < 64 ? g.vpr : 64;
  g.NG = 64 / g.G;
  g.cchunks = (g.vpr + 63) / 64;
  return g;
}

// bf16 rows take 8 elements per lane (16-byte loads), fp32 rows 4; fewer
// when the dimension or a pointer's alignment does not allow them
static int eb_pick_vec(int32_t D, size_t esize, std::initializer_list<const void*> ptrs) {
  int vec = (esize == 2 && D % 8 == 0) ? 8 : (D % 4 == 0 ? 4 : (D % 2 == 0 ? 2 : 1));
  for (;;) {
    bool ok = true;
    for (const void* p : ptrs)
      if (p && ((uintptr_t)p % (vec * esize) != 0 || (uintptr_t)p % (vec * 4) != 0)) ok = false;
    if (ok || vec == 1) return vec;
    vec >>= 1;
  }
}

// selected-sample count
__device__ __forceinline__ int32_t eb_nsel(const int32_t* ids, const int32_t* n_dev, int32_t n_max) {
  if (ids && n_dev) return min(max(*n_dev, 0), n_max);
  return n_max;
}

// ----------------------------------------------------------------------------- forward
// A row group takes FC (bags of about one lookup) or 1 (multi-hot bags)
// consecutive bag slots of the selection (slot q = bag j of selected sample
// q / bps) and issues the loads of all of them before using any: offsets,
// then codes, then rows, so FC rows per lane are in flight.  When every bag of
// the chunk holds one lookup (one-hot features) that is the whole work;
// otherwise bags are pooled one by one (eb_bag).
//
// A bag's sum is the sum of its hot rows plus the sum of its staging (cold)
// rows, each in CSR order, so that the two halves can run apart with
// identical results: PART 0 does both, PART 1 only the hot rows (writing the
// partial sum), PART 2 adds the cold rows' sum onto the stored partial sum
// (bags without cold rows are left alone).  The hot half needs no fetched row,
// so it runs while the working parameters still travel over the host link.
#ifndef FC
#define FC 4  // bag slots per row group of the forward (4 measured fastest of 4, 6, 8, 12, 16)
#endif
__device__ __forceinline__ bool eb_code_row(uint32_t cu, uint32_t n_hot, uint32_t k_cap, int32_t stg_rows,
                                            int64_t* row, bool* stg) {
  if (cu < n_hot) {
    *row = cu;
    *stg = false;
    return true;
  }
  if (cu >= k_cap && cu - k_cap < (uint32_t)stg_rows) {
    *row = cu - k_cap;
    *stg = true;
    return true;
  }
  return false;
}

// acc += the bag's rows of one kind (hot, or staging when COLD), in CSR order.
// Invalid codes are flagged by the hot pass only.  Called by a whole row
// group at once (its G lanes in the same control flow).  Row groups of 8 lanes
// or more load the codes of G lookups at once, one per lane, and take the row
// indices from each other by shuffles, 8 rows in flight; narrower groups load
// 4 codes, then 4 rows, at a time.  Either way each lane adds the rows in CSR
// order.
template <int VEC, bool BF, bool COLD>
__device__ __forceinline__ void eb_pass4(float* acc, const typename RowIO<VEC, BF>::T* w_hot,
                                         const typename RowIO<VEC, BF>::T* stg, int32_t stg_rows, uint32_t n_hot,
                                         uint32_t k_cap, const int32_t* __restrict__ codes, int32_t lo, int32_t hi,
                                         eb_geom g, int64_t col, bool cact, int gl, uint32_t* err, bool* any) {
  for (int32_t i = lo; i < hi; i += 4) {
    uint32_t cc[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) cc[k] = i + k < hi ? (uint32_t)codes[i + k] : 0u;
    float v[4][VEC];
    bool use[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      int64_t r = 0;
      bool st = false;
      const bool in = i + k < hi;
      const bool ok = in && eb_code_row(cc[k], n_hot, k_cap, stg_rows, &r, &st);
      use[k] = ok && st == COLD;
      *any = *any || use[k];
      if (use[k] && cact) RowIO<VEC, BF>::load((COLD ? stg : w_hot) + r * g.D + col, v[k]);
      if (!COLD && in && !ok && gl == 0) hl_flag(err, HL_DEVERR_BAD_CODE);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (use[k] && cact)
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[e] += v[k][e];
  }
}

#ifndef EB_SEG_ROWS
#define EB_SEG_ROWS 8  // rows in flight per lane in the passes' wide form
#endif

// The wide form's segment: the codes of lookups b0 .. b0 + G - 1 of [b0, hi),
// one per lane of the group (an invalid code past hi; a lane's own code that
// names no row is flagged when `flag`).
__device__ __forceinline__ uint32_t eb_seg_code(const int32_t* __restrict__ codes, int32_t b0, int32_t hi, int gl,
                                                uint32_t n_hot, uint32_t k_cap, int32_t stg_rows, bool flag,
                                                uint32_t* err) {
  const int32_t i = b0 + gl;
  if (i >= hi) return ~0u;
  const uint32_t c = (uint32_t)codes[i];
  int64_t r;
  bool st;
  if (flag && !eb_code_row(c, n_hot, k_cap, stg_rows, &r, &st)) hl_flag(err, HL_DEVERR_BAD_CODE);
  return c;
}

// acc += the bag's rows of one kind (hot, or staging when COLD), in CSR order;
// *any: some row of that kind was found.  Invalid codes are flagged by the hot
// pass only.  Called by a whole row group at once (its G lanes in the same
// control flow).  Row groups of 8 lanes or more load the codes of G lookups at
// once, one per lane, and take them from each other by shuffles, 8 rows in
// flight; narrower groups load 4 codes, then 4 rows, at a time.  Either way
// each lane adds the rows in CSR order.
template <int VEC, bool BF, bool COLD>
__device__ __forceinline__ void eb_pass(float* acc, const typename RowIO<VEC, BF>::T* w_hot,
                                        const typename RowIO<VEC, BF>::T* stg, int32_t stg_rows, uint32_t n_hot,
                                        uint32_t k_cap, const int32_t* __restrict__ codes, int32_t lo, int32_t hi,
                                        eb_geom g, int64_t col, bool cact, int gl, uint32_t* err, bool* any) {
  if (g.G < EB_SEG_ROWS) {
    eb_pass4<VEC, BF, COLD>(acc, w_hot, stg, stg_rows, n_hot, k_cap, codes, lo, hi, g, col, cact, gl, err, any);
    return;
  }
  const int g0 = (int)(threadIdx.x & 63) - gl;  // the group's first lane
  for (int32_t b0 = lo; b0 < hi; b0 += g.G) {
    const uint32_t mine = eb_seg_code(codes, b0, hi, gl, n_hot, k_cap, stg_rows, !COLD, err);
    const int n = min(g.G, hi - b0);
    for (int k0 = 0; k0 < n; k0 += EB_SEG_ROWS) {
      bool use[EB_SEG_ROWS];
      typename RowIO<VEC, BF>::Raw rv[EB_SEG_ROWS];
#pragma unroll
      for (int k = 0; k < EB_SEG_ROWS; ++k) {
        const uint32_t c = (uint32_t)__shfl((int)mine, g0 + min(k0 + k, n - 1));
        int64_t r = 0;
        bool st = false;
        use[k] = k0 + k < n && eb_code_row(c, n_hot, k_cap, stg_rows, &r, &st) && st == COLD;
        *any = *any || use[k];
        if (use[k] && cact) rv[k] = RowIO<VEC, BF>::load_raw((COLD ? stg : w_hot) + r * g.D + col);
      }
#pragma unroll
      for (int k = 0; k < EB_SEG_ROWS; ++k)
        if (use[k] && cact) {
          float v[VEC];
          RowIO<VEC, BF>::unpack(rv[k], v);
#pragma unroll
          for (int e = 0; e < VEC; ++e) acc[e] += v[e];
        }
    }
  }
}

// Both kinds at once, into separate sums (hot into acc_h, staging into acc_c,
// each in CSR order: the sums the two single-kind passes give), with one code
// load per segment.  *anyc: some staging row was found.
template <int VEC, bool BF>
__device__ __forceinline__ void eb_pass_both(float* acc_h, float* acc_c, bool* anyc,
                                             const typename RowIO<VEC, BF>::T* w_hot,
                                             const typename RowIO<VEC, BF>::T* stg, int32_t stg_rows, uint32_t n_hot,
                                             uint32_t k_cap, const int32_t* __restrict__ codes, int32_t lo, int32_t hi,
                                             eb_geom g, int64_t col, bool cact, int gl, uint32_t* err) {
  if (g.G < EB_SEG_ROWS) {
    bool anyh = false;
    eb_pass4<VEC, BF, false>(acc_h, w_hot, stg, stg_rows, n_hot, k_cap, codes, lo, hi, g, col, cact, gl, err, &anyh);
    eb_pass4<VEC, BF, true>(acc_c, w_hot, stg, stg_rows, n_hot, k_cap, codes, lo, hi, g, col, cact, gl, err, anyc);
    return;
  }
  const int g0 = (int)(threadIdx.x & 63) - gl;
  for (int32_t b0 = lo; b0 < hi; b0 += g.G) {
    const uint32_t mine = eb_seg_code(codes, b0, hi, gl, n_hot, k_cap, stg_rows, true, err);
    const int n = min(g.G, hi - b0);
    for (int k0 = 0; k0 < n; k0 += EB_SEG_ROWS) {
      bool use[EB_SEG_ROWS], cold[EB_SEG_ROWS];
      typename RowIO<VEC, BF>::Raw rv[EB_SEG_ROWS];
#pragma unroll
      for (int k = 0; k < EB_SEG_ROWS; ++k) {
        const uint32_t c = (uint32_t)__shfl((int)mine, g0 + min(k0 + k, n - 1));
        int64_t r = 0;
        bool st = false;
        use[k] = k0 + k < n && eb_code_row(c, n_hot, k_cap, stg_rows, &r, &st);
        cold[k] = st;
        *anyc = *anyc || (use[k] && st);
        if (use[k] && cact) rv[k] = RowIO<VEC, BF>::load_raw((st ? stg : w_hot) + r * g.D + col);
      }
#pragma unroll
      for (int k = 0; k < EB_SEG_ROWS; ++k)
        if (use[k] && cact) {
          float v[VEC];
          RowIO<VEC, BF>::unpack(rv[k], v);
          float* a = cold[k] ? acc_c : acc_h;
#pragma unroll
          for (int e = 0; e < VEC; ++e) a[e] += v[e];
        }
    }
  }
}

// One bag pooled into *o (the row group's slice of the bag's output row):
// PART 0 sums the hot rows and the staging rows apart (each in CSR order) and
// stores their sum (the hot sum alone when no staging row is in the bag);
// PART 1 stores the hot sum; PART 2 adds the staging rows' sum onto the stored
// hot sum (bags without staging rows are left alone).  So PART 1 then PART 2
// store what PART 0 does.
template <int VEC, bool BF, int PART>
__device__ __forceinline__ void eb_bag(float* o, const typename RowIO<VEC, BF>::T* w_hot,
                                       const typename RowIO<VEC, BF>::T* stg, int32_t stg_rows, uint32_t n_hot,
                                       uint32_t k_cap, const int32_t* __restrict__ codes, int32_t lo, int32_t hi,
                                       eb_geom g, int64_t col, bool cact, int gl, uint32_t* err) {
  float acc[VEC], accc[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) {
    acc[e] = 0.f;
    accc[e] = 0.f;
  }
  bool anyc = false;
  if (PART == 0) {
    eb_pass_both<VEC, BF>(acc, accc, &anyc, w_hot, stg, stg_rows, n_hot, k_cap, codes, lo, hi, g, col, cact, gl,
                          err);
  } else if (PART == 1) {
    bool anyh = false;
    eb_pass<VEC, BF, false>(acc, w_hot, stg, stg_rows, n_hot, k_cap, codes, lo, hi, g, col, cact, gl, err, &anyh);
  } else {
    eb_pass<VEC, BF, true>(accc, w_hot, stg, stg_rows, n_hot, k_cap, codes, lo, hi, g, col, cact, gl, err, &anyc);
    if (!anyc) return;
    if (cact) ld_f32<VEC>(o, acc);
  }
  if (anyc)
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] += accc[e];
  if (cact) st_f32_nt<VEC>(o, acc);
}

// The forward's work of block bid of nblk (each of blockDim.x / 64 waves).
template <int VEC, bool BF, int PART>
__device__ __forceinline__ void eb_fwd_body(uint32_t bid, uint32_t nblk, const void* w_hot_, const void* stg_,
                                            int32_t stg_rows, uint32_t n_hot, uint32_t k_cap,
                                            const int32_t* __restrict__ codes, const int32_t* __restrict__ bag_ptr,
                                            int32_t bps, const int32_t* __restrict__ sample_ids,
                                            const int32_t* n_sel_dev, int32_t n_sel_max, float* __restrict__ out,
                                            eb_geom g, int32_t n_samples, int32_t nbg, uint32_t* err) {
  typedef typename RowIO<VEC, BF>::T T;
  const T* w_hot = (const T*)w_hot_;
  const T* stg = (const T*)stg_;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int gi = lane / g.G, gl = lane - gi * g.G;
  if (gi >= g.NG) return;
  const int32_t colv = blockIdx.y * 64 + gl;
  const bool cact = colv < g.vpr;
  const int64_t col = (int64_t)colv * VEC;
  const int64_t total = (int64_t)eb_nsel(sample_ids, n_sel_dev, n_sel_max) * bps;
  const int64_t chunks = (total + nbg - 1) / nbg;
  const int64_t stride = (int64_t)nblk * nw * g.NG;
  for (int64_t c = ((int64_t)bid * nw + w) * g.NG + gi; c < chunks; c += stride) {
    const int64_t q0 = c * nbg;
    int64_t si = q0 / bps, j = q0 - si * bps;
    int64_t bag[FC];
    bool val[FC];
#pragma unroll
    for (int u = 0; u < FC; ++u) {
      val[u] = u < nbg && q0 + u < total;
      int64_t smp = si;
      if (val[u] && sample_ids) smp = sample_ids[si];
      if (val[u] && (smp < 0 || smp >= n_samples)) {
        if (gl == 0 && PART != 2) hl_flag(err, HL_DEVERR_OUT_OF_RANGE);
        val[u] = false;
      }
      bag[u] = smp * bps + j;
      if (++j == bps) {
        j = 0;
        ++si;
      }
    }
    int32_t lo[FC], hi[FC];
    bool one = true;
#pragma unroll
    for (int u = 0; u < FC; ++u) {
      lo[u] = val[u] ? bag_ptr[bag[u]] : 0;
      hi[u] = val[u] ? bag_ptr[bag[u] + 1] : 1;
    }
#pragma unroll
    for (int u = 0; u < FC; ++u) one = one && (hi[u] - lo[u] == 1);
    if (one) {
      uint32_t cu[FC];
#pragma unroll
      for (int u = 0; u < FC; ++u) cu[u] = val[u] ? (uint32_t)codes[lo[u]] : 0u;
      float v[FC][VEC];
      bool wr[FC];
#pragma unroll
      for (int u = 0; u < FC; ++u) {
        int64_t r = 0;
        bool st = false;
        const bool ok = val[u] && eb_code_row(cu[u], n_hot, k_cap, stg_rows, &r, &st);
        // PART 0 and 1 write every valid bag (PART 1 a zero for a cold row); PART 2 only cold ones
        const bool take = ok && (PART == 0 || (PART == 1 ? !st : st));
        wr[u] = val[u] && (PART == 2 ? take : true);
        if (take && cact) RowIO<VEC, BF>::load((st ? stg : w_hot) + r * g.D + col, v[u]);
        else {
#pragma unroll
          for (int e = 0; e < VEC; ++e) v[u][e] = 0.f;
        }
        if (PART != 2 && val[u] && !ok && gl == 0) hl_flag(err, HL_DEVERR_BAD_CODE);
      }
      // the sum starts from 0 (PART 2: from the stored hot partial sum, which is 0)
#pragma unroll
      for (int u = 0; u < FC; ++u)
        if (wr[u] && cact) {
          float o[VEC];
          if (PART == 2) ld_f32<VEC>(out + bag[u] * g.D + col, o);
          else
#pragma unroll
            for (int e = 0; e < VEC; ++e) o[e] = 0.f;
#pragma unroll
          for (int e = 0; e < VEC; ++e) o[e] += v[u][e];
          st_f32_nt<VEC>(out + bag[u] * g.D + col, o);
        }
      continue;
    }
    for (int u = 0; u < FC; ++u) {
      if (!val[u]) continue;
      eb_bag<VEC, BF, PART>(out + bag[u] * g.D + col, w_hot, stg, stg_rows, n_hot, k_cap, codes, lo[u], hi[u], g,
                            col, cact, gl, err);
    }
  }
}

template <int VEC, bool BF, int PART>
__global__ void __launch_bounds__(256)
eb_fwd(const void* w_hot, const void* stg, int32_t stg_rows, uint32_t n_hot, uint32_t k_cap,
       const int32_t* __restrict__ codes, const int32_t* __restrict__ bag_ptr, int32_t bps,
       const int32_t* __restrict__ sample_ids, const int32_t* n_sel_dev, int32_t n_sel_max,
       float* __restrict__ out, eb_geom g, int64_t n_lookups, int64_t n_bags_total, int32_t n_samples,
       int32_t nbg, uint32_t* err, hl_hook hk) {
  hl_hook_head(hk);
  if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0 && bag_ptr[n_bags_total] != n_lookups)
    hl_flag(err, HL_DEVERR_SHAPE);
  // (thread 0, which carries the handover, is in the first row group of every block)
  eb_fwd_body<VEC, BF, PART>(blockIdx.x, gridDim.x, w_hot, stg, stg_rows, n_hot, k_cap, codes, bag_ptr, bps,
                             sample_ids, n_sel_dev, n_sel_max, out, g, n_samples, nbg, err);
  hl_hook_tail(hk);
}

// The forward of a one-hot mini-batch over every sample (as many lookups as
// bags: bag j is expected to hold lookup j alone), PART 0 or 1, wave by wave:
// a wave takes a unit of NG * OH_RPG consecutive bags (OH_RPG per row group,
// at most 256 bags), loads their offsets and codes one bag per lane and
// passes the codes to the row groups through LDS; when every bag of the unit
// holds exactly its own lookup, each row group issues its rows' loads all at
// once, then stores them, so a unit costs two dependent rounds of loads.  A
// unit with a bag that is not one-hot is pooled bag by bag as eb_fwd does.
// Same sums, same outputs: the row itself (PART 1: its hot rows only, zero
// for a staging row; zero for a code that names no row).
#define OH_RPG(VEC) ((VEC) >= 8 ? 8 : 16)  // rows per row group per unit (at most): up to 64 floats per lane in flight
#define OH_UNIT 256                // bags per unit (at most)
#define OH_MAXW (GT_THREADS / 64)

// The work of block bid of nblk (each of blockDim.x / 64 waves).
template <int VEC, bool BF, int PART>
__device__ __forceinline__ void eb_fwd_oh_body(uint32_t bid, uint32_t nblk, const void* w_hot_, const void* stg_,
                                               int32_t stg_rows, uint32_t n_hot, uint32_t k_cap,
                                               const int32_t* __restrict__ codes,
                                               const int32_t* __restrict__ bag_ptr, float* __restrict__ out,
                                               eb_geom g, int64_t n_lookups, int64_t n_bags, uint32_t* err) {
  static_assert(PART == 0 || PART == 1, "whole forward or its hot half");
  typedef typename RowIO<VEC, BF>::T T;
  __shared__ uint32_t s_code[OH_MAXW][OH_UNIT];
  const T* w_hot = (const T*)w_hot_;
  const T* stg = (const T*)stg_;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int gi = lane / g.G, gl = lane - gi * g.G;
  if (bid == 0 && blockIdx.y == 0 && threadIdx.x == 0 && bag_ptr[n_bags] != n_lookups)
    hl_flag(err, HL_DEVERR_SHAPE);
  const bool gact = gi < g.NG;
  const int32_t colv = blockIdx.y * 64 + gl;
  const bool cact = gact && colv < g.vpr;
  const int64_t col = (int64_t)colv * VEC;
  constexpr int RPG = OH_RPG(VEC);
  const int rpg = g.NG * RPG <= OH_UNIT ? RPG : OH_UNIT / g.NG;
  const int64_t ub = (int64_t)g.NG * rpg;  // bags per unit
  const int64_t units = (n_bags + ub - 1) / ub;
  uint32_t* sc = s_code[w];
  for (int64_t u = (int64_t)bid * nw + w; u < units; u += (int64_t)nblk * nw) {
    const int64_t b0 = u * ub;
    // offsets and codes, one bag per lane
    bool bad = false;
#pragma unroll
    for (int k = 0; k < OH_UNIT / 64; ++k) {
      const int64_t q = (int64_t)k * 64 + lane, b = b0 + q;
      if (q < ub && b < n_bags) {
        const int32_t lo = bag_ptr[b], hi = bag_ptr[b + 1];
        const uint32_t cu = (uint32_t)codes[b];
        sc[q] = cu;
        bad = bad || lo != b || hi != b + 1;
        if (!bad && !(cu < n_hot || (cu >= k_cap && cu - k_cap < (uint32_t)stg_rows))) hl_flag(err, HL_DEVERR_BAD_CODE);
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (__ballot(bad)) {
      // some bag of the unit is not one-hot: bag by bag, its hot rows then
      // (PART 0) its staging rows, in CSR order
      if (gact)
        for (int i = 0; i < rpg; ++i) {
          const int64_t b = b0 + (int64_t)gi * rpg + i;
          if (b >= n_bags) break;
          eb_bag<VEC, BF, PART>(out + b * g.D + col, w_hot, stg, stg_rows, n_hot, k_cap, codes, bag_ptr[b],
                                bag_ptr[b + 1], g, col, cact, gl, err);
        }
    } else if (gact) {
      float v[RPG][VEC];
#pragma unroll
      for (int i = 0; i < RPG; ++i) {
        const int64_t b = b0 + (int64_t)gi * rpg + i;
        const uint32_t cu = i < rpg ? sc[gi * rpg + i] : 0u;
        const bool in = i < rpg && b < n_bags && cact;
        const bool hot = cu < n_hot;
        const bool cold = PART == 0 && cu >= k_cap && cu - k_cap < (uint32_t)stg_rows;
        if (in && (hot || cold)) {
          const T* p = hot ? w_hot + (int64_t)cu * g.D : stg + (int64_t)(cu - k_cap) * g.D;
          RowIO<VEC, BF>::load(p + col, v[i]);
        } else {
#pragma unroll
          for (int e = 0; e < VEC; ++e) v[i][e] = 0.f;
        }
      }
#pragma unroll
      for (int i = 0; i < RPG; ++i) {
        const int64_t b = b0 + (int64_t)gi * rpg + i;
        if (i < rpg && b < n_bags && cact) st_f32_nt<VEC>(out + b * g.D + col, v[i]);
      }
    }
    // (the next unit's codes overwrite sc: every lane has read this one's)
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

template <int VEC, bool BF, int PART>
__global__ void __launch_bounds__(256)
eb_fwd_oh(const void* w_hot, const void* stg, int32_t stg_rows, uint32_t n_hot, uint32_t k_cap,
          const int32_t* __restrict__ codes, const int32_t* __restrict__ bag_ptr, float* __restrict__ out, eb_geom g,
          int64_t n_lookups, int64_t n_bags, uint32_t* err, hl_hook hk) {
  hl_hook_head(hk);
  // (thread 0, which carries the handover, is in the first row group of every block)
  eb_fwd_oh_body<VEC, BF, PART>(blockIdx.x, gridDim.x, w_hot, stg, stg_rows, n_hot, k_cap, codes, bag_ptr, out, g,
                                n_lookups, n_bags, err);
  hl_hook_tail(hk);
}

// The forward over every bag of a one-hot mini-batch and the backward's
// grouping in one launch: blocks [0, T) each sort a table (the grouping's
// second step, after gt_prep: gt_sort_body), the others pool the bags.  The
// sort reads the prep's keys and writes the grouping, the forward reads the
// codes and rows and writes the pooled outputs: nothing one writes is read by
// the other, so they run side by side (the sort on a few compute units at LDS
// and latency speed, the HBM-bound forward on the rest).
template <int VEC, bool BF, int ITEMS>
__global__ void __launch_bounds__(GT_THREADS)
eb_fwd_gt(const void* w_hot, const void* stg, int32_t stg_rows, uint32_t n_hot, uint32_t k_cap,
          const int32_t* __restrict__ codes, const int32_t* __restrict__ bag_ptr, float* __restrict__ out, eb_geom g,
          int64_t n_lookups, int64_t n_bags, const uint32_t* __restrict__ keys_tm, const uint32_t* __restrict__ cum,
          uint32_t nblk, uint32_t E, int32_t T, const uint32_t* __restrict__ tb, uint32_t* __restrict__ kout,
          uint32_t* __restrict__ vout, uint32_t* err, int ballot_only, hl_hook hk) {
  hl_hook_head(hk);
  if (blockIdx.x < (uint32_t)T) {
    gt_sort_body<ITEMS>(blockIdx.x, keys_tm, cum, nblk, E, T, (uint32_t)n_bags, tb, n_hot, kout, vout, err,
                        ballot_only);
  } else {
    eb_fwd_oh_body<VEC, BF, 0>(blockIdx.x - T, gridDim.x - T, w_hot, stg, stg_rows, n_hot, k_cap, codes, bag_ptr,
                               out, g, n_lookups, n_bags, err);
  }
}

// ----------------------------------------------------------------------------- backward
struct bw_ws {
  hl_sort_ws sort;
  uint8_t* mask;     // [max_bags]
  float* tfirst;     // [tiles][D]
  float* tlast;      // [tiles][D]
  uint32_t* tflag;   // [tiles]
  uint32_t* tkey;    // [tiles]
  float* gc;         // [n_max][D] gradient sums of staging rows, kept between the two halves of the apply
  uint32_t* bnd;     // [1] first sorted position whose key is not a hot slot (set by the first half)
  uint32_t tiles, gc_rows;
};

static uint32_t bw_tile_entries(int32_t D, int vec) {
  eb_geom g = eb_make_geom(D, vec);
  return (uint32_t)(RB_WAVES * g.NG * RB_EN(vec));
}

// compact: no staging-row sums (gc), for plans whose apply is whole (part 0)
static void bw_carve(hl_carver& c, bw_ws& ws, uint32_t n_max, int64_t max_bags, int32_t D, bool compact = false) {
  hl_sort_ws_carve(c, ws.sort, n_max);
  ws.mask = c.take<uint8_t>((size_t)max_bags + 1);
  // the smallest tile (largest count) over the vector widths the call may pick
  uint32_t te = bw_tile_entries(D, 1);
  uint32_t te2 = bw_tile_entries(D, D % 2 == 0 ? 2 : 1), te4 = bw_tile_entries(D, D % 4 == 0 ? 4 : 1);
  te = te < te2 ? te : te2;
  te = te < te4 ? te : te4;
  ws.tiles = n_max ? hl_div_up(n_max, te) : 1;
  ws.tfirst = c.take<float>((size_t)ws.tiles * D);
  ws.tlast = c.take<float>((size_t)ws.tiles * D);
  ws.tflag = c.take<uint32_t>(ws.tiles);
  ws.tkey = c.take<uint32_t>(ws.tiles);
  ws.gc_rows = compact ? 0 : n_max;
  ws.gc = c.take<float>((size_t)ws.gc_rows * D);
  ws.bnd = c.take<uint32_t>(1);
}

size_t hl_bwd_ws_bytes(const hl_handle* h, int64_t max_lookups, int64_t max_bags) {
  hl_carver c = hl_carver::after_header(nullptr, 0);
  bw_ws ws;
  bw_carve(c, ws, (uint32_t)max_lookups, max_bags, h->dim);
  return c.off;
}

size_t hl_bwd_ws_bytes_compact(const hl_handle* h, int64_t max_lookups, int64_t max_bags) {
  hl_carver c = hl_carver::after_header(nullptr, 0);
  bw_ws ws;
  bw_carve(c, ws, (uint32_t)max_lookups, max_bags, h->dim, true);
  return c.off;
}

static size_t bw_bytes(const hl_handle* h, int64_t n, int64_t bags, bool compact) {
  return compact ? hl_bwd_ws_bytes_compact(h, n, bags) : hl_bwd_ws_bytes(h, n, bags);
}

__global__ void bw_mask(uint8_t* mask, int32_t n_samples, const int32_t* __restrict__ ids, const int32_t* n_dev,
                        int32_t n_max, int phase) {
  if (phase == 0) {
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n_samples; i += gridDim.x * blockDim.x) mask[i] = 0;
  } else {
    const int32_t n = eb_nsel(ids, n_dev, n_max);
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
      const int32_t s = ids[i];
      if (s >= 0 && s < n_samples) mask[s] = 1;
    }
  }
}

// (compressed key, bag) for every lookup of the mini-batch; lookups of
// unselected samples and invalid codes get the sentinel key (sorted last,
// ignored), and so do positions outside [bag_ptr[0], bag_ptr[n_bags]) (only if
// bag_ptr disagrees with n_lookups; bag_ptr is non-decreasing).

// the lookup positions no bag covers: [0, bag_ptr[0]) and [bag_ptr[n_bags], n)
__device__ __forceinline__ void bw_uncovered(const int32_t* bag_ptr, int64_t n_bags, int64_t n_lookups,
                                             int64_t* first, int64_t* covered) {
  *first = min((int64_t)max(bag_ptr[0], 0), n_lookups);
  *covered = max(min((int64_t)max(bag_ptr[n_bags], 0), n_lookups), *first);
}


// the bags [b0, b0 + nb) of one block: off[] holds their offsets.  The fused
// plan (cf.table) also writes the cold lookups' codes and frees their slots,
// as the cold plan's last kernel does.
template <int NT>
__device__ __forceinline__ void bw_prep_bags(int32_t* codes, const int32_t* off, int64_t b0, int nb, int32_t bps,
                                             const uint8_t* __restrict__ mask, uint32_t n_hot, uint32_t k_cap,
                                             int32_t stg_rows, uint32_t* __restrict__ keys,
                                             uint32_t* __restrict__ vals, int64_t n_lookups, uint32_t* err,
                                             const hl_cg_fused& cf, bool fits) {
  const int32_t lo = off[0], hi = min((int64_t)off[nb], n_lookups);
  for (int32_t i = lo + threadIdx.x; i < hi; i += NT) {
    int a = 0, b = nb;
    while (b - a > 1) {
      int m = (a + b) >> 1;
      if (off[m] <= i) a = m; else b = m;
    }
    const int64_t bag = b0 + a;
    uint32_t key = EB_SENT;
    if (!mask || mask[bag / bps]) {
      int32_t c = codes[i];
      if (cf.table && c == -1) {
        const uint32_t sl = cf.slotof[i];
        c = bw_fused_code(c, (uint32_t)i, cf, k_cap, fits);
        if (c != -1) codes[i] = c;
        if (sl < cf.S) cf.table[sl] = 0;
      }
      key = bw_key((uint32_t)c, n_hot, k_cap, stg_rows);
      if (key == EB_SENT) hl_flag(err, HL_DEVERR_BAD_CODE);
    }
    keys[i] = key;
    vals[i] = (uint32_t)bag;
  }
}


#define BP_BAGS 256
__global__ void __launch_bounds__(256)
bw_prep(const int32_t* __restrict__ codes, const int32_t* __restrict__ bag_ptr, int64_t n_bags, int32_t bps,
        const uint8_t* __restrict__ mask, uint32_t n_hot, uint32_t k_cap, int32_t stg_rows,
        uint32_t* __restrict__ keys, uint32_t* __restrict__ vals, int64_t n_lookups, uint32_t* sflag, uint32_t sv,
        uint32_t* err) {
  __shared__ int32_t off[BP_BAGS + 1];
  bw_start_signal(sflag, sv);
  const int64_t b0 = (int64_t)blockIdx.x * BP_BAGS;
  const int nb = (int)min((int64_t)BP_BAGS, n_bags - b0);
  for (int j = threadIdx.x; j <= nb; j += blockDim.x) off[j] = bag_ptr[b0 + j];
  if (blockIdx.x == 0 && threadIdx.x == 0 && bag_ptr[n_bags] != n_lookups) hl_flag(err, HL_DEVERR_SHAPE);
  __syncthreads();
  int64_t first, covered;
  bw_uncovered(bag_ptr, n_bags, n_lookups, &first, &covered);
  const int64_t gs = (int64_t)gridDim.x * blockDim.x, t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (int64_t i = t0; i < first; i += gs) keys[i] = EB_SENT;
  for (int64_t i = covered + t0; i < n_lookups; i += gs) keys[i] = EB_SENT;
  bw_prep_bags<256>(const_cast<int32_t*>(codes), off, b0, nb, bps, mask, n_hot, k_cap, stg_rows, keys, vals,
                    n_lookups, err, hl_cg_fused{}, false);
}

// bw_prep and the sort's digit histogram in one launch (no sample selection):
// blocks [0, hb) count the digits of every key, taking the keys from the codes
// by the same rule as the writers, and clear the first pass's status words;
// the other blocks write the (key, bag) pairs, bpb bags each (at most
// BPH_BAGS: fewer when bags hold many lookups, so the writers spread over
// the chip).  In the
// fused plan (cf.table) both roles take a cold lookup's code from the cold
// plan's state (the writers also store it; a reader that meets the stored
// code derives the same key), and the first writer block reports rows that do
// not fit the staging buffer.
#define BPH_THREADS 1024
#define BPH_BAGS 1024
template <int NB>
__global__ void __launch_bounds__(BPH_THREADS)
bw_prep_hist(int32_t* codes, const int32_t* __restrict__ bag_ptr, int64_t n_bags, int32_t bps, uint32_t n_hot,
             uint32_t k_cap, int32_t stg_rows, uint32_t* __restrict__ keys, uint32_t* __restrict__ vals,
             int64_t n_lookups, uint32_t hb, int passes, int b, uint32_t* __restrict__ part,
             uint32_t* __restrict__ zero, uint64_t n_zero, int32_t bpb, uint32_t* sflag, uint32_t sv, uint32_t* err,
             hl_cg_fused cf) {
  __shared__ uint32_t hst[HL_SORT_MAXPASS][NB];
  __shared__ int32_t off[BPH_BAGS + 1];
  bw_start_signal(sflag, sv);
  int64_t first, covered;
  bw_uncovered(bag_ptr, n_bags, n_lookups, &first, &covered);
  const bool fits = cf.table && *cf.ncold <= (uint32_t)cf.cap;
  if (blockIdx.x < hb) {
    const uint32_t gs = hb * BPH_THREADS;
    for (uint64_t i = (uint64_t)blockIdx.x * BPH_THREADS + threadIdx.x; i < n_zero; i += gs) zero[i] = 0;
    for (int j = threadIdx.x; j < HL_SORT_MAXPASS * NB; j += BPH_THREADS) (&hst[0][0])[j] = 0;
    __syncthreads();
    const uint32_t mask = (1u << b) - 1u;
    const uint32_t n = (uint32_t)n_lookups;
    for (uint32_t i0 = blockIdx.x * BPH_THREADS + threadIdx.x; i0 < n; i0 += 8 * gs) {
      uint32_t k[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const uint32_t i = i0 + u * gs;
        k[u] = i < n ? (uint32_t)codes[i] : 0u;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const uint32_t i = i0 + u * gs;
        if (i >= n) continue;
        const uint32_t c = (uint32_t)bw_fused_code((int32_t)k[u], i, cf, k_cap, fits);
        const uint32_t key = (int64_t)i < first || (int64_t)i >= covered ? EB_SENT : bw_key(c, n_hot, k_cap, stg_rows);
        for (int p = 0; p < passes; ++p) atomicAdd(&hst[p][(key >> (b * p)) & mask], 1u);
      }
    }
    __syncthreads();
    for (int p = 0; p < passes; ++p)
      for (int j = threadIdx.x; j < NB; j += BPH_THREADS)
        part[((size_t)p * HL_SORT_HIST_BLOCKS + blockIdx.x) * NB + j] = hst[p][j];
    return;
  }
  const uint32_t blk = blockIdx.x - hb;
  const int64_t b0 = (int64_t)blk * bpb;
  const int nb = (int)min((int64_t)bpb, n_bags - b0);
  for (int j = threadIdx.x; j <= nb; j += BPH_THREADS) off[j] = bag_ptr[b0 + j];
  if (blk == 0 && threadIdx.x == 0 && bag_ptr[n_bags] != n_lookups) hl_flag(err, HL_DEVERR_SHAPE);
  if (blk == 0 && threadIdx.x == 0 && cf.table && !fits) hl_flag(err, HL_DEVERR_CAPACITY);
  __syncthreads();
  const int64_t gs = (int64_t)(gridDim.x - hb) * BPH_THREADS, t0 = (int64_t)blk * BPH_THREADS + threadIdx.x;
  for (int64_t i = t0; i < first; i += gs) keys[i] = EB_SENT;
  for (int64_t i = covered + t0; i < n_lookups; i += gs) keys[i] = EB_SENT;
  bw_prep_bags<BPH_THREADS>(codes, off, b0, nb, bps, nullptr, n_hot, k_cap, stg_rows, keys, vals, n_lookups, err, cf,
                            fits);
}

template <int VEC, bool BF>
__device__ __forceinline__ typename RowIO<VEC, BF>::T* bw_row(void* w_hot, void* stg, uint32_t n_hot, int32_t D,
                                                             uint32_t key) {
  typedef typename RowIO<VEC, BF>::T T;
  return key < n_hot ? (T*)w_hot + (int64_t)key * D : (T*)stg + (int64_t)(key - n_hot) * D;
}

#define GF_F 1u
#define GF_W 2u
#define GF_L 4u

// SPLIT: the run of a staging row (key n_hot + u, u < gc_rows) stores its sum
// G in gc[u] instead of updating the row, and the row is not read; bw_cold
// applies it later (the staging rows may still be in flight then).
__device__ __forceinline__ bool bw_deferred(uint32_t key, uint32_t n_hot, uint32_t gc_rows) {
  return key >= n_hot && key != EB_SENT && key - n_hot < gc_rows;
}

template <int VEC, bool BF, bool SPLIT>
__global__ void __launch_bounds__(RB_BLOCK)
bw_reduce1(const uint32_t* __restrict__ keys, const uint32_t* __restrict__ vals, uint32_t n,
           const float* __restrict__ dY, eb_geom g, void* w_hot, void* stg, uint32_t n_hot, float lr,
           float* __restrict__ tfirst, float* __restrict__ tlast, uint32_t* __restrict__ tflag,
           uint32_t* __restrict__ tkey, float* __restrict__ gc, uint32_t gc_rows, uint32_t* __restrict__ bnd,
           hl_hook hk) {
  typedef typename RowIO<VEC, BF>::T T;
  constexpr int RB_E = RB_EN(VEC);
  __shared__ float pf[RB_WAVES * 64 * VEC], pl[RB_WAVES * 64 * VEC];
  hl_hook_head(hk);
  __shared__ uint32_t gflag[RB_WAVES * 64], gkey[RB_WAVES * 64];
  __shared__ uint32_t s_tflag;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int gi = lane / g.G, gl = lane - gi * g.G;
  const bool gact = gi < g.NG;
  const int grp = w * g.NG + gi;           // group index inside the block
  const int ngb = RB_WAVES * g.NG;         // groups per block
  const uint32_t te = (uint32_t)ngb * RB_E;
  const uint32_t tile = blockIdx.x;
  const uint64_t tb = (uint64_t)tile * te;
  const int32_t colv = blockIdx.y * 64 + gl;
  const bool cact = gact && colv < g.vpr;
  const int64_t col = (int64_t)colv * VEC;
  const int lds_off = (grp * g.G + gl) * VEC;
  if (threadIdx.x == 0) s_tflag = 0;
  if (gact) {
    const uint64_t e0 = tb + (uint64_t)grp * RB_E;
    uint32_t kk[RB_E], bb[RB_E];
#pragma unroll
    for (int j = 0; j < RB_E; ++j) {
      const uint64_t idx = e0 + j;
      kk[j] = idx < n ? keys[idx] : EB_SENT;
      bb[j] = idx < n ? vals[idx] : 0u;
    }
    const uint32_t prevk = (e0 > 0 && e0 - 1 < n) ? keys[e0 - 1] : EB_SENT;
    const uint32_t nextk = (e0 + RB_E < n) ? keys[e0 + RB_E] : EB_SENT;
    if (SPLIT && blockIdx.y == 0 && gl == 0) {
      // the one position where the hot slots end (keys are sorted; n if they never do)
#pragma unroll
      for (int j = 0; j < RB_E; ++j) {
        const uint64_t idx = e0 + j;
        const uint32_t kp = j == 0 ? (e0 > 0 ? prevk : 0u) : kk[j - 1];
        if (idx < n && kk[j] >= n_hot && (idx == 0 || kp < n_hot)) *bnd = (uint32_t)idx;
        if (idx + 1 == n && kk[j] < n_hot) *bnd = (uint32_t)n;
      }
    }
    const bool cprev = kk[0] != EB_SENT && prevk == kk[0];
    const bool cnext = kk[RB_E - 1] != EB_SENT && nextk == kk[RB_E - 1];
    // gradient rows
    float dv[RB_E][VEC];
#pragma unroll
    for (int j = 0; j < RB_E; ++j) {
      if (kk[j] != EB_SENT && cact) ld_f32<VEC>(dY + (int64_t)bb[j] * g.D + col, dv[j]);
      else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) dv[j][e] = 0.f;
      }
    }
    // rows of complete runs (issued before the sums are formed)
    typename RowIO<VEC, BF>::Raw wr[RB_E];
    bool cpl[RB_E];
    bool from0 = true;
#pragma unroll
    for (int j = 0; j < RB_E; ++j) {
      const bool valid = kk[j] != EB_SENT;
      if (j > 0 && valid && kk[j - 1] != kk[j]) from0 = false;
      const bool end = valid && (j == RB_E - 1 || kk[j + 1] != kk[j]);
      cpl[j] = end && !(from0 && cprev) && !(j == RB_E - 1 && cnext);
      if (cpl[j] && cact && !(SPLIT && bw_deferred(kk[j], n_hot, gc_rows)))
        wr[j] = RowIO<VEC, BF>::load_raw(bw_row<VEC, BF>(w_hot, stg, n_hot, g.D, kk[j]) + col);
    }
    float acc[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] = 0.f;
    uint32_t gf = 0;
    from0 = true;
#pragma unroll
    for (int j = 0; j < RB_E; ++j) {
      const bool valid = kk[j] != EB_SENT;
      if (j > 0 && valid && kk[j - 1] != kk[j]) from0 = false;
      if (valid) {
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[e] += dv[j][e];
      }
      const bool end = valid && (j == RB_E - 1 || kk[j + 1] != kk[j]);
      if (end) {
        if (cpl[j]) {
          if (cact) {
            if (SPLIT && bw_deferred(kk[j], n_hot, gc_rows)) {
              st_f32<VEC>(gc + (int64_t)(kk[j] - n_hot) * g.D + col, acc);
            } else {
              float wv[VEC], nw[VEC];
              RowIO<VEC, BF>::unpack(wr[j], wv);
#pragma unroll
              for (int e = 0; e < VEC; ++e) nw[e] = wv[e] - lr * acc[e];
              RowIO<VEC, BF>::store(bw_row<VEC, BF>(w_hot, stg, n_hot, g.D, kk[j]) + col, nw);
            }
          }
        } else {
          const bool first = from0 && cprev, lastp = (j == RB_E - 1) && cnext;
          if (first) {
            gf |= GF_F | (lastp ? GF_W | GF_L : 0u);
#pragma unroll
            for (int e = 0; e < VEC; ++e) pf[lds_off + e] = acc[e];
          } else if (lastp) {
            gf |= GF_L;
#pragma unroll
            for (int e = 0; e < VEC; ++e) pl[lds_off + e] = acc[e];
          }
        }
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[e] = 0.f;
      }
    }
    if (gl == 0) {
      gflag[grp] = gf;
      gkey[grp] = kk[RB_E - 1];
    }
  }
  __syncthreads();
  if (gact) {
    const uint32_t gf = gflag[grp];
    // a segment that starts in this group and continues into the next ones
    if ((gf & GF_L) && !(gf & GF_W)) {
      float acc[VEC];
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] = pl[lds_off + e];
      bool done = false;
      for (int g2 = grp + 1; g2 < ngb; ++g2) {
        const int o2 = (g2 * g.G + gl) * VEC;
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[e] += pf[o2 + e];
        if (!(gflag[g2] & GF_W)) { done = true; break; }
      }
      const uint32_t key = gkey[grp];
      if (done) {
        if (cact && SPLIT && bw_deferred(key, n_hot, gc_rows)) {
          st_f32<VEC>(gc + (int64_t)(key - n_hot) * g.D + col, acc);
        } else if (cact) {
          T* p = bw_row<VEC, BF>(w_hot, stg, n_hot, g.D, key) + col;
          float wv[VEC];
          RowIO<VEC, BF>::load(p, wv);
#pragma unroll
          for (int e = 0; e < VEC; ++e) wv[e] -= lr * acc[e];
          RowIO<VEC, BF>::store(p, wv);
        }
      } else {
        if (cact) st_f32<VEC>(tlast + (int64_t)tile * g.D + col, acc);
        if (gl == 0) {
          atomicOr(&s_tflag, GF_L);
          if (blockIdx.y == 0) tkey[tile] = key;
        }
      }
    }
    // the piece of a segment that began in an earlier tile
    if (grp == 0 && (gf & GF_F)) {
      float acc[VEC];
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] = pf[lds_off + e];
      bool whole = (gf & GF_W) != 0;
      if (whole) {
        for (int g2 = 1; g2 < ngb; ++g2) {
          const int o2 = (g2 * g.G + gl) * VEC;
#pragma unroll
          for (int e = 0; e < VEC; ++e) acc[e] += pf[o2 + e];
          if (!(gflag[g2] & GF_W)) { whole = false; break; }
        }
      }
      if (cact) st_f32<VEC>(tfirst + (int64_t)tile * g.D + col, acc);
      if (gl == 0) atomicOr(&s_tflag, GF_F | (whole ? GF_W : 0u));
    }
  }
  __syncthreads();
  if (threadIdx.x == 0 && blockIdx.y == 0) tflag[tile] = s_tflag;
  hl_hook_tail(hk);
}

// Segments spanning tiles: the tile where a segment starts (flag L) sums its
// own piece and the next tiles' first pieces up to the first tile that is not
// wholly inside the segment.  Piece p is summed by group p % groups in
// ascending p, then groups are added in order.  The loads that need nothing
// but the tile index (its flag, key and piece, the next tiles' flags) are
// issued together, and the row with the pieces of the later tiles, so a
// segment takes two dependent rounds of loads.
template <int VEC, bool BF, bool SPLIT>
__device__ __forceinline__ void bw_reduce2_body(uint32_t t, uint32_t n_tiles, eb_geom g, void* w_hot, void* stg,
                                                uint32_t n_hot, float lr, const float* __restrict__ tfirst,
                                                const float* __restrict__ tlast, const uint32_t* __restrict__ tflag,
                                                const uint32_t* __restrict__ tkey, float* __restrict__ gc,
                                                uint32_t gc_rows) {
  typedef typename RowIO<VEC, BF>::T T;
  __shared__ uint32_t s_end;
  __shared__ float part[RB_WAVES * 64 * VEC];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int gi = lane / g.G, gl = lane - gi * g.G;
  const bool gact = gi < g.NG;
  const int grp = w * g.NG + gi, ngb = RB_WAVES * g.NG;
  const int32_t colv = blockIdx.y * 64 + gl;
  const bool cact = gact && colv < g.vpr;
  const int64_t col = (int64_t)colv * VEC;
  const uint32_t f = tflag[t];
  const uint32_t key = tkey[t];
  const uint32_t t2 = t + 1 + threadIdx.x;
  const uint32_t f2 = t2 < n_tiles ? tflag[t2] : GF_W;
  float v0[VEC];  // piece 0 (this tile's), summed by group 0
#pragma unroll
  for (int e = 0; e < VEC; ++e) v0[e] = 0.f;
  if (grp == 0 && cact) ld_f32<VEC>(tlast + (int64_t)t * g.D + col, v0);
  if (threadIdx.x == 0) s_end = n_tiles;
  __syncthreads();
  if (!(f & GF_L)) return;  // (the same for every thread of the block)
  // the row, for group 0 (its address needs only the key)
  const bool defer = SPLIT && bw_deferred(key, n_hot, gc_rows);
  float wv[VEC];
  T* rp = bw_row<VEC, BF>(w_hot, stg, n_hot, g.D, key) + col;
  if (grp == 0 && cact && !defer) RowIO<VEC, BF>::load(rp, wv);
  // the first tile after t that is not wholly inside the segment holds its
  // last piece (a window of RB_BLOCK tiles at a time)
  if (!(f2 & GF_W)) atomicMin(&s_end, t2);
  __syncthreads();
  uint32_t tend = s_end;
  for (uint32_t base = t + 1 + RB_BLOCK; tend == n_tiles && base < n_tiles; base += RB_BLOCK) {
    const uint32_t t3 = base + threadIdx.x;
    if (t3 < n_tiles && !(tflag[t3] & GF_W)) atomicMin(&s_end, t3);
    __syncthreads();
    tend = s_end;
  }
  const uint32_t npieces = (tend < n_tiles ? tend : n_tiles - 1) - t + 1;
  if (gact) {
    float acc[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] = 0.f;
    if (grp == 0)
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] += v0[e];
    if (cact) {
      // (four pieces in flight, added in ascending order)
      for (uint32_t p = grp == 0 ? ngb : grp; p < npieces; p += 4 * ngb) {
        float v[4][VEC];
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (p + i * ngb < npieces) ld_f32<VEC>(tfirst + (int64_t)(t + p + i * ngb) * g.D + col, v[i]);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (p + i * ngb < npieces)
#pragma unroll
            for (int e = 0; e < VEC; ++e) acc[e] += v[i][e];
      }
    }
#pragma unroll
    for (int e = 0; e < VEC; ++e) part[(grp * g.G + gl) * VEC + e] = acc[e];
  }
  __syncthreads();
  if (gact && grp == 0 && cact) {
    float acc[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] = 0.f;
    for (int q = 0; q < ngb; ++q)
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] += part[(q * g.G + gl) * VEC + e];
    if (defer) {
      st_f32<VEC>(gc + (int64_t)(key - n_hot) * g.D + col, acc);
      return;
    }
#pragma unroll
    for (int e = 0; e < VEC; ++e) wv[e] -= lr * acc[e];
    RowIO<VEC, BF>::store(rp, wv);
  }
}

template <int VEC, bool BF, bool SPLIT>
__global__ void __launch_bounds__(RB_BLOCK)
bw_reduce2(uint32_t n_tiles, eb_geom g, void* w_hot, void* stg, uint32_t n_hot, float lr,
           const float* __restrict__ tfirst, const float* __restrict__ tlast, const uint32_t* __restrict__ tflag,
           const uint32_t* __restrict__ tkey, float* __restrict__ gc, uint32_t gc_rows) {
  bw_reduce2_body<VEC, BF, SPLIT>(blockIdx.x, n_tiles, g, w_hot, stg, n_hot, lr, tfirst, tlast, tflag, tkey, gc,
                                  gc_rows);
}

// The deferred staging-row updates: every run end in the sorted keys whose key
// is a staging row below gc_rows applies row <- round(row - lr * gc[u]), the
// same arithmetic as the one-pass update.  Only the sorted tail from *bnd (the
// end of the hot slots, found by the first half) is scanned.  A wave tests
// CW_POS positions at a time (one per lane), then its row groups take the run
// ends found, each group its share at once (at most CW_POS / NG rows per
// group, all loads in flight together), so a wave's positions cost one round
// of row loads.
#define CW_POS 16
template <int VEC, bool BF>
__global__ void __launch_bounds__(256)
bw_cold(const uint32_t* __restrict__ keys, uint32_t n, eb_geom g, void* stg, uint32_t n_hot, float lr,
        const float* __restrict__ gc, uint32_t gc_rows, const uint32_t* __restrict__ bnd, hl_hook hk) {
  typedef typename RowIO<VEC, BF>::T T;
  hl_hook_head(hk);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int gi = lane / g.G, gl = lane - gi * g.G;
  const int32_t colv = blockIdx.y * 64 + gl;
  const bool cact = gi < g.NG && colv < g.vpr;
  const int64_t col = (int64_t)colv * VEC;
  const uint32_t b0 = min(*bnd, n);
  constexpr int RPG = CW_POS / 4 > 0 ? CW_POS / 4 : 1;  // rows per group for groups of 16 lanes or wider
  for (uint64_t base = b0 + ((uint64_t)blockIdx.x * 4 + w) * CW_POS; base < n;
       base += (uint64_t)gridDim.x * 4 * CW_POS) {
    const uint64_t p = base + lane;
    const bool in = lane < CW_POS && p < n;
    const uint32_t k = in ? keys[p] : EB_SENT;
    const uint32_t kn = in && p + 1 < n ? keys[p + 1] : EB_SENT;
    uint64_t m = __ballot(in && k != kn && bw_deferred(k, n_hot, gc_rows));
    while (m) {
      // run end gi + NG j of the remaining ones goes to group gi
      uint64_t mm = m;
      for (int q = 0; q < gi; ++q) mm &= mm - 1;
      int src[RPG];
      bool has[RPG];
#pragma unroll
      for (int j = 0; j < RPG; ++j) {
        has[j] = mm != 0;
        src[j] = has[j] ? __ffsll((unsigned long long)mm) - 1 : 0;
        for (int q = 0; q < g.NG && mm; ++q) mm &= mm - 1;
      }
      int64_t u[RPG];
      float wv[RPG][VEC], gv[RPG][VEC];
#pragma unroll
      for (int j = 0; j < RPG; ++j) {
        u[j] = (int64_t)__shfl(k, src[j]) - n_hot;
        if (has[j] && cact) {
          RowIO<VEC, BF>::load((T*)stg + u[j] * g.D + col, wv[j]);
          ld_f32<VEC>(gc + u[j] * g.D + col, gv[j]);
        }
      }
#pragma unroll
      for (int j = 0; j < RPG; ++j)
        if (has[j] && cact) {
#pragma unroll
          for (int e = 0; e < VEC; ++e) wv[j][e] = wv[j][e] - lr * gv[j][e];
          RowIO<VEC, BF>::store((T*)stg + u[j] * g.D + col, wv[j]);
        }
      for (int q = 0; q < RPG * g.NG && m; ++q) m &= m - 1;
    }
  }
  hl_hook_tail(hk);
}

// The cold half of the forward from the backward's grouping: the sorted tail
// from *bnd holds a (staging key, bag) pair for every cold lookup.  A bag is
// completed by the pair of its first cold lookup in CSR order (the first copy
// of that pair): out[bag] += its staging rows in CSR order, the same sums as
// the forward's cold half over the non-popular mu-batch.  A group of lanes
// takes FT pairs at once.
#define FT 4
// (block bid of nblk, WAVES waves per block)
template <int VEC, bool BF, int WAVES>
__device__ __forceinline__ void eb_tail_body(uint32_t bid, uint32_t nblk, const uint32_t* __restrict__ keys,
                                             const uint32_t* __restrict__ vals, uint32_t n,
                                             const uint32_t* __restrict__ bnd, eb_geom g, const void* stg_,
                                             int32_t stg_rows, uint32_t n_hot, uint32_t k_cap,
                                             const int32_t* __restrict__ codes, const int32_t* __restrict__ bag_ptr,
                                             float* __restrict__ out, uint32_t* err) {
  typedef typename RowIO<VEC, BF>::T T;
  const T* stg = (const T*)stg_;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int gi = lane / g.G, gl = lane - gi * g.G;
  if (gi >= g.NG) return;
  const int32_t colv = blockIdx.y * 64 + gl;
  const bool cact = colv < g.vpr;
  const int64_t col = (int64_t)colv * VEC;
  const uint32_t b0 = min(*bnd, n);
  const uint64_t stride = (uint64_t)nblk * WAVES * g.NG * FT;
  for (uint64_t p0 = b0 + ((uint64_t)(bid * WAVES + w) * g.NG + gi) * FT; p0 < n; p0 += stride) {
    uint32_t key[FT], bag[FT];
    bool take[FT];
#pragma unroll
    for (int j = 0; j < FT; ++j) {
      const uint64_t p = p0 + j;
      key[j] = p < n ? keys[p] : EB_SENT;
      bag[j] = p < n ? vals[p] : 0u;
      const uint32_t kp = p > b0 && p < n ? keys[p - 1] : EB_SENT;
      const uint32_t bp = p > b0 && p < n ? vals[p - 1] : 0u;
      take[j] = key[j] != EB_SENT && key[j] >= n_hot && key[j] - n_hot < (uint32_t)stg_rows &&
                !(kp == key[j] && bp == bag[j]);
    }
    int32_t lo[FT], hi[FT];
#pragma unroll
    for (int j = 0; j < FT; ++j) {
      lo[j] = take[j] ? bag_ptr[bag[j]] : 0;
      hi[j] = take[j] ? bag_ptr[bag[j] + 1] : 0;
    }
#pragma unroll
    for (int j = 0; j < FT; ++j) {
      if (!take[j]) continue;
      const uint32_t u = key[j] - n_hot;
      if (hi[j] - lo[j] != 1) {
        // the bag's first cold lookup in CSR order names the pair that completes
        // it (row groups of 8 lanes or more search G codes at a time: a code
        // per lane, the first cold one by a ballot)
        bool mine = false;
        if (g.G >= EB_SEG_ROWS) {
          const int g0 = lane - gl;
          const uint64_t gm = g.G == 64 ? ~0ull : ((1ull << g.G) - 1ull);
          for (int32_t b0 = lo[j]; b0 < hi[j]; b0 += g.G) {
            const int32_t i = b0 + gl;
            const uint32_t c = i < hi[j] ? (uint32_t)codes[i] : ~0u;
            const bool cold = i < hi[j] && c >= k_cap && c - k_cap < (uint32_t)stg_rows;
            const uint64_t m = (__ballot(cold) >> g0) & gm;
            if (m) {
              const uint32_t cf = (uint32_t)__shfl((int)c, g0 + __ffsll((unsigned long long)m) - 1);
              mine = cf - k_cap == u;
              break;
            }
          }
        } else {
          for (int32_t i = lo[j]; i < hi[j]; ++i) {
            const uint32_t c = (uint32_t)codes[i];
            if (c >= k_cap && c - k_cap < (uint32_t)stg_rows) {
              mine = c - k_cap == u;
              break;
            }
          }
        }
        if (!mine) take[j] = false;
      }
    }
    float o[FT][VEC], v[FT][VEC];
#pragma unroll
    for (int j = 0; j < FT; ++j)
      if (take[j] && cact) {
        ld_f32<VEC>(out + (int64_t)bag[j] * g.D + col, o[j]);
        if (hi[j] - lo[j] == 1) RowIO<VEC, BF>::load(stg + (int64_t)(key[j] - n_hot) * g.D + col, v[j]);
      }
#pragma unroll
    for (int j = 0; j < FT; ++j) {
      if (!take[j]) continue;
      if (hi[j] - lo[j] == 1) {
        if (cact) {
#pragma unroll
          for (int e = 0; e < VEC; ++e) o[j][e] += v[j][e];
        }
      } else {
        // the staging rows' sum, onto the stored hot sum (as PART 2 of the forward adds it)
        float c[VEC];
#pragma unroll
        for (int e = 0; e < VEC; ++e) c[e] = 0.f;
        bool anyc = false;
        eb_pass<VEC, BF, true>(c, nullptr, stg, stg_rows, n_hot, k_cap, codes, lo[j], hi[j], g, col, cact, gl, err,
                               &anyc);
#pragma unroll
        for (int e = 0; e < VEC; ++e) o[j][e] += c[e];
      }
      if (cact) st_f32<VEC>(out + (int64_t)bag[j] * g.D + col, o[j]);
    }
  }
}

template <int VEC, bool BF>
__global__ void __launch_bounds__(256)
eb_fwd_tail(const uint32_t* __restrict__ keys, const uint32_t* __restrict__ vals, uint32_t n,
            const uint32_t* __restrict__ bnd, eb_geom g, const void* stg_, int32_t stg_rows, uint32_t n_hot,
            uint32_t k_cap, const int32_t* __restrict__ codes, const int32_t* __restrict__ bag_ptr,
            float* __restrict__ out, uint32_t* err) {
  eb_tail_body<VEC, BF, 4>(blockIdx.x, gridDim.x, keys, vals, n, bnd, g, stg_, stg_rows, n_hot, k_cap, codes, bag_ptr,
                           out, err);
}

// The cold half of the forward and the backward's segments that span tiles
// (bw_reduce2, split form) in one launch: blocks [0, n_tiles) take the
// segments, the others the sorted tail.  They share no data (the segments
// write hot rows and staging-row sums, the tail reads staging rows and
// writes pooled outputs).
template <int VEC, bool BF>
__global__ void __launch_bounds__(RB_BLOCK)
eb_tail_r2(uint32_t n_tiles, void* w_hot, uint32_t n_hot, float lr, const float* __restrict__ tfirst,
           const float* __restrict__ tlast, const uint32_t* __restrict__ tflag, const uint32_t* __restrict__ tkey,
           float* __restrict__ gc, uint32_t gc_rows, const uint32_t* __restrict__ keys,
           const uint32_t* __restrict__ vals, uint32_t n, const uint32_t* __restrict__ bnd, eb_geom g, void* stg,
           int32_t stg_rows, uint32_t k_cap, const int32_t* __restrict__ codes, const int32_t* __restrict__ bag_ptr,
           float* __restrict__ out, uint32_t* err) {
  if (blockIdx.x < n_tiles) {
    bw_reduce2_body<VEC, BF, true>(blockIdx.x, n_tiles, g, w_hot, stg, n_hot, lr, tfirst, tlast, tflag, tkey, gc,
                                   gc_rows);
    return;
  }
  eb_tail_body<VEC, BF, RB_WAVES>(blockIdx.x - n_tiles, gridDim.x - n_tiles, keys, vals, n, bnd, g, stg, stg_rows,
                                  n_hot, k_cap, codes, bag_ptr, out, err);
}

// The same launch for bags of several lookups (multi-hot), where nearly every
// bag holds a staging row: the cold half of the forward bag by bag (part 2 of
// the forward over every bag, one bag per row group) in place of the sorted
// tail.
template <int VEC, bool BF>
__global__ void __launch_bounds__(RB_BLOCK)
eb_bags_r2(uint32_t n_tiles, void* w_hot, uint32_t n_hot, float lr, const float* __restrict__ tfirst,
           const float* __restrict__ tlast, const uint32_t* __restrict__ tflag, const uint32_t* __restrict__ tkey,
           float* __restrict__ gc, uint32_t gc_rows, eb_geom g, void* stg, int32_t stg_rows, uint32_t k_cap,
           const int32_t* __restrict__ codes, const int32_t* __restrict__ bag_ptr, int32_t bps, int32_t n_samples,
           float* __restrict__ out, uint32_t* err) {
  if (blockIdx.x < n_tiles) {
    bw_reduce2_body<VEC, BF, true>(blockIdx.x, n_tiles, g, w_hot, stg, n_hot, lr, tfirst, tlast, tflag, tkey, gc,
                                   gc_rows);
    return;
  }
  eb_fwd_body<VEC, BF, 2>(blockIdx.x - n_tiles, gridDim.x - n_tiles, w_hot, stg, stg_rows, n_hot, k_cap, codes,
                          bag_ptr, bps, nullptr, nullptr, n_samples, out, g, n_samples, 1, err);
}

// ----------------------------------------------------------------------------- host side
static hl_status check_common(const hl_handle* h, const int32_t* codes, const int32_t* bag_ptr, int32_t n_samples,
                              int32_t bps, int64_t n_lookups, const int32_t* sample_ids, int32_t n_sel_max,
                              int32_t stg_rows) {
  if (!h || n_samples < 0 || bps < 1 || n_lookups < 0 || n_sel_max < 0 || stg_rows < 0) return HL_ERR_INVALID_ARG;
  if (!bag_ptr || (n_lookups > 0 && !codes)) return HL_ERR_INVALID_ARG;
  if (!sample_ids && n_sel_max > n_samples) return HL_ERR_INVALID_ARG;
  if ((int64_t)n_samples * bps >= (1ll << 31) || n_lookups >= (1ll << 30)) return HL_ERR_UNSUPPORTED;
  if ((uint64_t)h->k_cap + (uint64_t)stg_rows >= (1ull << 31)) return HL_ERR_UNSUPPORTED;
  return HL_OK;
}

template <int VEC, bool BF>
static void launch_fwd(const hl_handle* h, dim3 grid, hipStream_t s, const void* w_hot, const void* stg,
                       int32_t stg_rows, const int32_t* codes, const int32_t* bag_ptr, int32_t bps,
                       const int32_t* ids, const int32_t* n_dev, int32_t n_max, float* out, eb_geom g,
                       int64_t n_lookups, int64_t n_bags, int part, int32_t nbg) {
  const hl_hook hk = hl_hook_take(h);
#define EBF(P)                                                                                                   \
  HL_KERNEL(h, s, P == 0 ? "eb_fwd" : (P == 1 ? "eb_fwd_hot" : "eb_fwd_cold"), (eb_fwd<VEC, BF, P>), grid,       \
            dim3(256), 0, s, w_hot, stg, stg_rows, h->n_hot, h->k_cap, codes, bag_ptr, bps, ids, n_dev, n_max, out, \
            g, n_lookups, n_bags, (int32_t)(n_bags / bps), nbg, h->d_err, hk);
  if (part == 0) { EBF(0) }
  else if (part == 1) { EBF(1) }
  else { EBF(2) }
#undef EBF
}

// grid of the one-hot forward: about 8 resident blocks per compute unit, each
// row group taking several chunks in turn
#define EB_OH_BLOCKS 1024
template <int VEC, bool BF>
static void launch_fwd_oh(const hl_handle* h, hipStream_t s, const void* w_hot, const void* stg, int32_t stg_rows,
                          const int32_t* codes, const int32_t* bag_ptr, float* out, eb_geom g, int64_t n_lookups,
                          int64_t n_bags, int part) {
  const hl_hook hk = hl_hook_take(h);
  const int64_t chunks = (n_bags + FC - 1) / FC;
  int64_t blocks = (chunks + 4 * g.NG - 1) / (4 * g.NG);
  if (blocks > EB_OH_BLOCKS) blocks = EB_OH_BLOCKS;
  const dim3 grid((uint32_t)blocks, g.cchunks);
  if (part == 0)
    HL_KERNEL(h, s, "eb_fwd", (eb_fwd_oh<VEC, BF, 0>), grid, dim3(256), 0, s, w_hot, stg, stg_rows, h->n_hot,
              h->k_cap, codes, bag_ptr, out, g, n_lookups, n_bags, h->d_err, hk);
  else
    HL_KERNEL(h, s, "eb_fwd_hot", (eb_fwd_oh<VEC, BF, 1>), grid, dim3(256), 0, s, w_hot, stg, stg_rows, h->n_hot,
              h->k_cap, codes, bag_ptr, out, g, n_lookups, n_bags, h->d_err, hk);
}

extern "C" hl_status hl_embbag_fwd_part(const hl_handle* h, const void* w_hot, const void* staging, int32_t stg_rows,
                                        const int32_t* codes, const int32_t* bag_ptr, int32_t n_samples, int32_t bps,
                                        int64_t n_lookups, const int32_t* sample_ids, const int32_t* n_sel_dev,
                                        int32_t n_sel_max, float* out, int32_t part, hl_stream stream) {
  hl_status st = check_common(h, codes, bag_ptr, n_samples, bps, n_lookups, sample_ids, n_sel_max, stg_rows);
  if (st != HL_OK) return st;
  if (part < 0 || part > 2) return HL_ERR_INVALID_ARG;
  if (n_sel_max == 0) return HL_OK;
  if (!out || (h->n_hot && !w_hot) || (stg_rows && !staging)) return HL_ERR_INVALID_ARG;
  const size_t es = h->dtype == HL_F32 ? 4 : 2;
  const int vec = eb_pick_vec(h->dim, es, {w_hot, staging, out});
  eb_geom g = eb_make_geom(h->dim, vec);
  const int64_t nb = (int64_t)n_samples * bps;
  // bags of several lookups each (multi-hot): one bag per row group, so that
  // more groups pool at once; bags of about one lookup: FC per group
  const int32_t nbg = n_lookups > 2 * nb ? 1 : FC;
  const int64_t chunks = ((int64_t)n_sel_max * bps + nbg - 1) / nbg;
  int64_t blocks = (chunks + 4 * g.NG - 1) / (4 * g.NG);
  if (blocks > (1 << 20)) blocks = 1 << 20;
  dim3 grid((uint32_t)blocks, g.cchunks);
  hipStream_t s = (hipStream_t)stream;
  const bool bf = h->dtype == HL_BF16;
  if (part != 2 && !sample_ids && n_sel_max == n_samples && n_lookups == nb) {
    // every sample of a one-hot mini-batch
#define FOH(V, B) launch_fwd_oh<V, B>(h, s, w_hot, staging, stg_rows, codes, bag_ptr, out, g, n_lookups, nb, part)
    if (vec == 8) FOH(8, true);  // (bf16 only)
    else if (vec == 4) { if (bf) FOH(4, true); else FOH(4, false); }
    else if (vec == 2) { if (bf) FOH(2, true); else FOH(2, false); }
    else { if (bf) FOH(1, true); else FOH(1, false); }
#undef FOH
    HL_LAUNCHED();
    return HL_OK;
  }
#define FWD(V, B) launch_fwd<V, B>(h, grid, s, w_hot, staging, stg_rows, codes, bag_ptr, bps, sample_ids, n_sel_dev, \
                                   n_sel_max, out, g, n_lookups, nb, part, nbg)
  if (vec == 8) FWD(8, true);  // (bf16 only)
  else if (vec == 4) { if (bf) FWD(4, true); else FWD(4, false); }
  else if (vec == 2) { if (bf) FWD(2, true); else FWD(2, false); }
  else { if (bf) FWD(1, true); else FWD(1, false); }
#undef FWD
  HL_LAUNCHED();
  return HL_OK;
}

extern "C" hl_status hl_embbag_fwd(const hl_handle* h, const void* w_hot, const void* staging, int32_t stg_rows,
                                   const int32_t* codes, const int32_t* bag_ptr, int32_t n_samples, int32_t bps,
                                   int64_t n_lookups, const int32_t* sample_ids, const int32_t* n_sel_dev,
                                   int32_t n_sel_max, float* out, hl_stream stream) {
  return hl_embbag_fwd_part(h, w_hot, staging, stg_rows, codes, bag_ptr, n_samples, bps, n_lookups, sample_ids,
                            n_sel_dev, n_sel_max, out, 0, stream);
}

// Keys are compressed codes: hot slot, or n_hot + staging row.
static int bw_key_bits(const hl_handle* h, int32_t stg_rows) {
  return hl_bit_width((uint64_t)h->n_hot + (uint64_t)stg_rows);
}

template <int VEC, bool BF>
static void launch_bwd(const hl_handle* h, uint32_t tiles, hipStream_t s, const uint32_t* sk, const uint32_t* sv,
                       uint32_t n, const float* dY, eb_geom g, void* w_hot, void* stg, uint32_t n_hot, float lr,
                       bw_ws& ws, int part) {
  const dim3 grid(tiles, g.cchunks);
  if (part == 0) {
    HL_KERNEL(h, s, "bw_reduce1", (bw_reduce1<VEC, BF, false>), grid, dim3(RB_BLOCK), 0, s, sk, sv, n, dY, g,
              w_hot, stg, n_hot, lr, ws.tfirst, ws.tlast, ws.tflag, ws.tkey, ws.gc, ws.gc_rows, ws.bnd, hl_hook{});
    HL_KERNEL(h, s, "bw_reduce2", (bw_reduce2<VEC, BF, false>), grid, dim3(RB_BLOCK), 0, s, tiles, g, w_hot, stg,
              n_hot, lr, ws.tfirst, ws.tlast, ws.tflag, ws.tkey, ws.gc, ws.gc_rows);
  } else if (part == 1 || part == 3) {
    HL_KERNEL(h, s, "bw_reduce1", (bw_reduce1<VEC, BF, true>), grid, dim3(RB_BLOCK), 0, s, sk, sv, n, dY, g,
              w_hot, stg, n_hot, lr, ws.tfirst, ws.tlast, ws.tflag, ws.tkey, ws.gc, ws.gc_rows, ws.bnd,
              part == 3 ? hl_hook_take(h) : hl_hook{});
    if (part == 1)
      HL_KERNEL(h, s, "bw_reduce2", (bw_reduce2<VEC, BF, true>), grid, dim3(RB_BLOCK), 0, s, tiles, g, w_hot, stg,
                n_hot, lr, ws.tfirst, ws.tlast, ws.tflag, ws.tkey, ws.gc, ws.gc_rows);
  } else {
    // the tail (cold lookups: about a tenth of a mini-batch here) is a part of
    // n the device knows; a grid of a few thousand waves strides over it
    uint32_t b = hl_div_up(n, 4 * CW_POS);
    if (b > 1024) b = 1024;
    HL_KERNEL(h, s, "bw_cold", (bw_cold<VEC, BF>), dim3(b, g.cchunks), dim3(256), 0, s, sk, n, g, stg, n_hot, lr,
              ws.gc, ws.gc_rows, ws.bnd, hl_hook{});
  }
}

extern "C" hl_status hl_embbag_bwd_plan(hl_handle* h, int32_t stg_rows, const int32_t* codes, const int32_t* bag_ptr,
                                        int32_t n_samples, int32_t bps, int64_t n_lookups, const int32_t* sample_ids,
                                        const int32_t* n_sel_dev, int32_t n_sel_max, void* workspace, size_t ws_bytes,
                                        hl_stream stream) {
  bool sent = false;
  return hl_embbag_bwd_plan_signal(h, stg_rows, const_cast<int32_t*>(codes), bag_ptr, n_samples, bps, n_lookups,
                                   sample_ids, n_sel_dev, n_sel_max, workspace, ws_bytes, stream, nullptr, 0, &sent,
                                   nullptr);
}

hl_status hl_embbag_bwd_plan_signal(hl_handle* h, int32_t stg_rows, int32_t* codes, const int32_t* bag_ptr,
                                    int32_t n_samples, int32_t bps, int64_t n_lookups, const int32_t* sample_ids,
                                    const int32_t* n_sel_dev, int32_t n_sel_max, void* workspace, size_t ws_bytes,
                                    hl_stream stream, uint32_t* sflag, uint32_t sval, bool* sent,
                                    const hl_cg_fused* cf, bool compact) {
  *sent = false;
  if (compact && cf && cf->table) return HL_ERR_INVALID_ARG;  // the fused plan's state follows the full layout
  if (cf && cf->table && sample_ids) return HL_ERR_INVALID_ARG;  // the fused plan selects every sample
  hl_status st = check_common(h, codes, bag_ptr, n_samples, bps, n_lookups, sample_ids, n_sel_max, stg_rows);
  if (st != HL_OK) return st;
  if (!workspace) return HL_ERR_INVALID_ARG;
  const int64_t n_bags = (int64_t)n_samples * bps;
  if (ws_bytes < bw_bytes(h, n_lookups, n_bags, compact)) return HL_ERR_CAPACITY;
  hl_ws_note(h, workspace, HL_WSK_OTHER);
  if (n_samples == 0 || n_lookups == 0 || n_sel_max == 0) {
    hl_ws_note(h, workspace, HL_WSK_BWD_PLAN, 0, n_bags, stg_rows);
    hl_ws_find(h, workspace)->compact = compact;
    return HL_OK;
  }
  hipStream_t s = (hipStream_t)stream;
  hl_carver c = hl_carver::after_header(workspace, ws_bytes);
  bw_ws ws;
  bw_carve(c, ws, (uint32_t)n_lookups, n_bags, h->dim, compact);
  const uint8_t* mask = nullptr;
  if (sample_ids) {
    uint32_t gb = hl_div_up(n_samples, 256);
    if (gb > 4096) gb = 4096;
    HL_KERNEL(h, s, "bw_mask", bw_mask, dim3(gb), dim3(256), 0, s, ws.mask, n_samples, sample_ids, n_sel_dev, n_sel_max, 0);
    HL_KERNEL(h, s, "bw_mask", bw_mask, dim3(gb), dim3(256), 0, s, ws.mask, n_samples, sample_ids, n_sel_dev, n_sel_max, 1);
    mask = ws.mask;
  }
  uint32_t *sk, *sv;
  const int bits = bw_key_bits(h, stg_rows);
  if (mask) {
    HL_KERNEL(h, s, "bw_prep", bw_prep, dim3(hl_div_up(n_bags, BP_BAGS)), dim3(256), 0, s, codes, bag_ptr, n_bags,
              bps, mask, h->n_hot, h->k_cap, stg_rows, ws.sort.k0, ws.sort.v0, n_lookups, sflag, sval, h->d_err);
    HL_LAUNCHED();
    *sent = sflag != nullptr;
    st = hl_sort_pairs(h, ws.sort, nullptr, (uint32_t)n_lookups, bits, s, &sk, &sv);
  } else if (hl_group_by_table_ok(h, n_lookups, n_bags)) {
    // one lookup per bag: grouped table by table (hl_group.hip), into the
    // buffers where the sort leaves its result; the others hold the
    // table-major pairs
    if ((uint64_t)n_lookups > ws.sort.n_max) return HL_ERR_CAPACITY;
    uint32_t *rk, *rv;
    hl_sort_result(ws.sort, bits, &rk, &rv);
    uint32_t* tk = rk == ws.sort.k0 ? ws.sort.k1 : ws.sort.k0;
    uint32_t* tv = rv == ws.sort.v0 ? ws.sort.v1 : ws.sort.v0;
    st = hl_group_by_table(h, codes, bag_ptr, n_bags, stg_rows, tk, tv, rk, rv, sflag, sval,
                           cf && cf->table ? cf : nullptr, s);
    *sent = sflag != nullptr;
  } else {
    if ((uint64_t)n_lookups > ws.sort.n_max) return HL_ERR_CAPACITY;
    const hl_sort_geom sg = hl_sort_geometry((uint32_t)n_lookups, bits, hl_stream_cus(s));
    // bags per writer block: up to about 8192 lookups each, 64 to BPH_BAGS bags
    int32_t bpb = BPH_BAGS;
    while (bpb > 64 && (int64_t)bpb * n_lookups > 8192 * n_bags) bpb >>= 1;
    const dim3 grid(sg.hist_blocks + (uint32_t)hl_div_up(n_bags, bpb));
#define BPH(NB)                                                                                                  \
  HL_KERNEL(h, s, "bw_prep_hist", bw_prep_hist<NB>, grid, dim3(BPH_THREADS), 0, s, codes, bag_ptr, n_bags, bps, h->n_hot, \
            h->k_cap, stg_rows, ws.sort.k0, ws.sort.v0, n_lookups, sg.hist_blocks, sg.passes, sg.b, ws.sort.part,   \
            ws.sort.st[0], sg.n_zero, bpb, sflag, sval, h->d_err, cf ? *cf : hl_cg_fused{})
    if (sg.nb == 256) BPH(256);
    else if (sg.nb == 1024) BPH(1024);
    else BPH(2048);
#undef BPH
    HL_LAUNCHED();
    *sent = sflag != nullptr;
    st = hl_sort_passes(h, ws.sort, nullptr, (uint32_t)n_lookups, bits, s, &sk, &sv);
  }
  if (st != HL_OK) return st;
  hl_ws_note(h, workspace, HL_WSK_BWD_PLAN, n_lookups, n_bags, stg_rows);
  hl_ws_find(h, workspace)->compact = compact;
  return HL_OK;
}

// Compute units of the handle's device.
static int eb_device_cus(const hl_handle* h) {
  static int cus[64];
  const int d = h->device >= 0 && h->device < 64 ? h->device : 0;
  if (cus[d] <= 0) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, h->device) != hipSuccess || v <= 0) v = 1;
    cus[d] = v;
  }
  return cus[d];
}

template <int VEC, bool BF>
static void launch_fwd_gt(hl_handle* h, hipStream_t s, const void* w_hot, const void* stg, int32_t stg_rows,
                          const int32_t* codes, const int32_t* bag_ptr, float* out, eb_geom g, int64_t n_lookups,
                          int64_t n_bags, const uint32_t* k_tm, const uint32_t* cum, uint32_t nblk, uint32_t* kout,
                          uint32_t* vout) {
  const int32_t T = h->n_tables;
  const uint32_t E = (uint32_t)(n_bags / T);
  // one block per compute unit (each holds the sort's LDS): the tables' sorts
  // and, on the other units, the forward
  const int cus = eb_device_cus(h);
  const uint32_t nf = (uint32_t)(cus > 2 * T ? cus - T : cus);
  const hl_hook hk = hl_hook_take(h);
#define FGT(I)                                                                                                    \
  HL_KERNEL(h, s, "eb_fwd_gt", (eb_fwd_gt<VEC, BF, I>), dim3(T + nf), dim3(GT_THREADS), 0, s, w_hot, stg, stg_rows, \
            h->n_hot, h->k_cap, codes, bag_ptr, out, g, n_lookups, n_bags, k_tm, cum, nblk, E, T, h->d_tb, kout,     \
            vout, h->d_err, h->ballot_ranks, hk)
  if (E <= 4 * GT_THREADS) FGT(4);
  else FGT(8);
#undef FGT
}

extern "C" hl_status hl_embbag_fwd_plan(hl_handle* h, const void* w_hot, const void* staging, int32_t stg_rows,
                                        const int32_t* codes, const int32_t* bag_ptr, int32_t n_samples, int32_t bps,
                                        int64_t n_lookups, float* out, void* workspace, size_t ws_bytes,
                                        hl_stream stream) {
  hl_status st = check_common(h, codes, bag_ptr, n_samples, bps, n_lookups, nullptr, n_samples, stg_rows);
  if (st != HL_OK) return st;
  if (!workspace) return HL_ERR_INVALID_ARG;
  const int64_t n_bags = (int64_t)n_samples * bps;
  const size_t es = h->dtype == HL_F32 ? 4 : 2;
  const int vec = eb_pick_vec(h->dim, es, {w_hot, staging, out});
  const eb_geom g = eb_make_geom(h->dim, vec);
  const bool bf = h->dtype == HL_BF16;
  // (rows of 4 elements per lane: wider rows would spill in blocks of GT_THREADS)
  const bool fused = n_samples > 0 && n_lookups > 0 && n_lookups == n_bags && g.cchunks == 1 && vec == 4 &&
                     hl_group_by_table_ok(h, n_lookups, n_bags);
  if (!fused) {
    // the two calls one after the other
    st = hl_embbag_fwd(h, w_hot, staging, stg_rows, codes, bag_ptr, n_samples, bps, n_lookups, nullptr, nullptr,
                       n_samples, out, stream);
    if (st != HL_OK) return st;
    return hl_embbag_bwd_plan(h, stg_rows, codes, bag_ptr, n_samples, bps, n_lookups, nullptr, nullptr, n_samples,
                              workspace, ws_bytes, stream);
  }
  if (!out || (h->n_hot && !w_hot) || (stg_rows && !staging)) return HL_ERR_INVALID_ARG;
  if (ws_bytes < bw_bytes(h, n_lookups, n_bags, false)) return HL_ERR_CAPACITY;
  hl_ws_note(h, workspace, HL_WSK_OTHER);
  hipStream_t s = (hipStream_t)stream;
  hl_carver c = hl_carver::after_header(workspace, ws_bytes);
  bw_ws ws;
  bw_carve(c, ws, (uint32_t)n_lookups, n_bags, h->dim, false);
  if ((uint64_t)n_lookups > ws.sort.n_max) return HL_ERR_CAPACITY;
  uint32_t *rk, *rv;
  hl_sort_result(ws.sort, bw_key_bits(h, stg_rows), &rk, &rv);
  uint32_t* tk = rk == ws.sort.k0 ? ws.sort.k1 : ws.sort.k0;
  uint32_t* tv = rv == ws.sort.v0 ? ws.sort.v1 : ws.sort.v0;
  const uint32_t nblk = hl_group_prep(h, const_cast<int32_t*>(codes), bag_ptr, n_bags, stg_rows, tk, tv, nullptr, 0,
                                      nullptr, s);
#define FG(V, B) launch_fwd_gt<V, B>(h, s, w_hot, staging, stg_rows, codes, bag_ptr, out, g, n_lookups, n_bags, tk, tv, \
                                     nblk, rk, rv)
  if (bf) FG(4, true);
  else FG(4, false);
#undef FG
  HL_LAUNCHED();
  hl_ws_note(h, workspace, HL_WSK_BWD_PLAN, n_lookups, n_bags, stg_rows);
  hl_ws_find(h, workspace)->compact = false;
  return HL_OK;
}

extern "C" hl_status hl_embbag_bwd_apply_part(hl_handle* h, void* w_hot, void* staging, int32_t stg_rows,
                                              int32_t n_samples, int32_t bps, int64_t n_lookups, const float* dY,
                                              float lr, int32_t part, void* workspace, size_t ws_bytes,
                                              hl_stream stream) {
  if (part < 0 || part > 2) return HL_ERR_INVALID_ARG;
  return hl_embbag_bwd_apply_any(h, w_hot, staging, stg_rows, n_samples, bps, n_lookups, dY, lr, part, workspace,
                                 ws_bytes, stream);
}

// parts 0-2 of hl_embbag_bwd_apply_part, and 3: the first half without its
// spanning segments (hl_embbag_finish_cold completes them)
hl_status hl_embbag_bwd_apply_any(hl_handle* h, void* w_hot, void* staging, int32_t stg_rows, int32_t n_samples,
                                  int32_t bps, int64_t n_lookups, const float* dY, float lr, int32_t part,
                                  void* workspace, size_t ws_bytes, hl_stream stream) {
  if (!h || n_samples < 0 || bps < 1 || n_lookups < 0 || stg_rows < 0 || !workspace) return HL_ERR_INVALID_ARG;
  if (part < 0 || part > 3) return HL_ERR_INVALID_ARG;
  const int64_t n_bags = (int64_t)n_samples * bps;
  hl_ws_rec* rec = hl_ws_find(h, workspace);
  if (!rec || rec->n != n_lookups || rec->bags != n_bags || rec->stg != stg_rows)
    return HL_ERR_INVALID_ARG;  // no matching plan is held by this workspace
  if (part == 2 && rec->part1 != 1) return HL_ERR_INVALID_ARG;  // the first half has not run on this plan
  if (part != 0 && rec->compact) return HL_ERR_INVALID_ARG;      // no room for the staging-row sums
  if (n_lookups == 0 || n_samples == 0) {
    if (part == 1 || part == 3) rec->part1 = part == 1 ? 1 : 3;
    return HL_OK;
  }
  if ((part != 2 && (!dY || (h->n_hot && !w_hot))) || (stg_rows && !staging)) return HL_ERR_INVALID_ARG;
  if (ws_bytes < bw_bytes(h, n_lookups, n_bags, rec->compact)) return HL_ERR_CAPACITY;
  hipStream_t s = (hipStream_t)stream;
  hl_carver c = hl_carver::after_header(workspace, ws_bytes);
  bw_ws ws;
  bw_carve(c, ws, (uint32_t)n_lookups, n_bags, h->dim, rec->compact);
  uint32_t *sk, *sv;
  hl_sort_result(ws.sort, bw_key_bits(h, stg_rows), &sk, &sv);
  const uint32_t n = (uint32_t)n_lookups;
  const size_t es = h->dtype == HL_F32 ? 4 : 2;
  const int vec = eb_pick_vec(h->dim, es, {w_hot, staging, part == 2 ? nullptr : dY});
  eb_geom g = eb_make_geom(h->dim, vec);
  const uint32_t te = (uint32_t)(RB_WAVES * g.NG * RB_EN(vec));
  const uint32_t tiles = hl_div_up(n, te);
  if (tiles > ws.tiles) return HL_ERR_CAPACITY;
  const bool bf = h->dtype == HL_BF16;
#define BWD(V, B) launch_bwd<V, B>(h, tiles, s, sk, sv, n, dY, g, w_hot, staging, h->n_hot, lr, ws, part)
  if (vec == 8) BWD(8, true);  // (bf16 only)
  else if (vec == 4) { if (bf) BWD(4, true); else BWD(4, false); }
  else if (vec == 2) { if (bf) BWD(2, true); else BWD(2, false); }
  else { if (bf) BWD(1, true); else BWD(1, false); }
#undef BWD
  HL_LAUNCHED();
  if (part == 1 || part == 3) {
    rec->part1 = part == 1 ? 1 : 3;
    rec->vec = vec;
  }
  return HL_OK;
}

hl_status hl_embbag_fwd_cold_sorted(hl_handle* h, const void* staging, int32_t stg_rows, const int32_t* codes,
                                    const int32_t* bag_ptr, int32_t n_samples, int32_t bps, int64_t n_lookups,
                                    float* out, void* workspace, size_t ws_bytes, hl_stream stream) {
  hl_status st = check_common(h, codes, bag_ptr, n_samples, bps, n_lookups, nullptr, n_samples, stg_rows);
  if (st != HL_OK) return st;
  if (!workspace || !out || (stg_rows && !staging)) return HL_ERR_INVALID_ARG;
  const int64_t n_bags = (int64_t)n_samples * bps;
  hl_ws_rec* rec = hl_ws_find(h, workspace);
  if (!rec || rec->n != n_lookups || rec->bags != n_bags || rec->stg != stg_rows || !rec->part1)
    return HL_ERR_INVALID_ARG;  // the grouping and the first apply half must be in this workspace
  if (n_lookups == 0 || n_samples == 0) return HL_OK;
  if (ws_bytes < bw_bytes(h, n_lookups, n_bags, rec->compact)) return HL_ERR_CAPACITY;
  hl_carver c = hl_carver::after_header(workspace, ws_bytes);
  bw_ws ws;
  bw_carve(c, ws, (uint32_t)n_lookups, n_bags, h->dim, rec->compact);
  uint32_t *sk, *sv;
  hl_sort_result(ws.sort, bw_key_bits(h, stg_rows), &sk, &sv);
  const size_t es = h->dtype == HL_F32 ? 4 : 2;
  const int vec = eb_pick_vec(h->dim, es, {staging, out});
  eb_geom g = eb_make_geom(h->dim, vec);
  const uint32_t n = (uint32_t)n_lookups;
  uint32_t b = hl_div_up(n, 4 * g.NG * FT);
  if (b > 512) b = 512;
  hipStream_t s = (hipStream_t)stream;
  const bool bf = h->dtype == HL_BF16;
#define TAIL(V, B)                                                                                                  \
  HL_KERNEL(h, s, "eb_fwd_tail", (eb_fwd_tail<V, B>), dim3(b, g.cchunks), dim3(256), 0, s, sk, sv, n, ws.bnd, g, \
            staging, stg_rows, h->n_hot, h->k_cap, codes, bag_ptr, out, h->d_err)
  if (vec == 8) TAIL(8, true);  // (bf16 only)
  else if (vec == 4) { if (bf) TAIL(4, true); else TAIL(4, false); }
  else if (vec == 2) { if (bf) TAIL(2, true); else TAIL(2, false); }
  else { if (bf) TAIL(1, true); else TAIL(1, false); }
#undef TAIL
  HL_LAUNCHED();
  return HL_OK;
}

// After apply part 3 and the fetch: the cold half of the forward from the
// sorted tail together with the first half's spanning segments, then the
// staging-row updates (part 2's kernel).
hl_status hl_embbag_finish_cold(hl_handle* h, void* w_hot, void* staging, int32_t stg_rows, const int32_t* codes,
                                const int32_t* bag_ptr, int32_t n_samples, int32_t bps, int64_t n_lookups, float lr,
                                float* out, void* workspace, size_t ws_bytes, hl_stream stream) {
  hl_status st = check_common(h, codes, bag_ptr, n_samples, bps, n_lookups, nullptr, n_samples, stg_rows);
  if (st != HL_OK) return st;
  if (!workspace || !out || (stg_rows && !staging) || (h->n_hot && !w_hot)) return HL_ERR_INVALID_ARG;
  const int64_t n_bags = (int64_t)n_samples * bps;
  hl_ws_rec* rec = hl_ws_find(h, workspace);
  if (!rec || rec->n != n_lookups || rec->bags != n_bags || rec->stg != stg_rows || rec->part1 != 3)
    return HL_ERR_INVALID_ARG;  // the grouping and apply part 3 must be in this workspace
  rec->part1 = 0;  // the plan is used up: no part 2 or second finish on it
  if (n_lookups == 0 || n_samples == 0) return HL_OK;
  if (ws_bytes < bw_bytes(h, n_lookups, n_bags, rec->compact)) return HL_ERR_CAPACITY;
  hl_carver c = hl_carver::after_header(workspace, ws_bytes);
  bw_ws ws;
  bw_carve(c, ws, (uint32_t)n_lookups, n_bags, h->dim, rec->compact);
  uint32_t *sk, *sv;
  hl_sort_result(ws.sort, bw_key_bits(h, stg_rows), &sk, &sv);
  // the first half's vector width (its tile sums' layout); out and the rows must allow it
  const size_t es = h->dtype == HL_F32 ? 4 : 2;
  const int vec = rec->vec;
  if (eb_pick_vec(h->dim, es, {w_hot, staging, out}) < vec) return HL_ERR_INVALID_ARG;
  eb_geom g = eb_make_geom(h->dim, vec);
  const uint32_t n = (uint32_t)n_lookups;
  const uint32_t te = (uint32_t)(RB_WAVES * g.NG * RB_EN(vec));
  const uint32_t tiles = hl_div_up(n, te);
  if (tiles > ws.tiles) return HL_ERR_CAPACITY;
  uint32_t tb = hl_div_up(n, RB_WAVES * g.NG * FT);
  if (tb > 1024) tb = 1024;  // (the tail, cold lookups only, is a part of n the device knows)
  // (as part 2: the tail, cold lookups only, is a part of n the device knows; a
  // grid of a few thousand waves strides over it)
  uint32_t cb = hl_div_up(n, 4 * CW_POS);
  if (cb > 1024) cb = 1024;
  hipStream_t s = (hipStream_t)stream;
  const bool bf = h->dtype == HL_BF16;
  // bags of several lookups: the cold half bag by bag, one bag per row group
  const bool multi = n_lookups > 2 * n_bags;
  const uint32_t fb = (uint32_t)std::min<int64_t>((n_bags + RB_WAVES * g.NG - 1) / (RB_WAVES * g.NG), 1 << 16);
#define FIN(V, B)                                                                                                   \
  do {                                                                                                             \
    if (multi)                                                                                                     \
      HL_KERNEL(h, s, "eb_bags_r2", (eb_bags_r2<V, B>), dim3(tiles + fb, g.cchunks), dim3(RB_BLOCK), 0, s, tiles,  \
                w_hot, h->n_hot, lr, ws.tfirst, ws.tlast, ws.tflag, ws.tkey, ws.gc, ws.gc_rows, g, staging,        \
                stg_rows, h->k_cap, codes, bag_ptr, bps, n_samples, out, h->d_err);                                \
    else                                                                                                           \
      HL_KERNEL(h, s, "eb_tail_r2", (eb_tail_r2<V, B>), dim3(tiles + tb, g.cchunks), dim3(RB_BLOCK), 0, s, tiles,  \
                w_hot, h->n_hot, lr, ws.tfirst, ws.tlast, ws.tflag, ws.tkey, ws.gc, ws.gc_rows, sk, sv, n, ws.bnd, \
                g, staging, stg_rows, h->k_cap, codes, bag_ptr, out, h->d_err);                                    \
    HL_KERNEL(h, s, "bw_cold", (bw_cold<V, B>), dim3(cb, g.cchunks), dim3(256), 0, s, sk, n, g, staging, h->n_hot, \
              lr, ws.gc, ws.gc_rows, ws.bnd, hl_hook_take(h));                                                     \
  } while (0)
  if (vec == 8) FIN(8, true);  // (bf16 only)
  else if (vec == 4) { if (bf) FIN(4, true); else FIN(4, false); }
  else if (vec == 2) { if (bf) FIN(2, true); else FIN(2, false); }
  else { if (bf) FIN(1, true); else FIN(1, false); }
#undef FIN
  HL_LAUNCHED();
  return HL_OK;
}

extern "C" hl_status hl_embbag_bwd_apply(hl_handle* h, void* w_hot, void* staging, int32_t stg_rows, int32_t n_samples,
                                         int32_t bps, int64_t n_lookups, const float* dY, float lr, void* workspace,
                                         size_t ws_bytes, hl_stream stream) {
  return hl_embbag_bwd_apply_part(h, w_hot, staging, stg_rows, n_samples, bps, n_lookups, dY, lr, 0, workspace,
                                  ws_bytes, stream);
}

extern "C" hl_status hl_embbag_bwd_sgd(hl_handle* h, void* w_hot, void* staging, int32_t stg_rows,
                                       const int32_t* codes, const int32_t* bag_ptr, int32_t n_samples, int32_t bps,
                                       int64_t n_lookups, const int32_t* sample_ids, const int32_t* n_sel_dev,
                                       int32_t n_sel_max, const float* dY, float lr, void* workspace, size_t ws_bytes,
                                       hl_stream stream) {
  hl_status st = check_common(h, codes, bag_ptr, n_samples, bps, n_lookups, sample_ids, n_sel_max, stg_rows);
  if (st != HL_OK) return st;
  if (n_samples == 0 || n_lookups == 0 || n_sel_max == 0) return HL_OK;
  if (!dY || !workspace || (h->n_hot && !w_hot) || (stg_rows && !staging)) return HL_ERR_INVALID_ARG;
  st = hl_embbag_bwd_plan(h, stg_rows, codes, bag_ptr, n_samples, bps, n_lookups, sample_ids, n_sel_dev, n_sel_max,
                          workspace, ws_bytes, stream);
  if (st != HL_OK) return st;
  return hl_embbag_bwd_apply(h, w_hot, staging, stg_rows, n_samples, bps, n_lookups, dY, lr, workspace, ws_bytes,
                             stream);
}

// The grouping that the last hl_embbag_bwd_plan on this workspace left (for
// inspection): the (key, bag) pairs in the order the reduction takes them.
extern "C" hl_status hl_embbag_bwd_grouping(hl_handle* h, int32_t stg_rows, int32_t n_samples, int32_t bps,
                                            int64_t n_lookups, const void* workspace, size_t ws_bytes,
                                            uint32_t* keys_out, uint32_t* bags_out, hl_stream stream) {
  if (!h || !workspace || n_samples < 0 || bps < 1 || n_lookups < 0 || stg_rows < 0) return HL_ERR_INVALID_ARG;
  if (n_lookups > 0 && (!keys_out || !bags_out)) return HL_ERR_INVALID_ARG;
  const int64_t n_bags = (int64_t)n_samples * bps;
  hl_ws_rec* rec = hl_ws_find(h, workspace);
  if (!rec || rec->n != n_lookups || rec->bags != n_bags || rec->stg != stg_rows) return HL_ERR_INVALID_ARG;
  if (n_lookups == 0) return HL_OK;
  if (ws_bytes < bw_bytes(h, n_lookups, n_bags, rec->compact)) return HL_ERR_CAPACITY;
  hl_carver c = hl_carver::after_header(const_cast<void*>(workspace), ws_bytes);
  bw_ws ws;
  bw_carve(c, ws, (uint32_t)n_lookups, n_bags, h->dim, rec->compact);
  uint32_t *sk, *sv;
  hl_sort_result(ws.sort, bw_key_bits(h, stg_rows), &sk, &sv);
  hipStream_t s = (hipStream_t)stream;
  if (hipMemcpyAsync(keys_out, sk, (size_t)n_lookups * 4, hipMemcpyDeviceToDevice, s) != hipSuccess ||
      hipMemcpyAsync(bags_out, sv, (size_t)n_lookups * 4, hipMemcpyDeviceToDevice, s) != hipSuccess)
    return HL_ERR_HIP;
  return HL_OK;
}
