// The one-hot grouping's sort of one table in one block of GT_THREADS
// threads (gt_sort_body), shared by the grouping's own launch (hl_group.hip)
// and by the launch that runs it beside the forward (hl_embbag.hip).  The
// grouping is described in hl_group.hip.
#pragma once
#include "hl_internal.h"

#define GT_S 32           // bag rows per gt_prep block
#define GT_PI ((GT_S * GT_TMAX + 255) / 256)  // bags per gt_prep thread (at most)
#define GT_TMAX 64        // tables the path takes
#define GT_THREADS 1024
#define GT_WAVES (GT_THREADS / 64)
#define GT_IMAX 8         // items per thread: at most GT_IMAX * GT_THREADS bags per table (no spills)
#define GT_DBITS 9        // largest digit of the sort
#define GT_NB (1 << GT_DBITS)

// Exclusive scan of one value per thread over the block; *total receives the sum.
__device__ __forceinline__ uint32_t gt_scan(uint32_t v, uint32_t* ws, uint32_t* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) ws[w] = x;
  __syncthreads();
  uint32_t off = 0, tot = 0;
  for (int q = 0; q < GT_WAVES; ++q) {
    const uint32_t c = ws[q];
    off += q < w ? c : 0u;
    tot += c;
  }
  *total = tot;
  __syncthreads();  // ws may be reused
  return x - v + off;
}

// Sorts table t (a block of GT_THREADS threads).
template <int ITEMS>
__device__ __forceinline__ void gt_sort_body(uint32_t t, const uint32_t* __restrict__ keys_tm,
                                             const uint32_t* __restrict__ cum, uint32_t nblk, uint32_t E, int32_t T,
                                             uint32_t n, const uint32_t* __restrict__ tb, uint32_t n_hot,
                                             uint32_t* __restrict__ kout, uint32_t* __restrict__ vout, uint32_t* err,
                                             int ballot_only) {
  // a sorted item in LDS: compressed key in the high word, table-major
  // position in the low word (one 8-byte store and load per item and pass)
  __shared__ uint64_t sx[ITEMS * GT_THREADS];
  __shared__ uint32_t wcnt[GT_WAVES][GT_NB];
  __shared__ uint32_t dofs[GT_NB];
  __shared__ uint32_t scan_ws[GT_WAVES];
  __shared__ uint32_t s_max, s_sent, s_hb, s_ht;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const uint32_t lo = tb[t], R = tb[t + 1] - lo;  // the table's hot slots
  // the table's keys, position w * 64 ITEMS + 64 k + lane (lookup order), and
  // the hot keys of the earlier tables (hb) and up to this one (ht) summed
  // over the prep blocks: all loads issued before any is waited for
  uint32_t key[ITEMS], pos[ITEMS];
#pragma unroll
  for (int k = 0; k < ITEMS; ++k) {
    const uint32_t ps = (uint32_t)w * (ITEMS * 64) + k * 64 + lane;
    key[k] = keys_tm[(uint64_t)t * E + min(ps, E - 1)];
    pos[k] = ps;
  }
  uint32_t hb = 0, ht = 0;
  for (uint32_t b = tid; b < nblk; b += GT_THREADS) {
    hb += cum[(uint64_t)b * (T + 1) + t];
    ht += cum[(uint64_t)b * (T + 1) + t + 1];
  }
  if (tid == 0) {
    s_max = 0;
    s_sent = 0;
    s_hb = 0;
    s_ht = 0;
  }
  for (int j = tid; j < GT_WAVES * GT_NB; j += GT_THREADS) (&wcnt[0][0])[j] = 0;
  __syncthreads();
  const uint64_t lt = (1ull << lane) - 1ull;
  for (int stable = ballot_only ? 1 : 0, fresh = 1; stable < 2; ++stable, fresh = 0) {
    if (!fresh) {
      // (sorting again: the keys as loaded)
#pragma unroll
      for (int k = 0; k < ITEMS; ++k) {
        const uint32_t ps = (uint32_t)w * (ITEMS * 64) + k * 64 + lane;
        key[k] = keys_tm[(uint64_t)t * E + min(ps, E - 1)];
        pos[k] = ps;
      }
    }
    // compressed: hot slot - lo, or R + staging row, or (skipped: an invalid
    // code, or a hot slot of another table's row) one past the largest
    uint32_t kmax = 0;
    bool foreign = false, anysent = false;
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
      const uint32_t ps = (uint32_t)w * (ITEMS * 64) + k * 64 + lane;
      const bool valid = ps < E;
      const uint32_t kk = key[k];
      uint32_t c = EB_SENT;
      if (kk < n_hot) {
        if (kk - lo < R) c = kk - lo;
        else foreign = true;
      } else if (kk != EB_SENT) {
        c = R + (kk - n_hot);
      }
      key[k] = c;
      if (valid && c != EB_SENT) kmax = max(kmax, c);
      anysent = anysent || (valid && c == EB_SENT);
    }
    if (foreign && fresh) hl_flag(err, HL_DEVERR_BAD_CODE);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) kmax = max(kmax, (uint32_t)__shfl_xor(kmax, o));
    if (lane == 0) atomicMax(&s_max, kmax);
    if (anysent) s_sent = 1;
    if (fresh) {
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        hb += __shfl_xor(hb, o);
        ht += __shfl_xor(ht, o);
      }
      if (lane == 0) {
        atomicAdd(&s_hb, hb);
        atomicAdd(&s_ht, ht);
      }
    }
    __syncthreads();
    const uint32_t sent = max(s_max + 1, R);  // after every valid key, never below R (not hot)
#pragma unroll
    for (int k = 0; k < ITEMS; ++k)
      if (key[k] == EB_SENT) key[k] = sent;
    const uint32_t top = s_sent ? sent : s_max;
    const int bits = 32 - __clz(top);
    const int passes = (bits + GT_DBITS - 1) / GT_DBITS;  // 0: every key is 0, already in order
    const int b = passes ? (bits + passes - 1) / passes : 1;
    const uint32_t mask = (1u << b) - 1u;
    bool broken = false;  // the check, on the last pass of the fast ranks
    for (int p = 0; p < passes; ++p) {
      const int shift = p * b;
      uint32_t dg[ITEMS], rk[ITEMS];
      if (stable) {
#pragma unroll
        for (int k = 0; k < ITEMS; ++k) {
          const bool valid = (uint32_t)w * (ITEMS * 64) + k * 64 + lane < E;
          dg[k] = (key[k] >> shift) & mask;
          const uint64_t peers = hl_match_digit(dg[k], b, valid);
          const int leader = __ffsll((unsigned long long)peers) - 1;
          uint32_t bs = 0;
          if (valid && lane == leader) bs = atomicAdd(&wcnt[w][dg[k]], (uint32_t)__popcll(peers));
          bs = __shfl(bs, leader < 0 ? 0 : leader);
          rk[k] = bs + (uint32_t)__popcll(peers & lt);
        }
      } else {
        // the lanes of the first lane's digit together (their lowest lane
        // adds their count, the others add its old value to their rank among
        // them), every other lane adds 1 and takes the old value: one counter
        // update per item, all issued before any old value is used (a wave's
        // LDS operations execute in the order issued)
        uint32_t later = 0;  // items whose rank waits for the lowest lane's old value
        int l0[ITEMS];       // (uniform)
#pragma unroll
        for (int k = 0; k < ITEMS; ++k) {
          const bool valid = (uint32_t)w * (ITEMS * 64) + k * 64 + lane < E;
          dg[k] = (key[k] >> shift) & mask;
          const uint32_t d0 = __builtin_amdgcn_readfirstlane(dg[k]);
          const uint64_t m0 = __ballot(valid && dg[k] == d0);
          const bool in0 = (m0 >> lane) & 1ull;
          const uint32_t pr = (uint32_t)__popcll(m0 & lt);
          l0[k] = m0 ? __ffsll((unsigned long long)m0) - 1 : 0;
          rk[k] = pr;
          if ((valid && !in0) || (in0 && pr == 0))
            rk[k] = atomicAdd(&wcnt[w][dg[k]], in0 ? (uint32_t)__popcll(m0) : 1u);
          if (in0 && pr != 0) later |= 1u << k;
        }
#pragma unroll
        for (int k = 0; k < ITEMS; ++k) {
          const uint32_t base = __builtin_amdgcn_readlane(rk[k], l0[k]);
          if ((later >> k) & 1u) rk[k] += base;
        }
      }
      __syncthreads();
      // per digit: offsets of the waves, then of the digits
      uint32_t tot = 0;
      if (tid <= (int)mask) {
#pragma unroll
        for (int q0 = 0; q0 < GT_WAVES; q0 += 8) {
          uint32_t x[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) x[q] = wcnt[q0 + q][tid];
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            wcnt[q0 + q][tid] = tot;
            tot += x[q];
          }
        }
      }
      uint32_t all;
      const uint32_t ex = gt_scan(tid <= (int)mask ? tot : 0u, scan_ws, &all);
      if (tid <= (int)mask) dofs[tid] = ex;
      __syncthreads();
#pragma unroll
      for (int k = 0; k < ITEMS; ++k) {
        if ((uint32_t)w * (ITEMS * 64) + k * 64 + lane < E) {
          const uint32_t q = dofs[dg[k]] + wcnt[w][dg[k]] + rk[k];
          sx[q] = ((uint64_t)key[k] << 32) | pos[k];
        }
      }
      __syncthreads();
      const bool last = p + 1 == passes;
#pragma unroll
      for (int k = 0; k < ITEMS; ++k) {
        const uint32_t ps = (uint32_t)w * (ITEMS * 64) + k * 64 + lane;
        if (ps < E) {
          const uint64_t x = sx[ps];
          key[k] = (uint32_t)(x >> 32);
          pos[k] = (uint32_t)x;
          // (key, position) strictly ascending (positions are distinct)
          if (last && !stable && ps > 0) broken = broken || sx[ps - 1] >= x;
        }
      }
      for (int j = tid; j < GT_WAVES * GT_NB; j += GT_THREADS) (&wcnt[0][0])[j] = 0;
      if (last) broken = __syncthreads_or(broken);
      else __syncthreads();
    }
    if (stable || !broken) break;
    if (tid == 0) {
      s_max = 0;
      s_sent = 0;
    }
    __syncthreads();
  }
  // hot pairs of this table (keys below R, sorted first): h of them, after
  // the earlier tables' H; the others before the earlier tables' E t - H
  const uint32_t H = s_hb, h = s_ht - s_hb;
  const uint64_t nb0 = (uint64_t)n - ((uint64_t)E * t - H) - (E - h);
  const uint32_t sent_key = max(s_max + 1, R);
#pragma unroll
  for (int k = 0; k < ITEMS; ++k) {
    const uint32_t ps = (uint32_t)w * (ITEMS * 64) + k * 64 + lane;
    if (ps >= E) continue;
    if ((ps + 1 == h && key[k] >= R) || (ps == h && key[k] < R)) hl_flag(err, HL_DEVERR_INTERNAL);
    uint64_t o;
    uint32_t kk;
    if (ps < h) {
      o = (uint64_t)H + ps;
      kk = key[k] + lo;
    } else {
      o = nb0 + (ps - h);
      kk = key[k] >= sent_key ? EB_SENT : n_hot + (key[k] - R);
    }
    if (o < n) {
      kout[o] = kk;
      vout[o] = pos[k] * (uint32_t)T + t;  // the bag of table-major position pos
    } else {
      hl_flag(err, HL_DEVERR_INTERNAL);
    }
  }
}
