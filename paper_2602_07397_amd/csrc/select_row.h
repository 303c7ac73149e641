// Top-tau selection of one row by one 256-thread workgroup (paper Alg. 1
// step 7 / Alg. 2 step 6; forced first and last blocks per Sec. 4.1).
//
// Thread t owns the contiguous key-block range [t*E, t*E + E), E =
// ceil(avail / 256), so block-wide scans run in index order. The
// (tau - |F|)-th largest walk value among the non-forced blocks is found by
// an 8-pass, 8-bit MSB-first radix select on order-preserving 64-bit keys of
// the fp64 values (integer LDS histograms, so the result does not depend on
// scheduling); equal values are taken in ascending block order; selected
// blocks are compacted in ascending order.
#pragma once

#include "sw_common.h"

namespace sw {


__device__ __forceinline__ int row_budget_dev(int avail, int nf, int k, int pct) {
  int t = (k > 0) ? k : (avail * pct + 99) / 100;
  t = max(t, nf);
  return min(t, avail);
}

// Kernels over rows of at most 256 * MAXE blocks hold MAXE values per
// thread (MAXE in {2, 4, 8, 16}); launchers pick the smallest that fits.
inline int row_maxe(int max_avail) {
  const int e = (max_avail + 255) / 256;
  return e <= 2 ? 2 : e <= 4 ? 4 : e <= 8 ? 8 : 16;
}

// This thread's values of a row: v[e] = vals[t*E + e] for the blocks it owns
// (E = ceil(avail / 256) <= MAXE; entries e >= E are never used). The loads
// carry no condition (the index is clamped into the row), so all of them are
// in flight before the first value is used.
template <int MAXE>
__device__ __forceinline__ void load_row_vals(const double* __restrict__ vals, int avail,
                                              double (&v)[MAXE]) {
  const int t = threadIdx.x;
  const int E = (avail + 255) / 256;
#pragma unroll
  for (int e = 0; e < MAXE; ++e) v[e] = vals[min(t * E + e, avail - 1)];
}

// Selects from the row held as per-thread values v (as load_row_vals lays
// them out) with forced set {first, last} (-1 = none). The radix passes
// start at the first byte where the smallest and largest candidate keys
// differ (the bytes before it put every candidate in one bin).
template <int MAXE>
__device__ __forceinline__ void select_row_vals(const double (&v)[MAXE], int avail, int first,
                                                int last, int k, int pct,
                                                int32_t* __restrict__ out,
                                                int32_t* __restrict__ cnt, int kmax) {
  static_assert(MAXE <= 32, "one mask bit per value");
  // the passes alternate between two copies of the histogram, the scan's
  // wavefront totals and the boundary bin, so a pass needs three barriers
  __shared__ int hist[2][256];
  __shared__ int scan_tmp[256];
  __shared__ int ptot[2][4];
  __shared__ int sh_digit[2], sh_need[2], sh_cnt[2];
  __shared__ unsigned long long klo[4], khi[4];
  const int t = threadIdx.x;
  const int E = (avail + 255) / 256;
  const int nf = (first >= 0) + (last >= 0 && last != first);
  const int tau = row_budget_dev(avail, nf, k, pct);
  const int m = tau - nf;                 // ranked blocks to take
  const int nc = avail - nf;              // ranked candidates

  unsigned long long key[MAXE];
  uint32_t candmask = 0, forcedmask = 0;
#pragma unroll
  for (int e = 0; e < MAXE; ++e) {
    key[e] = 0ull;
    const int j = t * E + e;
    if (e < E && j < avail) {
      if (j == first || j == last) {
        forcedmask |= 1u << e;
      } else {
        candmask |= 1u << e;
        key[e] = order_key(v[e]);
      }
    }
  }

  // Radix select of the m-th largest candidate key, MSB first. After each
  // pass the candidates matching `prefix` under `pmask` contain the boundary;
  // the loop stops early once every candidate in the boundary bin is taken.
  unsigned long long prefix = 0ull, pmask = 0ull;
  int need = m;
  bool take_all_eq = false;
  const bool partial = (m > 0 && m < nc);
  if (partial) {
    unsigned long long lo = ~0ull, hi = 0ull;
#pragma unroll
    for (int e = 0; e < MAXE; ++e)
      if ((candmask >> e) & 1u) {
        lo = key[e] < lo ? key[e] : lo;
        hi = key[e] > hi ? key[e] : hi;
      }
    for (int off = 32; off > 0; off >>= 1) {
      const unsigned long long ol = __shfl_xor(lo, off), oh = __shfl_xor(hi, off);
      lo = ol < lo ? ol : lo;
      hi = oh > hi ? oh : hi;
    }
    if ((t & 63) == 0) {
      klo[t >> 6] = lo;
      khi[t >> 6] = hi;
    }
    hist[0][t] = 0;
    __syncthreads();
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      lo = klo[w] < lo ? klo[w] : lo;
      hi = khi[w] > hi ? khi[w] : hi;
    }
    const int same = (lo == hi) ? 8 : (__clzll((long long)(lo ^ hi)) >> 3);
    if (same > 0) {
      pmask = (same == 8) ? ~0ull : (~0ull << (64 - 8 * same));
      prefix = lo & pmask;
    }
    for (int pass = same; pass < 8; ++pass) {
      const int shift = 56 - 8 * pass;
      const int cur = (pass - same) & 1;
#pragma unroll
      for (int e = 0; e < MAXE; ++e)
        if ((candmask >> e) & 1u)
          if ((key[e] & pmask) == prefix)
            atomicAdd(&hist[cur][(int)((key[e] >> shift) & 255ull)], 1);
      hist[cur ^ 1][t] = 0;                // the next pass's copy
      __syncthreads();
      // bins in descending digit order, exclusive prefix counts
      const int v = hist[cur][255 - t];
      const int x = wave_inclusive_scan(v);
      if ((t & 63) == 63) ptot[cur][t >> 6] = x;
      __syncthreads();
      int excl = x - v;
#pragma unroll
      for (int q = 0; q < 4; ++q) excl += (q < (t >> 6)) ? ptot[cur][q] : 0;
      if (v > 0 && excl < need && need <= excl + v) {
        sh_digit[cur] = 255 - t;
        sh_need[cur] = need - excl;
        sh_cnt[cur] = v;
      }
      __syncthreads();
      prefix |= ((unsigned long long)sh_digit[cur]) << shift;
      pmask |= 255ull << shift;
      need = sh_need[cur];
      if (sh_need[cur] == sh_cnt[cur]) {
        take_all_eq = true;
        break;
      }
    }
  }

  // rank of each boundary-valued candidate among equals, in index order
  int my_eq = 0;
  if (partial && !take_all_eq) {
#pragma unroll
    for (int e = 0; e < MAXE; ++e)
      if (((candmask >> e) & 1u) && (key[e] & pmask) == prefix) ++my_eq;
  }
  int dummy;
  int eq_before = block_exclusive_scan_256(my_eq, scan_tmp, &dummy);

  uint32_t selmask = forcedmask;
#pragma unroll
  for (int e = 0; e < MAXE; ++e) {
    if ((candmask >> e) & 1u) {
      bool take;
      const unsigned long long kk = key[e] & pmask;
      if (m >= nc) take = true;
      else if (m <= 0) take = false;
      else if (kk > prefix) take = true;
      else if (kk == prefix) take = take_all_eq || (eq_before++ < need);
      else take = false;
      if (take) selmask |= 1u << e;
    }
  }
  const int mine = __popc(selmask);
  int total_sel;
  int pos = block_exclusive_scan_256(mine, scan_tmp, &total_sel);
#pragma unroll
  for (int e = 0; e < MAXE; ++e)
    if ((selmask >> e) & 1u) out[pos++] = t * E + e;
  for (int q = tau + t; q < kmax; q += 256) out[q] = -1;
  if (t == 0) *cnt = tau;
}

// Selects from vals[0..avail) with forced set {first, last} (-1 = none).
template <int MAXE>
__device__ __forceinline__ void select_row_dev(const double* __restrict__ vals, int avail, int first,
                                               int last, int k, int pct, int32_t* __restrict__ out,
                                               int32_t* __restrict__ cnt, int kmax) {
  double v[MAXE];
  load_row_vals<MAXE>(vals, avail, v);
  select_row_vals<MAXE>(v, avail, first, last, k, pct, out, cnt, kmax);
}

}  // namespace sw
