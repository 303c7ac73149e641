// Top-tau block selection (paper Alg. 1 step 7 / Alg. 2 step 6; forced
// first and last blocks per Sec. 4.1).
//
// One 256-thread workgroup per row. Thread t owns the contiguous key-block
// range [t*E, t*E + E), so block-wide scans run in index order. The
// (tau - |F|)-th largest walk value among the non-forced blocks is found by
// an 8-pass, 8-bit MSB-first radix select on order-preserving 64-bit keys of
// the fp64 values (integer LDS histograms, so the result does not depend on
// scheduling); equal values are taken in ascending block order; selected
// blocks are compacted in ascending order.
#include "sw_common.h"
#include "sw_internal.h"

namespace sw {

constexpr int kMaxPerThread = SW_MAX_BLOCKS / 256;

__device__ __forceinline__ int row_budget_dev(int avail, int nf, int k, int pct) {
  int t = (k > 0) ? k : (avail * pct + 99) / 100;
  t = max(t, nf);
  return min(t, avail);
}

// Selects from vals[0..avail) with forced set {first, last} (-1 = none).
__device__ __forceinline__ void select_row_dev(const double* __restrict__ vals, int avail, int first, int last,
                               int k, int pct, int32_t* __restrict__ out, int32_t* __restrict__ cnt,
                               int kmax) {
  __shared__ int hist[256];
  __shared__ int scan_tmp[256];
  __shared__ int sh_digit, sh_need, sh_cnt;
  const int t = threadIdx.x;
  const int E = (avail + 255) / 256;
  const int nf = (first >= 0) + (last >= 0 && last != first);
  const int tau = row_budget_dev(avail, nf, k, pct);
  const int m = tau - nf;                 // ranked blocks to take
  const int nc = avail - nf;              // ranked candidates

  unsigned long long key[kMaxPerThread];
  uint32_t candmask = 0, forcedmask = 0;
#pragma unroll
  for (int e = 0; e < kMaxPerThread; ++e) {
    key[e] = 0ull;
    if (e < E) {
      const int j = t * E + e;
      if (j < avail) {
        if (j == first || j == last) {
          forcedmask |= 1u << e;
        } else {
          candmask |= 1u << e;
          key[e] = order_key(vals[j]);
        }
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
    for (int pass = 0; pass < 8; ++pass) {
      const int shift = 56 - 8 * pass;
      hist[t] = 0;
      __syncthreads();
#pragma unroll
      for (int e = 0; e < kMaxPerThread; ++e)
        if ((candmask >> e) & 1u)
          if ((key[e] & pmask) == prefix) atomicAdd(&hist[(int)((key[e] >> shift) & 255ull)], 1);
      __syncthreads();
      const int v = hist[255 - t];
      int total;
      const int excl = block_exclusive_scan_256(v, scan_tmp, &total);
      if (v > 0 && excl < need && need <= excl + v) {
        sh_digit = 255 - t;
        sh_need = need - excl;
        sh_cnt = v;
      }
      __syncthreads();
      prefix |= ((unsigned long long)sh_digit) << shift;
      pmask |= 255ull << shift;
      need = sh_need;
      const bool done = (sh_need == sh_cnt);
      __syncthreads();
      if (done) {
        take_all_eq = true;
        break;
      }
    }
  }

  // rank of each boundary-valued candidate among equals, in index order
  int my_eq = 0;
  if (partial && !take_all_eq) {
#pragma unroll
    for (int e = 0; e < kMaxPerThread; ++e)
      if (((candmask >> e) & 1u) && (key[e] & pmask) == prefix) ++my_eq;
  }
  int dummy;
  int eq_before = block_exclusive_scan_256(my_eq, scan_tmp, &dummy);

  uint32_t selmask = forcedmask;
#pragma unroll
  for (int e = 0; e < kMaxPerThread; ++e) {
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
  for (int e = 0; e < kMaxPerThread; ++e)
    if ((selmask >> e) & 1u) out[pos++] = t * E + e;
  for (int q = tau + t; q < kmax; q += 256) out[q] = -1;
  if (t == 0) *cnt = tau;
}

__global__ __launch_bounds__(256) void select_prefill_kernel(const double* __restrict__ R,
                                                             SeqMeta m, int k, int pct,
                                                             uint32_t flags,
                                                             int32_t* __restrict__ idx,
                                                             int32_t* __restrict__ cnt, int kmax) {
  const int row = blockIdx.x;
  const int s = seq_of_block(m, row);
  const int i = row - m.blk_start[s];
  const int b = m.blk_start[s + 1] - m.blk_start[s];
  const double* vals = R + m.mat_start[s] + (long long)i * b;
  const int first = (flags & SW_FORCE_FIRST) ? 0 : -1;
  const int last = (flags & SW_FORCE_LAST) ? i : -1;
  select_row_dev(vals, i + 1, first, last, k, pct, idx + (long long)row * kmax, cnt + row, kmax);
}

// One row per sequence (Alg. 2 step 6): the walk row over key blocks
// 0..b_cur of the token at pos[b]; forced set {0, b_cur}.
__global__ __launch_bounds__(256) void select_decode_kernel(const double* __restrict__ rows,
                                                            int b_max, int B,
                                                            const int32_t* __restrict__ pos, int k,
                                                            int pct, uint32_t flags,
                                                            int32_t* __restrict__ idx,
                                                            int32_t* __restrict__ cnt, int kmax) {
  const int bi = blockIdx.x;
  const int p = pos[bi];
  const int bc = p / B;
  if (p < 0 || bc >= b_max) return;
  const int first = (flags & SW_FORCE_FIRST) ? 0 : -1;
  const int last = (flags & SW_FORCE_LAST) ? bc : -1;
  select_row_dev(rows + (long long)bi * b_max, bc + 1, first, last, k, pct,
                 idx + (long long)bi * kmax, cnt + bi, kmax);
}

// The same with the walk row's normalisation first: the row is divided in
// place by its largest magnitude over blocks 0..b_cur (entries past b_cur are
// zeroed). Each thread rescales exactly the entries select_row_dev later
// reads in that thread (j = t*E + e), so no other thread's store is read.
__global__ __launch_bounds__(256) void select_decode_norm_kernel(double* __restrict__ rows,
                                                                 int b_max, int B,
                                                                 const int32_t* __restrict__ pos,
                                                                 int k, int pct, uint32_t flags,
                                                                 int32_t* __restrict__ idx,
                                                                 int32_t* __restrict__ cnt,
                                                                 int kmax) {
  __shared__ double tmp[4];
  const int bi = blockIdx.x;
  const int p = pos[bi];
  const int bc = p / B;
  if (p < 0 || bc >= b_max) return;
  double* row = rows + (long long)bi * b_max;
  const int avail = bc + 1;
  const int E = (avail + 255) / 256;
  const int t = threadIdx.x;
  double mx = 0.0;
  for (int e = 0; e < E; ++e) {
    const int j = t * E + e;
    if (j < avail) mx = fmax(mx, fabs(row[j]));
  }
  for (int off = 32; off > 0; off >>= 1) mx = fmax(mx, __shfl_xor(mx, off));
  if ((t & 63) == 0) tmp[t >> 6] = mx;
  __syncthreads();
  mx = fmax(fmax(tmp[0], tmp[1]), fmax(tmp[2], tmp[3]));
  const double inv = mx > 0.0 ? 1.0 / mx : 1.0;
  for (int e = 0; e < E; ++e) {
    const int j = t * E + e;
    if (j < avail) row[j] = row[j] * inv;
  }
  for (int j = avail + t; j < b_max; j += 256) row[j] = 0.0;
  const int first = (flags & SW_FORCE_FIRST) ? 0 : -1;
  const int last = (flags & SW_FORCE_LAST) ? bc : -1;
  select_row_dev(row, avail, first, last, k, pct, idx + (long long)bi * kmax, cnt + bi, kmax);
}

hipError_t launch_select_decode(const double* rows, int batch, int b_max, int B,
                                const int32_t* pos, int k, int pct, uint32_t flags, int32_t* idx,
                                int32_t* cnt, int kmax, hipStream_t st, double* normalize_rows) {
  if (normalize_rows != nullptr)
    hipLaunchKernelGGL(select_decode_norm_kernel, dim3((unsigned)batch), dim3(256), 0, st,
                       normalize_rows, b_max, B, pos, k, pct, flags, idx, cnt, kmax);
  else
    hipLaunchKernelGGL(select_decode_kernel, dim3((unsigned)batch), dim3(256), 0, st, rows, b_max,
                       B, pos, k, pct, flags, idx, cnt, kmax);
  return hipGetLastError();
}

hipError_t launch_select(const double* R, const SeqMeta& meta, int64_t nb, int k, int pct,
                         uint32_t flags, int32_t* idx, int32_t* cnt, int kmax, hipStream_t st) {
  hipLaunchKernelGGL(select_prefill_kernel, dim3((unsigned)nb), dim3(256), 0, st, R, meta, k, pct,
                     flags, idx, cnt, kmax);
  return hipGetLastError();
}

}  // namespace sw
