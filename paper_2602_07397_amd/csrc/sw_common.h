// Shared device/host helpers for the sketch-and-walk HIP library (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/sketchwalk.h"

namespace sw {

// Lane layouts of the matrix instructions used here (measured on gfx950):
//  v_mfma_f64_16x16x4f64: A[m][k] from lane m + 16k, B[k][n] from lane n + 16k,
//    D[m][n] in lane n + 16 (m % 4), element m / 4.
//  v_mfma_f32_32x32x16_bf16 / v_mfma_f32_32x32x2f32: A[m][k] from lane
//    m + 32 (k / K_lane), element k % K_lane (K_lane = 8 / 1), B[k][n] from lane
//    n + 32 (k / K_lane); D[m][n] in lane n + 32 ((m / 4) % 2), element
//    4 (m / 8) + m % 4.

// Per-call sequence layout, passed to kernels by value (fits the kernel
// argument space for up to SW_MAX_SEQS sequences).
struct SeqMeta {
  int n_seqs;
  int B;
  int max_b;                              // largest per-sequence block count
  int tok_start[SW_MAX_SEQS + 1];         // cu_seqlens
  int blk_start[SW_MAX_SEQS + 1];         // prefix sums of b_s = ceil(n_s / B)
  long long mat_start[SW_MAX_SEQS + 1];   // prefix sums of b_s * b_s
  int aux_start[SW_MAX_SEQS + 1];         // per-launch prefix (e.g. tile counts)
};

// Sequence that owns global block row `row` (blk_start is increasing).
__device__ __forceinline__ int seq_of_block(const SeqMeta& m, int row) {
  int lo = 0, hi = m.n_seqs - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (m.blk_start[mid] <= row) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(((uint32_t)h) << 16);
}

// fp32 -> bf16, round to nearest even (gfx950: v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  const __bf16 h = (__bf16)f;
  return *reinterpret_cast<const uint16_t*>(&h);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  bf16x2_t v;
  v[0] = (__bf16)lo;
  v[1] = (__bf16)hi;
  return *reinterpret_cast<const uint32_t*>(&v);
}

// Monotone map from a double to uint64 (larger double -> larger key);
// -0.0 is folded onto +0.0 so that equal values compare equal.
__device__ __forceinline__ unsigned long long order_key(double v) {
  v = v + 0.0;
  unsigned long long u = (unsigned long long)__double_as_longlong(v);
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

// Inclusive prefix sum over the 64 lanes of a wavefront with DPP moves:
// shifts by 1, 2, 4 and 8 lanes within each 16-lane row (lanes without a
// source add 0), then lane 15 of each row added to the next row and lane 31
// to the upper half.
__device__ __forceinline__ int wave_inclusive_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, true);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, true);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, true);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, true);   // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);  // row_bcast:15, rows 1 and 3
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);  // row_bcast:31, rows 2 and 3
  return x;
}

// Exclusive prefix sum over a 256-thread block (4 wavefronts): an inclusive
// scan inside each wavefront (DPP moves), then the wavefront totals
// through LDS. `tmp` holds at least 4 ints of LDS. Returns the exclusive
// prefix of `v`; `*total` receives the block sum. Contains two barriers.
__device__ __forceinline__ int block_exclusive_scan_256(int v, int* tmp, int* total) {
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  const int x = wave_inclusive_scan(v);
  if (lane == 63) tmp[w] = x;
  __syncthreads();
  int before = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) before += (q < w) ? tmp[q] : 0;
  *total = tmp[0] + tmp[1] + tmp[2] + tmp[3];
  __syncthreads();
  return before + x - v;
}

__device__ __forceinline__ void butterfly(double& a, double& b) {
  const double u = a, v = b;
  a = u + v;
  b = u - v;
}

// Unnormalised Walsh-Hadamard transform (natural order) of x[0..d) in LDS by
// one whole wavefront. Lane l holds elements l*E .. l*E + E - 1 with
// E = d / 64 (one element in lanes l < d when d < 64); stages of stride
// below E run inside the lane, the others exchange with lane l ^ (stride/E):
// the lane holding the lower index keeps u + v, the other u - v. The stages
// run in the order 1, 2, 4, ... as in the textbook iteration.
__device__ __forceinline__ void wave_fwht(double* x, int d) {
  const int lane = threadIdx.x & 63;
  const int E = d >= 64 ? d / 64 : 1;    // 1, 2 or 4 (d <= 256)
  double v[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) v[e] = (e < E && lane * E + e < d) ? x[lane * E + e] : 0.0;
  if (E >= 2) {                          // stride 1 inside the lane
    butterfly(v[0], v[1]);
    if (E == 4) butterfly(v[2], v[3]);
  }
  if (E == 4) {                          // stride 2 inside the lane
    butterfly(v[0], v[2]);
    butterfly(v[1], v[3]);
  }
  for (int len = E; len < d; len <<= 1) {
    const int lx = len / E;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (e < E) {
        const double o = __shfl_xor(v[e], lx);
        v[e] = (lane & lx) ? (o - v[e]) : (v[e] + o);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (e < E && lane * E + e < d) x[lane * E + e] = v[e];
}

}  // namespace sw
