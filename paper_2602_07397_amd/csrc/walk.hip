// Sketch-Determined Walk kernels (paper Sec. 2.3, Alg. 1 step 6).
//
//  walk_first_kernel  first walked layer: R = (A/c)^s, row-normalised.
//  walk_gemm_kernel   R = R_prev (A/c)^s. One wavefront per 16x16 output
//                     tile on fp64 MFMA 16x16x4; the element-wise power is
//                     taken while loading the B operand; tiles above the
//                     diagonal are written as zeros and the k-range of a tile
//                     is clipped to [j0, i_max] (both factors are lower
//                     triangular).
//  walk_norm_kernel   divides each row by its largest magnitude.
#include "sw_common.h"
#include "sw_internal.h"

namespace sw {

typedef double f64x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ double pow_int(double x, int s) {
  if (s == 8) {               // the paper's default exponent: three squarings
    const double x2 = x * x, x4 = x2 * x2;
    return x4 * x4;
  }
  double r = 1.0, b = x;
  while (s) {
    if (s & 1) r *= b;
    b *= b;
    s >>= 1;
  }
  return r;
}

__device__ __forceinline__ double scale_of(const double* A_scale, int s) {
  const double c = A_scale[s];
  return c > 0.0 ? c : 1.0;
}

__device__ __forceinline__ double block_max_256(double v, double* tmp) {
  for (int off = 32; off > 0; off >>= 1) v = fmax(v, __shfl_xor(v, off));
  if ((threadIdx.x & 63) == 0) tmp[threadIdx.x >> 6] = v;
  __syncthreads();
  v = fmax(fmax(tmp[0], tmp[1]), fmax(tmp[2], tmp[3]));
  __syncthreads();
  return v;
}

__global__ __launch_bounds__(256) void walk_first_kernel(const double* __restrict__ A,
                                                         const double* __restrict__ A_scale,
                                                         int s_exp, SeqMeta m,
                                                         double* __restrict__ R) {
  __shared__ double tmp[4];
  const int row = blockIdx.x;
  const int s = seq_of_block(m, row);
  const int i = row - m.blk_start[s];
  const int b = m.blk_start[s + 1] - m.blk_start[s];
  const double inv_c = 1.0 / scale_of(A_scale, s);
  const double* Ar = A + m.mat_start[s] + (long long)i * b;
  double* Rr = R + m.mat_start[s] + (long long)i * b;
  double mx = 0.0;
  for (int j = threadIdx.x; j < b; j += 256) {
    const double w = (j <= i) ? pow_int(Ar[j] * inv_c, s_exp) : 0.0;
    Rr[j] = w;
    mx = fmax(mx, fabs(w));
  }
  mx = block_max_256(mx, tmp);
  if (mx > 0.0) {
    const double inv = 1.0 / mx;
    for (int j = threadIdx.x; j <= i; j += 256) Rr[j] = Rr[j] * inv;
  }
}

__global__ __launch_bounds__(256) void walk_gemm_kernel(const double* __restrict__ A,
                                                        const double* __restrict__ A_scale,
                                                        int s_exp, SeqMeta m, int total_tiles,
                                                        const double* __restrict__ Rp,
                                                        double* __restrict__ R) {
  const int wave = threadIdx.x >> 6;
  const int l = threadIdx.x & 63;
  const int tile = blockIdx.x * 4 + wave;
  if (tile >= total_tiles) return;
  int s = 0;
  while (s + 1 < m.n_seqs && m.aux_start[s + 1] <= tile) ++s;
  const int b = m.blk_start[s + 1] - m.blk_start[s];
  const int tb = (b + 15) >> 4;
  const int lt = tile - m.aux_start[s];
  const int ti = lt / tb, tj = lt % tb;
  const double* As = A + m.mat_start[s];
  const double* Ps = Rp + m.mat_start[s];
  double* Rs = R + m.mat_start[s];
  if (tj > ti) {
    for (int v = 0; v < 4; ++v) {
      const int ri = ti * 16 + (l >> 4) + 4 * v, cj = tj * 16 + (l & 15);
      if (ri < b && cj < b) Rs[(long long)ri * b + cj] = 0.0;
    }
    return;
  }
  const double inv_c = 1.0 / scale_of(A_scale, s);
  const int ra = ti * 16 + (l & 15);   // A-operand row (output row)
  const int cb = tj * 16 + (l & 15);   // B-operand column (output column)
  const int kend = min(ti * 16 + 15, b - 1);
  f64x4 acc = {0.0, 0.0, 0.0, 0.0};
  for (int k0 = (tj * 16) & ~3; k0 <= kend; k0 += 4) {
    const int k = k0 + (l >> 4);
    const double av = (ra < b && k <= ra) ? Ps[(long long)ra * b + k] : 0.0;
    const double bv = (k < b && cb <= k) ? pow_int(As[(long long)k * b + cb] * inv_c, s_exp) : 0.0;
    acc = __builtin_amdgcn_mfma_f64_16x16x4f64(av, bv, acc, 0, 0, 0);
  }
  for (int v = 0; v < 4; ++v) {
    const int ri = ti * 16 + (l >> 4) + 4 * v, cj = tj * 16 + (l & 15);
    if (ri < b && cj < b) Rs[(long long)ri * b + cj] = (cj <= ri) ? acc[v] : 0.0;
  }
}

__global__ __launch_bounds__(256) void walk_norm_kernel(SeqMeta m, double* __restrict__ R) {
  __shared__ double tmp[4];
  const int row = blockIdx.x;
  const int s = seq_of_block(m, row);
  const int i = row - m.blk_start[s];
  const int b = m.blk_start[s + 1] - m.blk_start[s];
  double* Rr = R + m.mat_start[s] + (long long)i * b;
  double mx = 0.0;
  for (int j = threadIdx.x; j <= i; j += 256) mx = fmax(mx, fabs(Rr[j]));
  mx = block_max_256(mx, tmp);
  if (mx > 0.0) {
    const double inv = 1.0 / mx;
    for (int j = threadIdx.x; j <= i; j += 256) Rr[j] = Rr[j] * inv;
  }
}

hipError_t launch_walk(const double* A, const double* A_scale, int s_exp, const SeqMeta& meta,
                       int64_t nb, const double* R_prev, double* R_out, hipStream_t st) {
  if (R_prev == nullptr) {
    hipLaunchKernelGGL(walk_first_kernel, dim3((unsigned)nb), dim3(256), 0, st, A, A_scale, s_exp,
                       meta, R_out);
    return hipGetLastError();
  }
  SeqMeta m2 = meta;
  int total = 0;
  for (int s = 0; s < meta.n_seqs; ++s) {
    m2.aux_start[s] = total;
    const int b = meta.blk_start[s + 1] - meta.blk_start[s];
    const int tb = (b + 15) / 16;
    total += tb * tb;
  }
  m2.aux_start[meta.n_seqs] = total;
  hipLaunchKernelGGL(walk_gemm_kernel, dim3((unsigned)((total + 3) / 4)), dim3(256), 0, st, A,
                     A_scale, s_exp, m2, total, R_prev, R_out);
  hipLaunchKernelGGL(walk_norm_kernel, dim3((unsigned)nb), dim3(256), 0, st, meta, R_out);
  return hipGetLastError();
}

}  // namespace sw
