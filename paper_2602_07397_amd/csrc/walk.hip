// Sketch-Determined Walk kernels (paper Sec. 2.3, Alg. 1 step 6).
//
//  walk_first_kernel    first walked layer: R = W(A), row-normalised.
//  walk_gemm_kernel     C = X W(Y) for lower triangular X, Y. One workgroup per
//                       16x16 output tile on or below the diagonal, its four
//                       wavefronts splitting the tile's k-range (clipped to
//                       [j0, i_max]) on fp64 MFMA 16x16x4 and adding their
//                       partial tiles in a fixed order; the weight transform W
//                       is applied to the B operand. Entries above the
//                       diagonal of C are not written (the products never
//                       read them).
//  walk_softmax_kernel  causal row softmax of t*A (the transition matrix of
//                       the appendix lemma on the walk's stationary structure).
//  walk_norm_kernel     divides each row by its largest magnitude and writes
//                       the zeros above the diagonal.
//
// Weight transforms (template parameter): the element-wise power (A/c)^s of
// Alg. 1 step 6, the same power after clipping negative scores to zero, or
// the identity (the operand already holds weights). The matrix-power variant
// (the within-layer multi-hop walk of Sec. 1 and Fig. 2) is built from
// walk_gemm_kernel by binary exponentiation.
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

enum WeightFn { kWPow = 0, kWRelu = 1, kWIdent = 2 };

template <int F>
__device__ __forceinline__ double weight_of(double a, double inv_c, int s) {
  if constexpr (F == kWPow) return pow_int(a * inv_c, s);
  if constexpr (F == kWRelu) return pow_int(fmax(a, 0.0) * inv_c, s);
  return a;
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

__device__ __forceinline__ double block_sum_256(double v, double* tmp) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  if ((threadIdx.x & 63) == 0) tmp[threadIdx.x >> 6] = v;
  __syncthreads();
  v = (tmp[0] + tmp[1]) + (tmp[2] + tmp[3]);
  __syncthreads();
  return v;
}

// NORM = false writes W(A) itself (the factor of a matrix power).
template <int F, bool NORM = true>
__global__ __launch_bounds__(256) void walk_first_kernel(const double* __restrict__ A,
                                                         const double* __restrict__ A_scale,
                                                         int s_exp, SeqMeta m,
                                                         double* __restrict__ R) {
  __shared__ double tmp[4];
  const int row = blockIdx.x;
  const int s = seq_of_block(m, row);
  const int i = row - m.blk_start[s];
  const int b = m.blk_start[s + 1] - m.blk_start[s];
  const double inv_c = F == kWIdent ? 1.0 : 1.0 / scale_of(A_scale, s);
  const double* Ar = A + m.mat_start[s] + (long long)i * b;
  double* Rr = R + m.mat_start[s] + (long long)i * b;
  double mx = 0.0;
  for (int j = threadIdx.x; j < b; j += 256) {
    const double w = (j <= i) ? weight_of<F>(Ar[j], inv_c, s_exp) : 0.0;
    Rr[j] = w;
    mx = fmax(mx, fabs(w));
  }
  if (!NORM) return;
  mx = block_max_256(mx, tmp);
  if (mx > 0.0) {
    const double inv = 1.0 / mx;
    for (int j = threadIdx.x; j <= i; j += 256) Rr[j] = Rr[j] * inv;
  }
}

template <int F>
__global__ __launch_bounds__(256) void walk_gemm_kernel(const double* __restrict__ A,
                                                        const double* __restrict__ A_scale,
                                                        int s_exp, SeqMeta m, int total_tiles,
                                                        const double* __restrict__ Rp,
                                                        double* __restrict__ R) {
  __shared__ double red[4][64][4];
  const int wave = threadIdx.x >> 6;
  const int l = threadIdx.x & 63;
  const int tile = blockIdx.x;
  if (tile >= total_tiles) return;
  int s = 0;
  while (s + 1 < m.n_seqs && m.aux_start[s + 1] <= tile) ++s;
  const int b = m.blk_start[s + 1] - m.blk_start[s];
  const int tb = (b + 15) >> 4;
  // Lower tiles only, longest k-range first: group g = 0, 1, ... holds the
  // g + 1 tiles of diagonal ti - tj = tb - 1 - g.
  const int lt = tile - m.aux_start[s];
  int g = (int)((sqrt(8.0 * lt + 1.0) - 1.0) * 0.5);
  while ((g + 1) * (g + 2) / 2 <= lt) ++g;
  while (g * (g + 1) / 2 > lt) --g;
  const int tj = lt - g * (g + 1) / 2;
  const int ti = tj + tb - 1 - g;
  const double* As = A + m.mat_start[s];
  const double* Ps = Rp + m.mat_start[s];
  double* Rs = R + m.mat_start[s];
  const double inv_c = F == kWIdent ? 1.0 : 1.0 / scale_of(A_scale, s);
  const int ra = ti * 16 + (l & 15);   // A-operand row (output row)
  const int cb = tj * 16 + (l & 15);   // B-operand column (output column)
  const int kend = min(ti * 16 + 15, b - 1);
  // 32 k per chunk, 8 MFMA steps; in step u, lane group q = l / 16 carries
  // k = k0 + 8 q + u (the sum runs over every k once, in any order), so each
  // lane reads 8 consecutive entries of its A row. Wavefront w takes chunks
  // w, w + 4, w + 8, ...; its chunks are double-buffered in registers: the
  // loads of the next chunk are in flight during the MFMAs of the current one.
  const int kq = l >> 4;
  const long long rowA = (long long)min(ra, b - 1) * b;
  const int cbc = min(cb, b - 1);
  // the loads carry no condition (indices clamped into the matrix; the
  // entries outside the causal range are zeroed after loading), so all of a
  // chunk's loads are in flight together
  auto load = [&](int k0, double (&av)[8], double (&bv)[8]) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int k = k0 + 8 * kq + u;
      const int kc = min(k, b - 1);
      av[u] = Ps[rowA + kc];
      bv[u] = As[(long long)kc * b + cbc];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int k = k0 + 8 * kq + u;
      av[u] = (ra < b && k <= ra) ? av[u] : 0.0;
      bv[u] = (k < b && cb <= k) ? bv[u] : 0.0;
    }
  };
  f64x4 acc = {0.0, 0.0, 0.0, 0.0};
  auto compute = [&](const double (&av)[8], const double (&bv)[8]) {
#pragma unroll
    for (int u = 0; u < 8; ++u)
      acc = __builtin_amdgcn_mfma_f64_16x16x4f64(av[u], weight_of<F>(bv[u], inv_c, s_exp), acc, 0,
                                                 0, 0);
  };
  double a0[8], b0[8], a1[8], b1[8];
  int k0 = tj * 16 + 32 * wave;
  if (k0 <= kend) load(k0, a0, b0);
  for (; k0 <= kend; k0 += 256) {
    if (k0 + 128 <= kend) load(k0 + 128, a1, b1);
    compute(a0, b0);
    if (k0 + 128 > kend) break;
    if (k0 + 256 <= kend) load(k0 + 256, a0, b0);
    compute(a1, b1);
  }
#pragma unroll
  for (int v = 0; v < 4; ++v) red[wave][l][v] = acc[v];
  __syncthreads();
  if (wave != 0) return;
  for (int v = 0; v < 4; ++v) {
    const double sum = ((red[0][l][v] + red[1][l][v]) + red[2][l][v]) + red[3][l][v];
    const int ri = ti * 16 + (l >> 4) + 4 * v, cj = tj * 16 + (l & 15);
    if (ri < b && cj < b) Rs[(long long)ri * b + cj] = (cj <= ri) ? sum : 0.0;
  }
}

// Row i of W: exp(t A[i,j] - max) / sum over the causal blocks j <= i; zeros
// above the diagonal. The exponentials are stored, then scaled by 1/sum by
// the same thread that wrote them.
__global__ __launch_bounds__(256) void walk_softmax_kernel(const double* __restrict__ A,
                                                           double t, SeqMeta m,
                                                           double* __restrict__ W) {
  __shared__ double tmp[4];
  const int row = blockIdx.x;
  const int s = seq_of_block(m, row);
  const int i = row - m.blk_start[s];
  const int b = m.blk_start[s + 1] - m.blk_start[s];
  const double* Ar = A + m.mat_start[s] + (long long)i * b;
  double* Wr = W + m.mat_start[s] + (long long)i * b;
  double mx = -INFINITY;
  for (int j = threadIdx.x; j <= i; j += 256) mx = fmax(mx, t * Ar[j]);
  mx = block_max_256(mx, tmp);
  double sum = 0.0;
  for (int j = threadIdx.x; j < b; j += 256) {
    const double e = (j <= i) ? exp(t * Ar[j] - mx) : 0.0;
    Wr[j] = e;
    sum += e;
  }
  sum = block_sum_256(sum, tmp);
  const double inv = 1.0 / sum;
  for (int j = threadIdx.x; j <= i; j += 256) Wr[j] = Wr[j] * inv;
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
  const double inv = mx > 0.0 ? 1.0 / mx : 1.0;
  for (int j = threadIdx.x; j < b; j += 256) Rr[j] = (j <= i) ? Rr[j] * inv : 0.0;
}

namespace {

int gemm_tiles(const SeqMeta& meta, SeqMeta* m2) {
  *m2 = meta;
  int total = 0;
  for (int s = 0; s < meta.n_seqs; ++s) {
    m2->aux_start[s] = total;
    const int b = meta.blk_start[s + 1] - meta.blk_start[s];
    const int tb = (b + 15) / 16;
    total += tb * (tb + 1) / 2;
  }
  m2->aux_start[meta.n_seqs] = total;
  return total;
}

// C = X W(Y): X, Y, C lower triangular per sequence; only the lower
// triangle of C (and the diagonal tiles) is written.
template <int F>
void gemm(const double* X, const double* Y, const double* A_scale, int s_exp, const SeqMeta& m2,
          int total, double* C, hipStream_t st) {
  hipLaunchKernelGGL(walk_gemm_kernel<F>, dim3((unsigned)total), dim3(256), 0, st, Y,
                     A_scale, s_exp, m2, total, X, C);
}

}  // namespace

int64_t walk_workspace_bytes(int variant, int64_t nm) {
  if (variant == SW_WALK_SOFTMAX) return 8 * nm;
  if (variant == SW_WALK_MATPOW) return 16 * nm;
  return 0;
}

hipError_t launch_walk(int variant, const double* A, const double* A_scale, int s_exp,
                       double logit_scale, const SeqMeta& meta, int64_t nb, const double* R_prev,
                       double* R_out, double* ws, hipStream_t st) {
  const dim3 rows((unsigned)nb), blk(256);
  SeqMeta m2;
  const int total = gemm_tiles(meta, &m2);
  if (variant == SW_WALK_MATPOW && s_exp == 1) variant = SW_WALK_POWER;  // X^1 = X
  switch (variant) {
    case SW_WALK_POWER:
    case SW_WALK_RELU:
      if (R_prev == nullptr) {
        if (variant == SW_WALK_POWER)
          hipLaunchKernelGGL(walk_first_kernel<kWPow>, rows, blk, 0, st, A, A_scale, s_exp, meta,
                             R_out);
        else
          hipLaunchKernelGGL(walk_first_kernel<kWRelu>, rows, blk, 0, st, A, A_scale, s_exp, meta,
                             R_out);
        return hipGetLastError();
      }
      if (variant == SW_WALK_POWER)
        gemm<kWPow>(R_prev, A, A_scale, s_exp, m2, total, R_out, st);
      else
        gemm<kWRelu>(R_prev, A, A_scale, s_exp, m2, total, R_out, st);
      break;
    case SW_WALK_SOFTMAX: {
      double* W = R_prev == nullptr ? R_out : ws;
      hipLaunchKernelGGL(walk_softmax_kernel, rows, blk, 0, st, A, logit_scale, meta, W);
      if (R_prev != nullptr) gemm<kWIdent>(R_prev, W, nullptr, 1, m2, total, R_out, st);
      break;
    }
    case SW_WALK_MATPOW: {
      // Left-to-right binary exponentiation of X = A/c: square for every bit
      // below the leading one, multiply by X (read from A through the s = 1
      // power) where the bit is set. Two ping-pong buffers; without R_prev
      // the last product is written to R_out directly.
      const int64_t nm = meta.mat_start[meta.n_seqs];
      double* buf[2] = {ws, ws + nm};
      const int top = 31 - __builtin_clz((unsigned)s_exp);
      int nprod = 0;
      for (int bit = top - 1; bit >= 0; --bit) nprod += 1 + ((s_exp >> bit) & 1);
      hipLaunchKernelGGL((walk_first_kernel<kWPow, false>), rows, blk, 0, st, A, A_scale, 1, meta,
                         buf[0]);
      const double* cur = buf[0];
      int ci = 0, k = 0;
      for (int bit = top - 1; bit >= 0; --bit) {
        const int steps = 1 + ((s_exp >> bit) & 1);
        for (int step = 0; step < steps; ++step) {
          const bool last = ++k == nprod;
          double* dst = (last && R_prev == nullptr) ? R_out : buf[1 - ci];
          if (step == 0)
            gemm<kWIdent>(cur, cur, nullptr, 1, m2, total, dst, st);
          else
            gemm<kWPow>(cur, A, A_scale, 1, m2, total, dst, st);
          cur = dst;
          ci = 1 - ci;
        }
      }
      if (R_prev != nullptr) gemm<kWIdent>(R_prev, cur, nullptr, 1, m2, total, R_out, st);
      break;
    }
    default:
      return hipErrorInvalidValue;
  }
  hipLaunchKernelGGL(walk_norm_kernel, rows, blk, 0, st, meta, R_out);
  return hipGetLastError();
}

}  // namespace sw
