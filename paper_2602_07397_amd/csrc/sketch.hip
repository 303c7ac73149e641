// Small-World Sketching kernels (paper Sec. 2.2, Alg. 1 steps 1-5).
//
//  pool_kernel    head mean + block mean: streams Q and K once from HBM (one
//                 launch) with 16-byte loads; every workgroup sums one
//                 (block, head chunk) slice of Q or K in fp64 and writes a
//                 partial [d] vector.
//  fwht_kernel    per block row: fixed-order sum of the partials, divide by
//                 heads x tokens, random signs, in-LDS fast Walsh-Hadamard
//                 transform (natural order), column sampling, 1/sqrt(r).
//  scores_kernel  A = Qs Ks^T / sqrt(r) with fp64 MFMA 16x16x4 tiles, causal
//                 mask, per-sequence max |A| by integer atomicMax on the
//                 (non-negative) double bit pattern.
#include "sw_common.h"
#include "sw_internal.h"

namespace sw {

typedef double f64x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// One launch pools both Q and K: workgroups [0, nb * Pq) take Q, the rest K.
template <typename T>
__global__ __launch_bounds__(256) void pool_kernel(const T* __restrict__ Xq, int hcq, int Pq,
                                                   double* __restrict__ wsq,
                                                   const T* __restrict__ Xk, int hck, int Pk,
                                                   double* __restrict__ wsk, int nb, int d,
                                                   SeqMeta m, long long N) {
  constexpr int VEC = 16 / sizeof(T);
  __shared__ double red[256 * VEC];
  const bool is_q = (int)blockIdx.x < nb * Pq;
  const int bx = is_q ? (int)blockIdx.x : (int)blockIdx.x - nb * Pq;
  const T* X = is_q ? Xq : Xk;
  const int hc = is_q ? hcq : hck;
  const int P = is_q ? Pq : Pk;
  double* ws = is_q ? wsq : wsk;
  const int row = bx / P;
  const int p = bx % P;
  const int s = seq_of_block(m, row);
  const int i = row - m.blk_start[s];
  const int t0 = m.tok_start[s] + i * m.B;
  const int t1 = min(m.tok_start[s + 1], t0 + m.B);
  const int lpr = d / VEC;          // lanes per token row
  const int rpp = 256 / lpr;        // token rows per pass
  const int lane = threadIdx.x % lpr;
  const int r0 = threadIdx.x / lpr;

  double acc[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) acc[e] = 0.0;

  for (int hh = 0; hh < hc; ++hh) {
    const T* base = X + ((long long)(p * hc + hh) * N) * d + lane * VEC;
#pragma unroll 4
    for (int t = t0 + r0; t < t1; t += rpp) {
      // non-temporal: Q and K are streamed once here (the streaming hint
      // lifts the read rate)
      const u32x4 vv = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(base + (long long)t * d));
      const uint4 v = make_uint4(vv[0], vv[1], vv[2], vv[3]);
      if constexpr (sizeof(T) == 2) {
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[2 * e] += (double)__uint_as_float(w[e] << 16);
          acc[2 * e + 1] += (double)__uint_as_float(w[e] & 0xffff0000u);
        }
      } else {
        acc[0] += (double)__uint_as_float(v.x);
        acc[1] += (double)__uint_as_float(v.y);
        acc[2] += (double)__uint_as_float(v.z);
        acc[3] += (double)__uint_as_float(v.w);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < VEC; ++e) red[r0 * d + lane * VEC + e] = acc[e];
  __syncthreads();
  for (int c = threadIdx.x; c < d; c += 256) {
    double sum = 0.0;
    for (int k = 0; k < rpp; ++k) sum += red[k * d + c];
    ws[((long long)row * P + p) * d + c] = sum;
  }
}

__global__ __launch_bounds__(256) void fwht_kernel(const double* __restrict__ wsq,
                                                   const double* __restrict__ wsk, int Pq, int Pk,
                                                   int h_q, int h_kv, int d, SeqMeta m,
                                                   const int8_t* __restrict__ signs,
                                                   const int32_t* __restrict__ cols, int r,
                                                   double* __restrict__ Qs, double* __restrict__ Ks,
                                                   double* __restrict__ Qbar,
                                                   double* __restrict__ Kbar,
                                                   double* __restrict__ A_scale) {
  __shared__ double x[256];
  const int row = blockIdx.x;
  const bool isk = blockIdx.y == 1;
  const int s = seq_of_block(m, row);
  const int i = row - m.blk_start[s];
  const int t0 = m.tok_start[s] + i * m.B;
  const int cnt = min(m.tok_start[s + 1], t0 + m.B) - t0;
  const int P = isk ? Pk : Pq;
  const double* ws = isk ? wsk : wsq;
  const double inv = 1.0 / ((double)(isk ? h_kv : h_q) * (double)cnt);
  const int t = threadIdx.x;
  if (!isk && i == 0 && t == 0) A_scale[s] = 0.0;
  if (t < d) {
    double sum = 0.0;
    for (int pp = 0; pp < P; ++pp) sum += ws[((long long)row * P + pp) * d + t];
    const double mean = sum * inv;
    double* bar = isk ? Kbar : Qbar;
    if (bar) bar[(long long)row * d + t] = mean;
    x[t] = mean * (double)signs[t];
  }
  __syncthreads();
  for (int len = 1; len < d; len <<= 1) {
    if (t < d / 2) {
      const int a = (t / len) * 2 * len + (t % len);
      const double u = x[a], v = x[a + len];
      x[a] = u + v;
      x[a + len] = u - v;
    }
    __syncthreads();
  }
  if (t < r) {
    double* out = isk ? Ks : Qs;
    out[(long long)row * r + t] = x[cols[t] & (d - 1)] / sqrt((double)r);
  }
}

__global__ __launch_bounds__(256) void scores_kernel(const double* __restrict__ Qs,
                                                     const double* __restrict__ Ks, int r,
                                                     SeqMeta m,
                                                     int total_tiles, double* __restrict__ A,
                                                     double* __restrict__ A_scale) {
  const int wave = threadIdx.x >> 6;
  const int l = threadIdx.x & 63;
  const int tile = blockIdx.x * 4 + wave;
  if (tile >= total_tiles) return;
  // sequence owning the tile (aux_start holds the per-sequence tile prefix)
  int s = 0;
  while (s + 1 < m.n_seqs && m.aux_start[s + 1] <= tile) ++s;
  const int b = m.blk_start[s + 1] - m.blk_start[s];
  const int tb = (b + 15) >> 4;
  const int lt = tile - m.aux_start[s];
  const int ti = lt / tb, tj = lt % tb;
  const int bo = m.blk_start[s];
  double* As = A + m.mat_start[s];
  const double rs = 1.0 / sqrt((double)r);
  double maxabs = 0.0;
  if (tj > ti) {
    for (int v = 0; v < 4; ++v) {
      const int ri = ti * 16 + (l >> 4) + 4 * v, cj = tj * 16 + (l & 15);
      if (ri < b && cj < b) As[(long long)ri * b + cj] = 0.0;
    }
  } else {
    f64x4 acc = {0.0, 0.0, 0.0, 0.0};
    const int ra = ti * 16 + (l & 15);
    const int rb = tj * 16 + (l & 15);
    for (int k0 = 0; k0 < r; k0 += 4) {
      const int k = k0 + (l >> 4);
      const double av = (ra < b && k < r) ? Qs[(long long)(bo + ra) * r + k] : 0.0;
      const double bv = (rb < b && k < r) ? Ks[(long long)(bo + rb) * r + k] : 0.0;
      acc = __builtin_amdgcn_mfma_f64_16x16x4f64(av, bv, acc, 0, 0, 0);
    }
    for (int v = 0; v < 4; ++v) {
      const int ri = ti * 16 + (l >> 4) + 4 * v, cj = tj * 16 + (l & 15);
      if (ri < b && cj < b) {
        const double val = (cj <= ri) ? acc[v] * rs : 0.0;
        As[(long long)ri * b + cj] = val;
        maxabs = fmax(maxabs, fabs(val));
      }
    }
  }
  for (int off = 32; off > 0; off >>= 1) maxabs = fmax(maxabs, __shfl_xor(maxabs, off));
  if (l == 0 && maxabs > 0.0)
    atomicMax(reinterpret_cast<unsigned long long*>(A_scale + s),
              (unsigned long long)__double_as_longlong(maxabs));
}

static int heads_per_chunk(int h) {
  for (int c = 4; c >= 1; --c)
    if (h % c == 0) return c;
  return 1;
}

int64_t sketch_workspace_bytes(int h_q, int h_kv, int d, int64_t nb) {
  const int Pq = h_q / heads_per_chunk(h_q);
  const int Pk = h_kv / heads_per_chunk(h_kv);
  const int64_t qbytes = ((nb * Pq * d * 8) + 255) / 256 * 256;
  return qbytes + nb * Pk * d * 8;
}

hipError_t launch_sketch(int dtype, const void* Q, const void* K, int h_q, int h_kv, int d,
                         const SeqMeta& meta, int64_t nb, long long N, const int8_t* signs,
                         const int32_t* cols, int r, double* Qs, double* Ks, double* A,
                         double* A_scale, double* Qbar, double* Kbar, void* ws,
                         hipStream_t st) {
  const int hcq = heads_per_chunk(h_q), hck = heads_per_chunk(h_kv);
  const int Pq = h_q / hcq, Pk = h_kv / hck;
  double* wsq = reinterpret_cast<double*>(ws);
  const int64_t qbytes = ((nb * Pq * d * 8) + 255) / 256 * 256;
  double* wsk = reinterpret_cast<double*>(reinterpret_cast<char*>(ws) + qbytes);
  const unsigned pool_grid = (unsigned)(nb * (Pq + Pk));
  if (dtype == SW_BF16)
    hipLaunchKernelGGL(pool_kernel<uint16_t>, dim3(pool_grid), dim3(256), 0, st,
                       reinterpret_cast<const uint16_t*>(Q), hcq, Pq, wsq,
                       reinterpret_cast<const uint16_t*>(K), hck, Pk, wsk, (int)nb, d, meta, N);
  else
    hipLaunchKernelGGL(pool_kernel<float>, dim3(pool_grid), dim3(256), 0, st,
                       reinterpret_cast<const float*>(Q), hcq, Pq, wsq,
                       reinterpret_cast<const float*>(K), hck, Pk, wsk, (int)nb, d, meta, N);
  hipLaunchKernelGGL(fwht_kernel, dim3((unsigned)nb, 2), dim3(256), 0, st, wsq, wsk, Pq, Pk, h_q,
                     h_kv, d, meta, signs, cols, r, Qs, Ks, Qbar, Kbar, A_scale);
  // tile prefix per sequence
  SeqMeta m2 = meta;
  int total = 0;
  for (int s = 0; s < meta.n_seqs; ++s) {
    m2.aux_start[s] = total;
    const int b = meta.blk_start[s + 1] - meta.blk_start[s];
    const int tb = (b + 15) / 16;
    total += tb * tb;
  }
  m2.aux_start[meta.n_seqs] = total;
  hipLaunchKernelGGL(scores_kernel, dim3((unsigned)((total + 3) / 4)), dim3(256), 0, st, Qs, Ks,
                     r, m2, total, A, A_scale);
  return hipGetLastError();
}

}  // namespace sw
