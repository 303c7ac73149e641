// Small-World Sketching kernels (paper Sec. 2.2, Alg. 1 steps 1-5).
//
//  pool_sketch_kernel  one workgroup per block row: streams the row's tokens
//                      of every query head and every KV head once from HBM
//                      (16-byte non-temporal loads), sums them in fp64 (lanes
//                      of a wavefront combined by lane exchanges, then the
//                      wavefronts in a fixed order), divides by heads x
//                      tokens, applies the random signs, runs the
//                      Walsh-Hadamard transform of the query mean and of the
//                      key mean (one wavefront each, lane exchanges), samples
//                      the columns and scales by 1/sqrt(r).
//  scores_kernel       A = Qs Ks^T / sqrt(r) with fp64 MFMA 16x16x4 tiles,
//                      causal mask, per-sequence max |A| by integer atomicMax
//                      on the (non-negative) double bit pattern.
#include "sw_common.h"
#include "sw_internal.h"

#define SW_STR2(x) #x
#define SW_STR(x) SW_STR2(x)

namespace sw {

typedef double f64x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

#ifndef SW_POOL_THREADS
#define SW_POOL_THREADS 512
#endif
constexpr int kPoolThreads = SW_POOL_THREADS;
#ifndef SW_POOL_UNROLL
#define SW_POOL_UNROLL 8
#endif

template <typename T>
__global__ __launch_bounds__(kPoolThreads) void pool_sketch_kernel(
    const T* __restrict__ Q, const T* __restrict__ K, int h_q, int h_kv, int d, SeqMeta m,
    long long N, const int8_t* __restrict__ signs, const int32_t* __restrict__ cols, int r,
    double* __restrict__ Qs, double* __restrict__ Ks, double* __restrict__ Qbar,
    double* __restrict__ Kbar, double* __restrict__ A_scale) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int NW = kPoolThreads / 64;
  // per-wavefront sums of the query and key means, then (reused) the two
  // vectors the transforms work on
  __shared__ double red[2 * NW * 256];
  double* redq = red;
  double* redk = red + NW * 256;
  double* xq = red;
  double* xk = red + 256;
  const int row = blockIdx.x;
  const int s = seq_of_block(m, row);
  const int i = row - m.blk_start[s];
  const int t0 = m.tok_start[s] + i * m.B;
  const int cnt = min(m.tok_start[s + 1], t0 + m.B) - t0;
  const int t = threadIdx.x;
  const int lpr = d / VEC;               // lanes per token row (2 .. 64)
  const int slots = kPoolThreads / lpr;  // token rows in flight per pass
  const int lane = t % lpr;
  const int slot = t / lpr;
  if (i == 0 && t == 0) A_scale[s] = 0.0;

  auto add = [](double (&acc)[VEC], const T* p) {
    // non-temporal: Q and K are streamed once here
    const u32x4 vv = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[2 * e] += (double)__uint_as_float(vv[e] << 16);
        acc[2 * e + 1] += (double)__uint_as_float(vv[e] & 0xffff0000u);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[e] += (double)__uint_as_float(vv[e]);
    }
  };
  // item it = head * cnt + token, slot-strided
  double aq[VEC], ak[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) aq[e] = ak[e] = 0.0;
  // items (head, token) in head-major order, `slots` apart: the head and
  // token of the next item follow by subtraction, not division
  const int nq = h_q * cnt, nk = h_kv * cnt;
  const int dh = slots / cnt, dt = slots % cnt;
  {
    int h = slot / cnt, tok = slot % cnt;
_Pragma(SW_STR(unroll SW_POOL_UNROLL))
    for (int it = slot; it < nq; it += slots) {
      add(aq, Q + ((long long)h * N + t0 + tok) * d + lane * VEC);
      h += dh;
      tok += dt;
      if (tok >= cnt) {
        tok -= cnt;
        ++h;
      }
    }
  }
  {
    int h = slot / cnt, tok = slot % cnt;
_Pragma(SW_STR(unroll SW_POOL_UNROLL))
    for (int it = slot; it < nk; it += slots) {
      add(ak, K + ((long long)h * N + t0 + tok) * d + lane * VEC);
      h += dh;
      tok += dt;
      if (tok >= cnt) {
        tok -= cnt;
        ++h;
      }
    }
  }
  // the slots of a wavefront share dimensions across lanes lpr apart
  for (int off = lpr; off < 64; off <<= 1) {
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      aq[e] += __shfl_xor(aq[e], off);
      ak[e] += __shfl_xor(ak[e], off);
    }
  }
  const int wv = t >> 6;
  if ((t & 63) < lpr) {
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      redq[wv * d + lane * VEC + e] = aq[e];
      redk[wv * d + lane * VEC + e] = ak[e];
    }
  }
  __syncthreads();
  double mq = 0.0, mk = 0.0;
  if (t < d) {
    double sq = 0.0, sk = 0.0;
    for (int w = 0; w < NW; ++w) {
      sq += redq[w * d + t];
      sk += redk[w * d + t];
    }
    mq = sq / ((double)h_q * (double)cnt);
    mk = sk / ((double)h_kv * (double)cnt);
    if (Qbar) Qbar[(long long)row * d + t] = mq;
    if (Kbar) Kbar[(long long)row * d + t] = mk;
  }
  __syncthreads();                       // the sums are read; xq/xk reuse them
  if (t < d) {
    const double sg = (double)signs[t];
    xq[t] = mq * sg;
    xk[t] = mk * sg;
  }
  __syncthreads();
  if (wv == 0) wave_fwht(xq, d);
  else if (wv == 1) wave_fwht(xk, d);
  __syncthreads();
  if (t < r) {
    const int c = cols[t] & (d - 1);
    Qs[(long long)row * r + t] = xq[c] / sqrt((double)r);
    Ks[(long long)row * r + t] = xk[c] / sqrt((double)r);
  }
}

// Four 16 x 16 tiles per workgroup, one per wavefront; the per-sequence max
// |A| is reduced over the workgroup's tiles first, so a sequence receives one
// atomicMax per workgroup. The k-range is taken in chunks of 64: in a chunk,
// lane group q = l / 16 carries k = 64 c + 16 q + u in MFMA step u (the dot
// product runs over every k once), so each lane reads 16 consecutive entries
// of its row; every load of a chunk is issued before the first MFMA (indices
// clamped, entries past r zeroed after the load).
__global__ __launch_bounds__(256) void scores_kernel(const double* __restrict__ Qs,
                                                     const double* __restrict__ Ks, int r,
                                                     SeqMeta m,
                                                     int total_tiles, double* __restrict__ A,
                                                     double* __restrict__ A_scale) {
  __shared__ double wmax[4];
  __shared__ int wseq[4];
  const int wave = threadIdx.x >> 6;
  const int l = threadIdx.x & 63;
  const int tile = blockIdx.x * 4 + wave;
  double maxabs = 0.0;
  int s = -1;
  if (tile < total_tiles) {
    // sequence owning the tile (aux_start holds the per-sequence tile prefix)
    s = 0;
    while (s + 1 < m.n_seqs && m.aux_start[s + 1] <= tile) ++s;
    const int b = m.blk_start[s + 1] - m.blk_start[s];
    const int tb = (b + 15) >> 4;
    const int lt = tile - m.aux_start[s];
    const int ti = lt / tb, tj = lt % tb;
    const int bo = m.blk_start[s];
    double* As = A + m.mat_start[s];
    const double rs = 1.0 / sqrt((double)r);
    if (tj > ti) {
      for (int v = 0; v < 4; ++v) {
        const int ri = ti * 16 + (l >> 4) + 4 * v, cj = tj * 16 + (l & 15);
        if (ri < b && cj < b) As[(long long)ri * b + cj] = 0.0;
      }
    } else {
      f64x4 acc = {0.0, 0.0, 0.0, 0.0};
      // rows past the sequence's last block are clamped (their results are
      // not stored)
      const double* qa = Qs + (long long)(bo + min(ti * 16 + (l & 15), b - 1)) * r;
      const double* kb = Ks + (long long)(bo + min(tj * 16 + (l & 15), b - 1)) * r;
      const int kq = 16 * (l >> 4);
      for (int c0 = 0; c0 < r; c0 += 64) {
        double av[16], bv[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          const int k = min(c0 + kq + u, r - 1);
          av[u] = qa[k];
          bv[u] = kb[k];
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          const bool in = c0 + kq + u < r;
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64(in ? av[u] : 0.0, in ? bv[u] : 0.0, acc, 0,
                                                     0, 0);
        }
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
  }
  for (int off = 32; off > 0; off >>= 1) maxabs = fmax(maxabs, __shfl_xor(maxabs, off));
  if (l == 0) {
    wmax[wave] = maxabs;
    wseq[wave] = s;
  }
  __syncthreads();
  if (threadIdx.x < 4) {
    // wavefront w reports for its sequence if no earlier wavefront has it
    const int w = threadIdx.x, sw_ = wseq[w];
    bool first = sw_ >= 0;
    double mx = 0.0;
    for (int x = 0; x < 4; ++x) {
      if (wseq[x] == sw_) {
        if (x < w) first = false;
        mx = fmax(mx, wmax[x]);
      }
    }
    if (first && mx > 0.0)
      atomicMax(reinterpret_cast<unsigned long long*>(A_scale + sw_),
                (unsigned long long)__double_as_longlong(mx));
  }
}

int64_t sketch_workspace_bytes(int, int, int, int64_t) { return 0; }

hipError_t launch_sketch(int dtype, const void* Q, const void* K, int h_q, int h_kv, int d,
                         const SeqMeta& meta, int64_t nb, long long N, const int8_t* signs,
                         const int32_t* cols, int r, double* Qs, double* Ks, double* A,
                         double* A_scale, double* Qbar, double* Kbar, void* /*ws*/,
                         hipStream_t st) {
  if (dtype == SW_BF16)
    hipLaunchKernelGGL(pool_sketch_kernel<uint16_t>, dim3((unsigned)nb), dim3(kPoolThreads), 0, st,
                       reinterpret_cast<const uint16_t*>(Q), reinterpret_cast<const uint16_t*>(K),
                       h_q, h_kv, d, meta, N, signs, cols, r, Qs, Ks, Qbar, Kbar, A_scale);
  else
    hipLaunchKernelGGL(pool_sketch_kernel<float>, dim3((unsigned)nb), dim3(kPoolThreads), 0, st,
                       reinterpret_cast<const float*>(Q), reinterpret_cast<const float*>(K), h_q,
                       h_kv, d, meta, N, signs, cols, r, Qs, Ks, Qbar, Kbar, A_scale);
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
