// Decode path (paper Alg. 2) except the attention: one new token per sequence
// per layer.
//
//  decode_init_kernel     state of one sequence from its prompt's prefill sketch
//  kv_append_kernel       step 1: K_t, V_t into the caches at pos[b]
//  decode_reps_kernel     steps 2-3 (one workgroup per sequence): running means
//                         of the open query/key block, SRHT (in-LDS FWHT) of the
//                         token query and of both open representatives
//  decode_scores_kernel   step 4 over (sequence, 64-row chunk) workgroups, 4
//                         lanes per sketch row: (i) new score row (token query
//                         vs every earlier key block), (ii) new last column
//                         (every query block vs the open key block)
//  walk_row_strip_kernel  step 5 on the query row only: r = W[b_q, :] at the
//                         first walked layer, else r_prev W with W = (A/c)^s
//                         (or the clipped power) taken while streaming the fp32
//                         score cache; one workgroup per (sequence, 16-column
//                         strip), SW_STRIP_RG row groups reduced in LDS in a
//                         fixed order (16 columns measured 10 % faster than
//                         32 or 64: the longest strips set the time)
//  walk_row_norm_kernel   divides the row by its largest magnitude
#include "sw_common.h"
#include "sw_internal.h"

namespace sw {

// Tuning constants (overridable at build time).
#ifndef SW_STRIP_RG
#define SW_STRIP_RG 64        // row groups per walk-row strip workgroup
#endif

__device__ __forceinline__ double pow_int_d(double x, int s) {
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

// ---------------------------------------------------------------------------
// state initialisation from the prompt's prefill sketch (one sequence)
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void decode_init_kernel(char* __restrict__ state, int batch, int d,
                                                          int r, int b_max, int seq, int n, int B,
                                                          const double* __restrict__ Qs,
                                                          const double* __restrict__ Ks,
                                                          const double* __restrict__ A,
                                                          const double* __restrict__ A_scale,
                                                          const double* __restrict__ Qbar,
                                                          const double* __restrict__ Kbar) {
  const DecodeLayout L = decode_layout(batch, d, r, b_max);
  const int m = blockIdx.x;              // row of the score cache
  const int b = (n + B - 1) / B;
  float* Arow = reinterpret_cast<float*>(state + L.a) + ((long long)seq * b_max + m) * L.lda;
  for (int j = threadIdx.x; j < L.lda; j += 256)
    Arow[j] = (m < b && j < b) ? (float)A[(long long)m * b + j] : 0.0f;
  if (m < b) {
    double* qs = reinterpret_cast<double*>(state + L.qs) + ((long long)seq * b_max + m) * r;
    double* ks = reinterpret_cast<double*>(state + L.ks) + ((long long)seq * b_max + m) * r;
    for (int t = threadIdx.x; t < r; t += 256) {
      qs[t] = Qs[(long long)m * r + t];
      ks[t] = Ks[(long long)m * r + t];
    }
  }
  if (m == 0) {
    const int last = n - (b - 1) * B;    // tokens in the last (open) block
    double* bar = reinterpret_cast<double*>(state + L.bar) + (long long)seq * 2 * d;
    for (int t = threadIdx.x; t < d; t += 256) {
      bar[t] = Qbar[(long long)(b - 1) * d + t];
      bar[d + t] = Kbar[(long long)(b - 1) * d + t];
    }
    if (threadIdx.x == 0) {
      reinterpret_cast<double*>(state + L.scale)[seq] = A_scale[0];
      reinterpret_cast<int32_t*>(state + L.col0)[seq] = n / B;
      int32_t* cnt = reinterpret_cast<int32_t*>(state + L.cnt) + seq * 2;
      cnt[0] = last;
      cnt[1] = last;
    }
  }
}

// ---------------------------------------------------------------------------
// KV append
// ---------------------------------------------------------------------------

template <typename T>
__global__ __launch_bounds__(64) void kv_append_kernel(const T* __restrict__ k_new,
                                                       const T* __restrict__ v_new, T* __restrict__ Kc,
                                                       T* __restrict__ Vc, int h_kv, int d, int T_max,
                                                       const int32_t* __restrict__ pos) {
  const int bg = blockIdx.x;             // (sequence, kv head)
  const int bi = bg / h_kv;
  const int p = pos[bi];
  if (p < 0 || p >= T_max) return;
  const long long dst = ((long long)bg * T_max + p) * d;
  for (int t = threadIdx.x; t < d; t += 64) {
    Kc[dst + t] = k_new[(long long)bg * d + t];
    Vc[dst + t] = v_new[(long long)bg * d + t];
  }
}

// ---------------------------------------------------------------------------
// incremental sketch (one workgroup per sequence)
// ---------------------------------------------------------------------------

template <typename T>
__device__ __forceinline__ float load_f32(const T* p, long long i) {
  if constexpr (sizeof(T) == 2) {
    return bf16_to_f32(reinterpret_cast<const uint16_t*>(p)[i]);
  } else {
    return p[i];
  }
}

// APPEND: also writes k_new and v_new into the caches at pos (Alg. 2 step 1;
// Kc, Vc [batch][h_kv][T_max][d], 16-byte aligned rows).
template <typename T, bool APPEND>
__global__ __launch_bounds__(256) void decode_reps_kernel(const T* __restrict__ q_new,
                                                          const T* __restrict__ k_new, int h_q,
                                                          int h_kv, int d, int B,
                                                          const int32_t* __restrict__ pos,
                                                          const int8_t* __restrict__ signs,
                                                          const int32_t* __restrict__ cols, int r,
                                                          int batch, int b_max,
                                                          char* __restrict__ state,
                                                          const T* __restrict__ v_new,
                                                          T* __restrict__ Kc, T* __restrict__ Vc,
                                                          int T_max) {
  constexpr int V = 16 / (int)sizeof(T);             // elements per 16-byte load
  __shared__ double xq[256], xk[256], xb[256];
  __shared__ double pq[256 * V], pk[256 * V];
  const DecodeLayout L = decode_layout(batch, d, r, b_max);
  const int bi = blockIdx.x;
  const int t = threadIdx.x;
  const int p = pos[bi];
  const int bc = p / B;                  // open key block == query block
  if constexpr (APPEND) {
    if (p >= 0 && p < T_max) {
      const int cpr = d / V;
      for (int c = t; c < h_kv * cpr; c += 256) {
        const int g = c / cpr, o = (c % cpr) * V;
        const long long src = ((long long)bi * h_kv + g) * d + o;
        const long long dst = (((long long)bi * h_kv + g) * T_max + p) * d + o;
        *reinterpret_cast<uint4*>(Kc + dst) = *reinterpret_cast<const uint4*>(k_new + src);
        *reinterpret_cast<uint4*>(Vc + dst) = *reinterpret_cast<const uint4*>(v_new + src);
      }
    }
  }
  if (p < 0 || bc >= b_max) return;
  double* bar = reinterpret_cast<double*>(state + L.bar) + (long long)bi * 2 * d;
  int32_t* cnt = reinterpret_cast<int32_t*>(state + L.cnt) + bi * 2;
  double* Qs = reinterpret_cast<double*>(state + L.qs) + (long long)bi * b_max * r;
  double* Ks = reinterpret_cast<double*>(state + L.ks) + (long long)bi * b_max * r;
  double* qt = reinterpret_cast<double*>(state + L.qt) + (long long)bi * r;
  // head sums: thread (group, chunk) adds the 16-byte chunk `chunk` (V dims)
  // of the heads u = group, group + P, ...; then the P groups are added per dim
  const int dpc = d / V;                           // chunks per head row
  const int P = 256 / dpc;                         // head groups
  const int ch = t % dpc, grp = t / dpc;
  double sq[V], sk[V];
#pragma unroll
  for (int e = 0; e < V; ++e) sq[e] = sk[e] = 0.0;
  auto add_chunk = [&](const T* src, double (&acc)[V]) {
    const uint4 raw = *reinterpret_cast<const uint4*>(src);
    const T* v = reinterpret_cast<const T*>(&raw);
#pragma unroll
    for (int e = 0; e < V; ++e) acc[e] += (double)load_f32(v, e);
  };
#pragma unroll 4
  for (int u = grp; u < h_q; u += P) add_chunk(q_new + ((long long)bi * h_q + u) * d + ch * V, sq);
#pragma unroll 4
  for (int g = grp; g < h_kv; g += P) add_chunk(k_new + ((long long)bi * h_kv + g) * d + ch * V, sk);
#pragma unroll
  for (int e = 0; e < V; ++e) {
    pq[grp * d + ch * V + e] = sq[e];
    pk[grp * d + ch * V + e] = sk[e];
  }
  const bool fresh = (p % B) == 0;
  const int qc = cnt[0], kc = cnt[1];
  __syncthreads();
  double qa = 0.0, ka = 0.0, qbn = 0.0, kbn = 0.0;
  if (t < d) {
    for (int x = 0; x < P; ++x) {
      qa += pq[x * d + t];
      ka += pk[x * d + t];
    }
    qa /= (double)h_q;
    ka /= (double)h_kv;
    qbn = fresh ? qa : ((double)qc * bar[t] + qa) / (double)(qc + 1);
    kbn = fresh ? ka : ((double)kc * bar[d + t] + ka) / (double)(kc + 1);
  }
  __syncthreads();                       // every read of the old state is done
  if (t < d) {
    bar[t] = qbn;
    bar[d + t] = kbn;
    const double sg = (double)signs[t];
    xq[t] = qa * sg;
    xb[t] = qbn * sg;
    xk[t] = kbn * sg;
  }
  if (t == 0) {
    cnt[0] = fresh ? 1 : qc + 1;
    cnt[1] = fresh ? 1 : kc + 1;
  }
  __syncthreads();
  for (int len = 1; len < d; len <<= 1) {
    if (t < d / 2) {
      const int a = (t / len) * 2 * len + (t % len);
      double u, v;
      u = xq[a]; v = xq[a + len]; xq[a] = u + v; xq[a + len] = u - v;
      u = xb[a]; v = xb[a + len]; xb[a] = u + v; xb[a + len] = u - v;
      u = xk[a]; v = xk[a + len]; xk[a] = u + v; xk[a + len] = u - v;
    }
    __syncthreads();
  }
  const double rs = 1.0 / sqrt((double)r);
  if (t < r) {
    const int c = cols[t] & (d - 1);
    qt[t] = xq[c] * rs;
    Qs[(long long)bc * r + t] = xb[c] * rs;
    Ks[(long long)bc * r + t] = xk[c] * rs;
  }
}

constexpr int kScoreChunk = 64;

// Rows [64c, 64c+64): row entries A[bc][j] (j < bc) and column entries
// A[m][bc] (m <= bc), four threads per row.
__global__ __launch_bounds__(256) void decode_scores_kernel(const int32_t* __restrict__ pos, int r,
                                                            int B, int batch, int d, int b_max,
                                                            char* __restrict__ state) {
  const DecodeLayout L = decode_layout(batch, d, r, b_max);
  const int bi = blockIdx.x;
  const int c = blockIdx.y;
  const int p = pos[bi];
  const int bc = p / B;
  if (p < 0 || bc >= b_max) return;
  const int r0 = c * kScoreChunk;
  if (r0 > bc) return;
  const double* Qs = reinterpret_cast<const double*>(state + L.qs) + (long long)bi * b_max * r;
  const double* Ks = reinterpret_cast<const double*>(state + L.ks) + (long long)bi * b_max * r;
  const double* qt = reinterpret_cast<const double*>(state + L.qt) + (long long)bi * r;
  float* A = reinterpret_cast<float*>(state + L.a) + (long long)bi * b_max * L.lda;
  const double rs = 1.0 / sqrt((double)r);
  // four threads per row j (kScoreChunk rows per workgroup); thread q4 takes
  // the sketch coordinates k = 4 i + q4, all loads independent
  const int t = threadIdx.x;
  const int q4 = t & 3;
  const int j = r0 + (t >> 2);
  double accr = 0.0, accc = 0.0;
  if (j <= bc) {
    const double* qsj = Qs + (long long)j * r;
    const double* ksj = Ks + (long long)j * r;
    const double* ksb = Ks + (long long)bc * r;
#pragma unroll 16
    for (int k = q4; k < r; k += 4) {
      accc += qsj[k] * ksb[k];
      accr += qt[k] * ksj[k];
    }
  }
  accr += __shfl_xor(accr, 1);
  accc += __shfl_xor(accc, 1);
  accr += __shfl_xor(accr, 2);
  accc += __shfl_xor(accc, 2);
  if (q4 == 0 && j <= bc) {
    if (j < bc) A[(long long)bc * L.lda + j] = (float)(accr * rs);
    A[(long long)j * L.lda + bc] = (float)(accc * rs);
  }
}

// ---------------------------------------------------------------------------
// walk row
// ---------------------------------------------------------------------------

constexpr int kStrip = 16;               // columns per workgroup (4 lanes x 4)
constexpr int kRowGroups = SW_STRIP_RG;  // row groups per workgroup
constexpr int kStripThreads = (kStrip / 4) * kRowGroups;

// S8: s = 8, the paper's exponent (three squarings, no loop). RELU: negative
// scores are clipped to zero before the power.
template <bool S8, bool RELU>
__global__ __launch_bounds__(kStripThreads) void walk_row_strip_kernel(const char* __restrict__ state,
                                                             int batch, int d, int r, int b_max,
                                                             int B, const int32_t* __restrict__ pos,
                                                             int s_exp,
                                                             const double* __restrict__ r_prev,
                                                             double* __restrict__ r_out) {
  __shared__ double red[kRowGroups][kStrip];
  const DecodeLayout L = decode_layout(batch, d, r, b_max);
  const int bi = blockIdx.x;
  const int j0 = blockIdx.y * kStrip;
  const int p = pos[bi];
  const int bc = p / B;
  if (p < 0 || bc >= b_max) return;
  if (j0 > bc) return;
  const double c0 = reinterpret_cast<const double*>(state + L.scale)[bi];
  const double inv_c = 1.0 / (c0 > 0.0 ? c0 : 1.0);
  const int col0 = reinterpret_cast<const int32_t*>(state + L.col0)[bi];
  const float* A = reinterpret_cast<const float*>(state + L.a) + (long long)bi * b_max * L.lda;
  auto pw = [&](double x) {
    if constexpr (RELU) x = fmax(x, 0.0);
    if constexpr (S8) {
      const double x2 = x * x, x4 = x2 * x2;
      return x4 * x4;
    } else {
      return pow_int_d(x, s_exp);
    }
  };
  const int t = threadIdx.x;
  const int cq = t % (kStrip / 4), rg = t / (kStrip / 4);
  const int j = j0 + cq * 4;                       // first of this thread's 4 columns
  const bool jok = j < L.lda;                      // lda % 4 == 0: j..j+3 inside the row
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  if (!jok) {
    // columns past the padded row: nothing to accumulate
  } else if (r_prev == nullptr) {
    // first walked layer: the query row of W itself
    if (rg == 0) {
      const float4 a = *reinterpret_cast<const float4*>(A + (long long)bc * L.lda + j);
      const float av[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[e] = pw((double)av[e] * inv_c);
    }
  } else {
    const double* rp = r_prev + (long long)bi * b_max;
    // rows that can be non-zero in these columns: m >= column (causal) or any
    // row for the columns decode filled (>= col0)
    const int mstart = (j0 + kStrip - 1 >= col0) ? 0 : j0;
    int m = mstart + rg;
    for (; m + 7 * kRowGroups <= bc; m += 8 * kRowGroups) {
      float4 a[8];
      double w[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        a[u] = *reinterpret_cast<const float4*>(A + (long long)(m + u * kRowGroups) * L.lda + j);
        w[u] = rp[m + u * kRowGroups];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int mm = m + u * kRowGroups;
        const float av[4] = {a[u].x, a[u].y, a[u].z, a[u].w};
#pragma unroll
        for (int e = 0; e < 4; ++e)
          acc[e] += (j + e <= mm || j + e >= col0) ? w[u] * pw((double)av[e] * inv_c) : 0.0;
      }
    }
    for (; m <= bc; m += kRowGroups) {
      const float4 a = *reinterpret_cast<const float4*>(A + (long long)m * L.lda + j);
      const double wv = rp[m];
      const float av[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
      for (int e = 0; e < 4; ++e)
        acc[e] += (j + e <= m || j + e >= col0) ? wv * pw((double)av[e] * inv_c) : 0.0;
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) red[rg][cq * 4 + e] = acc[e];
  __syncthreads();
  if (t < kStrip) {
    double v = 0.0;
    for (int g = 0; g < kRowGroups; ++g) v += red[g][t];
    const int jj = j0 + t;
    if (jj < b_max) r_out[(long long)bi * b_max + jj] = (jj <= bc) ? v : 0.0;
  }
}

__global__ __launch_bounds__(256) void walk_row_norm_kernel(int b_max, int B,
                                                            const int32_t* __restrict__ pos,
                                                            double* __restrict__ r_out) {
  __shared__ double tmp[4];
  const int bi = blockIdx.x;
  const int p = pos[bi];
  const int bc = p / B;
  if (p < 0 || bc >= b_max) return;
  double* out = r_out + (long long)bi * b_max;
  double mx = 0.0;
  for (int j = threadIdx.x; j <= bc; j += 256) mx = fmax(mx, fabs(out[j]));
  for (int off = 32; off > 0; off >>= 1) mx = fmax(mx, __shfl_xor(mx, off));
  if ((threadIdx.x & 63) == 0) tmp[threadIdx.x >> 6] = mx;
  __syncthreads();
  mx = fmax(fmax(tmp[0], tmp[1]), fmax(tmp[2], tmp[3]));
  const double inv = mx > 0.0 ? 1.0 / mx : 1.0;
  for (int j = threadIdx.x; j < b_max; j += 256) out[j] = (j <= bc) ? out[j] * inv : 0.0;
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------

hipError_t launch_decode_init(char* state, int batch, int d, int r, int b_max, int seq, int n, int B,
                              const double* Qs, const double* Ks, const double* A,
                              const double* A_scale, const double* Qbar, const double* Kbar,
                              hipStream_t st) {
  hipLaunchKernelGGL(decode_init_kernel, dim3((unsigned)b_max), dim3(256), 0, st, state, batch, d,
                     r, b_max, seq, n, B, Qs, Ks, A, A_scale, Qbar, Kbar);
  return hipGetLastError();
}

hipError_t launch_kv_append(int dtype, const void* k_new, const void* v_new, void* Kc, void* Vc,
                            int batch, int h_kv, int d, int T_max, const int32_t* pos,
                            hipStream_t st) {
  if (dtype == SW_BF16)
    hipLaunchKernelGGL(kv_append_kernel<uint16_t>, dim3((unsigned)(batch * h_kv)), dim3(64), 0, st,
                       reinterpret_cast<const uint16_t*>(k_new),
                       reinterpret_cast<const uint16_t*>(v_new), reinterpret_cast<uint16_t*>(Kc),
                       reinterpret_cast<uint16_t*>(Vc), h_kv, d, T_max, pos);
  else
    hipLaunchKernelGGL(kv_append_kernel<float>, dim3((unsigned)(batch * h_kv)), dim3(64), 0, st,
                       reinterpret_cast<const float*>(k_new), reinterpret_cast<const float*>(v_new),
                       reinterpret_cast<float*>(Kc), reinterpret_cast<float*>(Vc), h_kv, d, T_max,
                       pos);
  return hipGetLastError();
}

namespace {

template <typename T>
void launch_reps(const void* q_new, const void* k_new, int batch, int h_q, int h_kv, int d, int B,
                 const int32_t* pos, const int8_t* signs, const int32_t* cols, int r, int b_max,
                 char* state, const void* v_new, void* Kc, void* Vc, int T_max, hipStream_t st) {
  const T* q = reinterpret_cast<const T*>(q_new);
  const T* k = reinterpret_cast<const T*>(k_new);
  const T* v = reinterpret_cast<const T*>(v_new);
  if (Kc != nullptr)
    hipLaunchKernelGGL((decode_reps_kernel<T, true>), dim3((unsigned)batch), dim3(256), 0, st, q, k,
                       h_q, h_kv, d, B, pos, signs, cols, r, batch, b_max, state, v,
                       reinterpret_cast<T*>(Kc), reinterpret_cast<T*>(Vc), T_max);
  else
    hipLaunchKernelGGL((decode_reps_kernel<T, false>), dim3((unsigned)batch), dim3(256), 0, st, q, k,
                       h_q, h_kv, d, B, pos, signs, cols, r, batch, b_max, state, v,
                       static_cast<T*>(nullptr), static_cast<T*>(nullptr), T_max);
}

}  // namespace

hipError_t launch_decode_sketch(int dtype, const void* q_new, const void* k_new, int batch, int h_q,
                                int h_kv, int d, int B, const int32_t* pos, const int8_t* signs,
                                const int32_t* cols, int r, int b_max, char* state,
                                hipStream_t st, const void* v_new, void* Kc, void* Vc, int T_max) {
  if (dtype == SW_BF16)
    launch_reps<uint16_t>(q_new, k_new, batch, h_q, h_kv, d, B, pos, signs, cols, r, b_max, state,
                          v_new, Kc, Vc, T_max, st);
  else
    launch_reps<float>(q_new, k_new, batch, h_q, h_kv, d, B, pos, signs, cols, r, b_max, state,
                       v_new, Kc, Vc, T_max, st);
  const int nch = (b_max + kScoreChunk - 1) / kScoreChunk;
  hipLaunchKernelGGL(decode_scores_kernel, dim3((unsigned)batch, (unsigned)nch), dim3(256), 0, st,
                     pos, r, B, batch, d, b_max, state);
  return hipGetLastError();
}

hipError_t launch_decode_walk(const char* state, int batch, int d, int r, int b_max, int B,
                              const int32_t* pos, int s_exp, bool relu, const double* r_prev,
                              double* r_out, hipStream_t st, bool normalize) {
  const int nstrip = (b_max + kStrip - 1) / kStrip;
  const dim3 grid((unsigned)batch, (unsigned)nstrip), blk(kStripThreads);
  if (s_exp == 8 && !relu)
    hipLaunchKernelGGL((walk_row_strip_kernel<true, false>), grid, blk, 0, st, state, batch, d, r,
                       b_max, B, pos, s_exp, r_prev, r_out);
  else if (s_exp == 8)
    hipLaunchKernelGGL((walk_row_strip_kernel<true, true>), grid, blk, 0, st, state, batch, d, r,
                       b_max, B, pos, s_exp, r_prev, r_out);
  else if (!relu)
    hipLaunchKernelGGL((walk_row_strip_kernel<false, false>), grid, blk, 0, st, state, batch, d, r,
                       b_max, B, pos, s_exp, r_prev, r_out);
  else
    hipLaunchKernelGGL((walk_row_strip_kernel<false, true>), grid, blk, 0, st, state, batch, d, r,
                       b_max, B, pos, s_exp, r_prev, r_out);
  if (normalize)
    hipLaunchKernelGGL(walk_row_norm_kernel, dim3((unsigned)batch), dim3(256), 0, st, b_max, B, pos,
                       r_out);
  return hipGetLastError();
}

}  // namespace sw
