// Decode path (paper Alg. 2): one new token per sequence per layer.
//
//  decode_init_kernel     state of one sequence from its prompt's prefill sketch
//  kv_append_kernel       step 1: K_t, V_t into the caches at pos[b]
//  decode_sketch_kernel   steps 2-4: running means of the open query/key
//                         block, SRHT of the token query and of both open
//                         representatives (in-LDS FWHT), new score row
//                         (token query vs every key block) and new last column
//                         (every query block vs the open key block)
//  walk_row_partial/finish step 5 on the query row only: r = W[b_q, :] at the
//                         first walked layer, else r_prev W, with W = (A/c)^s
//                         taken while streaming the fp32 score cache; partial
//                         sums over 64-row chunks are reduced in a fixed order
//                         (deterministic), then the row is divided by its
//                         largest magnitude
//  attn_decode_kernel     step 7, split-K: each workgroup streams an equal share
//                         of the selected tokens of one (sequence, KV head) for
//                         all G query heads of the group with 16-byte loads and
//                         keeps an online softmax per (key lane group, head)
//  attn_merge_kernel      log-sum-exp merge of the splits
#include "sw_common.h"
#include "sw_internal.h"

namespace sw {

constexpr float kLog2eD = 1.4426950408889634f;

__device__ __forceinline__ double pow_int_d(double x, int s) {
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
  float* Arow = reinterpret_cast<float*>(state + L.a) + ((long long)seq * b_max + m) * b_max;
  for (int j = threadIdx.x; j < b_max; j += 256)
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
__device__ __forceinline__ double load_f64(const T* p, long long i) {
  if constexpr (sizeof(T) == 2) {
    return (double)bf16_to_f32(reinterpret_cast<const uint16_t*>(p)[i]);
  } else {
    return (double)p[i];
  }
}

template <typename T>
__global__ __launch_bounds__(256) void decode_sketch_kernel(const T* __restrict__ q_new,
                                                            const T* __restrict__ k_new, int h_q,
                                                            int h_kv, int d, int B,
                                                            const int32_t* __restrict__ pos,
                                                            const int8_t* __restrict__ signs,
                                                            const int32_t* __restrict__ cols, int r,
                                                            int batch, int b_max,
                                                            char* __restrict__ state) {
  __shared__ double xq[256], xk[256], xb[256];
  __shared__ double qt[256], kn[256], qn[256];
  const DecodeLayout L = decode_layout(batch, d, r, b_max);
  const int bi = blockIdx.x;
  const int t = threadIdx.x;
  const int p = pos[bi];
  const int bc = p / B;                  // open key block == query block
  if (p < 0 || bc >= b_max) return;
  double* bar = reinterpret_cast<double*>(state + L.bar) + (long long)bi * 2 * d;
  int32_t* cnt = reinterpret_cast<int32_t*>(state + L.cnt) + bi * 2;
  double* Qs = reinterpret_cast<double*>(state + L.qs) + (long long)bi * b_max * r;
  double* Ks = reinterpret_cast<double*>(state + L.ks) + (long long)bi * b_max * r;
  float* A = reinterpret_cast<float*>(state + L.a) + (long long)bi * b_max * b_max;
  const bool fresh = (p % B) == 0;
  const int qc = cnt[0], kc = cnt[1];
  double qa = 0.0, ka = 0.0, qbn = 0.0, kbn = 0.0;
  if (t < d) {
    for (int u = 0; u < h_q; ++u) qa += load_f64(q_new, ((long long)bi * h_q + u) * d + t);
    for (int g = 0; g < h_kv; ++g) ka += load_f64(k_new, ((long long)bi * h_kv + g) * d + t);
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
    qn[t] = xb[c] * rs;
    kn[t] = xk[c] * rs;
    Qs[(long long)bc * r + t] = qn[t];
    Ks[(long long)bc * r + t] = kn[t];
  }
  __syncthreads();
  // groups of 8 lanes per dot product
  const int grp = t >> 3, sub = t & 7;
  // (i) new query row: token query vs key blocks j < bc (j = bc comes from (ii))
  for (int j0 = 0; j0 < bc; j0 += 32) {
    const int j = j0 + grp;
    double acc = 0.0;
    if (j < bc)
      for (int k = sub; k < r; k += 8) acc += qt[k] * Ks[(long long)j * r + k];
    acc += __shfl_xor(acc, 4);
    acc += __shfl_xor(acc, 2);
    acc += __shfl_xor(acc, 1);
    if (j < bc && sub == 0) A[(long long)bc * b_max + j] = (float)(acc * rs);
  }
  // (ii) last column: query blocks m <= bc vs the open key block
  for (int m0 = 0; m0 <= bc; m0 += 32) {
    const int m = m0 + grp;
    double acc = 0.0;
    if (m <= bc) {
      const double* qrow = (m == bc) ? qn : Qs + (long long)m * r;
      for (int k = sub; k < r; k += 8) acc += qrow[k] * kn[k];
    }
    acc += __shfl_xor(acc, 4);
    acc += __shfl_xor(acc, 2);
    acc += __shfl_xor(acc, 1);
    if (m <= bc && sub == 0) A[(long long)m * b_max + bc] = (float)(acc * rs);
  }
}

// ---------------------------------------------------------------------------
// walk row
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void walk_row_partial_kernel(const char* __restrict__ state,
                                                               int batch, int d, int r, int b_max,
                                                               int B, const int32_t* __restrict__ pos,
                                                               int s_exp,
                                                               const double* __restrict__ r_prev,
                                                               double* __restrict__ partial) {
  const DecodeLayout L = decode_layout(batch, d, r, b_max);
  const int bi = blockIdx.x;
  const int ch = blockIdx.y;
  const int p = pos[bi];
  const int bc = p / B;
  if (p < 0 || bc >= b_max) return;
  const int m0 = ch * kWalkRowChunk;
  if (m0 > bc) return;
  const int m1 = min(m0 + kWalkRowChunk, bc + 1);
  const double c0 = reinterpret_cast<const double*>(state + L.scale)[bi];
  const double inv_c = 1.0 / (c0 > 0.0 ? c0 : 1.0);
  const int col0 = reinterpret_cast<const int32_t*>(state + L.col0)[bi];
  const float* A = reinterpret_cast<const float*>(state + L.a) + (long long)bi * b_max * b_max;
  const double* rp = r_prev + (long long)bi * b_max;
  const int nch = (b_max + kWalkRowChunk - 1) / kWalkRowChunk;
  double* out = partial + ((long long)bi * nch + ch) * b_max;
  __shared__ double rv[kWalkRowChunk];
  for (int m = m0 + threadIdx.x; m < m1; m += 256) rv[m - m0] = rp[m];
  __syncthreads();
  for (int j = threadIdx.x; j <= bc; j += 256) {
    double acc = 0.0;
    // W[m][j] can be non-zero for j <= m (causal) or j >= col0 (columns
    // filled by decode for every earlier query block)
    if (j < m1 || j >= col0) {
      const int mlo = (j >= col0) ? m0 : max(m0, j);
      for (int m = mlo; m < m1; ++m)
        acc += rv[m - m0] * pow_int_d((double)A[(long long)m * b_max + j] * inv_c, s_exp);
    }
    out[j] = acc;
  }
}

__global__ __launch_bounds__(256) void walk_row_finish_kernel(const char* __restrict__ state,
                                                              int batch, int d, int r, int b_max,
                                                              int B, const int32_t* __restrict__ pos,
                                                              int s_exp, int first,
                                                              const double* __restrict__ partial,
                                                              double* __restrict__ r_out) {
  __shared__ double tmp[4];
  const DecodeLayout L = decode_layout(batch, d, r, b_max);
  const int bi = blockIdx.x;
  const int p = pos[bi];
  const int bc = p / B;
  if (p < 0 || bc >= b_max) return;
  const double c0 = reinterpret_cast<const double*>(state + L.scale)[bi];
  const double inv_c = 1.0 / (c0 > 0.0 ? c0 : 1.0);
  const float* Arow = reinterpret_cast<const float*>(state + L.a) + ((long long)bi * b_max + bc) * b_max;
  const int nch = (b_max + kWalkRowChunk - 1) / kWalkRowChunk;
  const int used = bc / kWalkRowChunk + 1;
  double* out = r_out + (long long)bi * b_max;
  double mx = 0.0;
  for (int j = threadIdx.x; j < b_max; j += 256) {
    double v = 0.0;
    if (j <= bc) {
      if (first) {
        v = pow_int_d((double)Arow[j] * inv_c, s_exp);
      } else {
        for (int c = 0; c < used; ++c) v += partial[((long long)bi * nch + c) * b_max + j];
      }
    }
    out[j] = v;
    mx = fmax(mx, fabs(v));
  }
  for (int off = 32; off > 0; off >>= 1) mx = fmax(mx, __shfl_xor(mx, off));
  if ((threadIdx.x & 63) == 0) tmp[threadIdx.x >> 6] = mx;
  __syncthreads();
  mx = fmax(fmax(tmp[0], tmp[1]), fmax(tmp[2], tmp[3]));
  if (mx > 0.0) {
    const double inv = 1.0 / mx;
    for (int j = threadIdx.x; j <= bc; j += 256) out[j] = out[j] * inv;
  }
}

// ---------------------------------------------------------------------------
// split-K decode attention
// ---------------------------------------------------------------------------

// LPK lanes share one key row (8 elements of 16 bytes each... per lane: 8
// elements); KPW = 64 / LPK keys per wavefront per step.
template <typename T, int D, int G>
__global__ __launch_bounds__(256) void attn_decode_kernel(const T* __restrict__ q,
                                                          const T* __restrict__ Kc,
                                                          const T* __restrict__ Vc, int h_kv,
                                                          int T_max, int B,
                                                          const int32_t* __restrict__ pos,
                                                          const int32_t* __restrict__ idx,
                                                          const int32_t* __restrict__ cnt,
                                                          int kmax, float sl2, int S,
                                                          float* __restrict__ ws) {
  constexpr int EPL = 16 / sizeof(T);            // elements per lane per row
  constexpr int LPK = D / EPL;                   // lanes per key row
  constexpr int KPW = 64 / LPK;                  // key rows per wave per step
  constexpr int NG = 4 * KPW;                    // key groups per workgroup
  __shared__ float sm_m[NG][G], sm_l[NG][G];
  __shared__ float sm_o[NG][G][D];
  const int sp = blockIdx.x % S;
  const int bg = blockIdx.x / S;                 // (sequence, kv head)
  const int bi = bg / h_kv;
  const int g = bg % h_kv;
  const int h_q = h_kv * G;
  const int tid = threadIdx.x;
  const int w = tid >> 6, l = tid & 63;
  const int kg = l / LPK, sub = l % LPK;
  const int grp = w * KPW + kg;                  // key group id in the workgroup
  const int p = pos[bi];
  const bool ok = p >= 0 && p < T_max;
  const int bc = ok ? p / B : 0;
  const int tau = ok ? max(0, min(cnt[bi], kmax)) : 0;
  const long long total = (long long)tau * B;
  const long long f0 = total * sp / S, f1 = total * (sp + 1) / S;
  const int32_t* sel = idx + (long long)bi * kmax;

  float qv[G][EPL];
#pragma unroll
  for (int u = 0; u < G; ++u) {
    const T* qp = q + ((long long)bi * h_q + g * G + u) * D + sub * EPL;
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      if constexpr (sizeof(T) == 2)
        qv[u][e] = bf16_to_f32(reinterpret_cast<const uint16_t*>(qp)[e]) * sl2;
      else
        qv[u][e] = qp[e] * sl2;
    }
  }
  float mrun[G], lrun[G], o[G][EPL];
#pragma unroll
  for (int u = 0; u < G; ++u) {
    mrun[u] = -INFINITY;
    lrun[u] = 0.0f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) o[u][e] = 0.0f;
  }
  const T* Kb = Kc + (long long)bg * T_max * D + sub * EPL;
  const T* Vb = Vc + (long long)bg * T_max * D + sub * EPL;

  for (long long f = f0 + grp; f < f1; f += NG) {
    const int jj = (int)(f / B);
    const int off = (int)(f % B);
    const int j = sel[jj];
    const int tok = j * B + off;
    const bool valid = (j >= 0 && j <= bc && tok <= p);
    uint4 kraw = make_uint4(0, 0, 0, 0), vraw = make_uint4(0, 0, 0, 0);
    if (valid) {
      kraw = *reinterpret_cast<const uint4*>(Kb + (long long)tok * D);
      vraw = *reinterpret_cast<const uint4*>(Vb + (long long)tok * D);
    }
    float kf[EPL], vf[EPL];
    if constexpr (sizeof(T) == 2) {
      const uint32_t kw[4] = {kraw.x, kraw.y, kraw.z, kraw.w};
      const uint32_t vw[4] = {vraw.x, vraw.y, vraw.z, vraw.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        kf[2 * e] = __uint_as_float(kw[e] << 16);
        kf[2 * e + 1] = __uint_as_float(kw[e] & 0xffff0000u);
        vf[2 * e] = __uint_as_float(vw[e] << 16);
        vf[2 * e + 1] = __uint_as_float(vw[e] & 0xffff0000u);
      }
    } else {
      kf[0] = __uint_as_float(kraw.x); kf[1] = __uint_as_float(kraw.y);
      kf[2] = __uint_as_float(kraw.z); kf[3] = __uint_as_float(kraw.w);
      vf[0] = __uint_as_float(vraw.x); vf[1] = __uint_as_float(vraw.y);
      vf[2] = __uint_as_float(vraw.z); vf[3] = __uint_as_float(vraw.w);
    }
    float s[G];
#pragma unroll
    for (int u = 0; u < G; ++u) {
      float a = 0.0f;
#pragma unroll
      for (int e = 0; e < EPL; ++e) a += qv[u][e] * kf[e];
#pragma unroll
      for (int off2 = LPK / 2; off2 > 0; off2 >>= 1) a += __shfl_xor(a, off2);
      s[u] = valid ? a : -INFINITY;
    }
    if (valid) {
#pragma unroll
      for (int u = 0; u < G; ++u) {
        const float mnew = fmaxf(mrun[u], s[u]);
        const float alpha = exp2f(mrun[u] - mnew);
        const float pv = exp2f(s[u] - mnew);
        mrun[u] = mnew;
        lrun[u] = lrun[u] * alpha + pv;
#pragma unroll
        for (int e = 0; e < EPL; ++e) o[u][e] = o[u][e] * alpha + pv * vf[e];
      }
    }
  }
  // combine the key groups of the workgroup
#pragma unroll
  for (int u = 0; u < G; ++u) {
    if (sub == 0) {
      sm_m[grp][u] = mrun[u];
      sm_l[grp][u] = lrun[u];
    }
#pragma unroll
    for (int e = 0; e < EPL; ++e) sm_o[grp][u][sub * EPL + e] = o[u][e];
  }
  __syncthreads();
  const int nsp = S;
  float* ws_ml = ws;                                          // [bi][u][S][2]
  float* ws_o = ws + (long long)gridDim.x / S * G * nsp * 2;  // [bi][u][S][D]
  for (int x = tid; x < G * D; x += 256) {
    const int u = x / D, dim = x % D;
    float M = -INFINITY;
    for (int k = 0; k < NG; ++k) M = fmaxf(M, sm_m[k][u]);
    float Lsum = 0.0f, Osum = 0.0f;
    if (M != -INFINITY) {
      for (int k = 0; k < NG; ++k) {
        const float sc = exp2f(sm_m[k][u] - M);
        Lsum += sm_l[k][u] * sc;
        Osum += sm_o[k][u][dim] * sc;
      }
    }
    const long long hu = (long long)bi * h_q + g * G + u;   // global (sequence, q head)
    ws_o[(hu * nsp + sp) * D + dim] = Osum;
    if (dim == 0) {
      ws_ml[(hu * nsp + sp) * 2 + 0] = M;
      ws_ml[(hu * nsp + sp) * 2 + 1] = Lsum;
    }
  }
}

template <typename T>
__global__ __launch_bounds__(128) void attn_merge_kernel(const float* __restrict__ ws, int S, int D,
                                                         long long n_hu, T* __restrict__ O) {
  const long long hu = blockIdx.x;
  const float* ws_ml = ws;
  const float* ws_o = ws + n_hu * S * 2;
  float M = -INFINITY;
  for (int s = 0; s < S; ++s) M = fmaxf(M, ws_ml[(hu * S + s) * 2]);
  for (int dim = threadIdx.x; dim < D; dim += 128) {
    float Lsum = 0.0f, Osum = 0.0f;
    if (M != -INFINITY) {
      for (int s = 0; s < S; ++s) {
        const float sc = exp2f(ws_ml[(hu * S + s) * 2] - M);
        Lsum += ws_ml[(hu * S + s) * 2 + 1] * sc;
        Osum += ws_o[(hu * S + s) * D + dim] * sc;
      }
    }
    const float v = Lsum > 0.0f ? Osum / Lsum : 0.0f;
    if constexpr (sizeof(T) == 2)
      reinterpret_cast<uint16_t*>(O)[hu * D + dim] = f32_to_bf16(v);
    else
      O[hu * D + dim] = v;
  }
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

hipError_t launch_decode_sketch(int dtype, const void* q_new, const void* k_new, int batch, int h_q,
                                int h_kv, int d, int B, const int32_t* pos, const int8_t* signs,
                                const int32_t* cols, int r, int b_max, char* state,
                                hipStream_t st) {
  if (dtype == SW_BF16)
    hipLaunchKernelGGL(decode_sketch_kernel<uint16_t>, dim3((unsigned)batch), dim3(256), 0, st,
                       reinterpret_cast<const uint16_t*>(q_new),
                       reinterpret_cast<const uint16_t*>(k_new), h_q, h_kv, d, B, pos, signs, cols,
                       r, batch, b_max, state);
  else
    hipLaunchKernelGGL(decode_sketch_kernel<float>, dim3((unsigned)batch), dim3(256), 0, st,
                       reinterpret_cast<const float*>(q_new), reinterpret_cast<const float*>(k_new),
                       h_q, h_kv, d, B, pos, signs, cols, r, batch, b_max, state);
  return hipGetLastError();
}

hipError_t launch_decode_walk(const char* state, int batch, int d, int r, int b_max, int B,
                              const int32_t* pos, int s_exp, const double* r_prev, double* r_out,
                              double* partial, hipStream_t st) {
  const int nch = (b_max + kWalkRowChunk - 1) / kWalkRowChunk;
  if (r_prev != nullptr)
    hipLaunchKernelGGL(walk_row_partial_kernel, dim3((unsigned)batch, (unsigned)nch), dim3(256), 0,
                       st, state, batch, d, r, b_max, B, pos, s_exp, r_prev, partial);
  hipLaunchKernelGGL(walk_row_finish_kernel, dim3((unsigned)batch), dim3(256), 0, st, state, batch,
                     d, r, b_max, B, pos, s_exp, r_prev == nullptr ? 1 : 0, partial, r_out);
  return hipGetLastError();
}

int decode_attn_splits(int batch, int h_kv) {
  const int pairs = batch * h_kv;
  int S = (1024 + pairs - 1) / pairs;
  if (S < 1) S = 1;
  if (S > kDecodeMaxSplits) S = kDecodeMaxSplits;
  return S;
}

template <typename T, int D>
static void launch_attn_decode_t(int G, dim3 grid, hipStream_t st, const T* q, const T* Kc,
                                 const T* Vc, int h_kv, int T_max, int B, const int32_t* pos,
                                 const int32_t* idx, const int32_t* cnt, int kmax, float sl2,
                                 int S, float* ws) {
  switch (G) {
    case 1: hipLaunchKernelGGL((attn_decode_kernel<T, D, 1>), grid, dim3(256), 0, st, q, Kc, Vc, h_kv, T_max, B, pos, idx, cnt, kmax, sl2, S, ws); break;
    case 2: hipLaunchKernelGGL((attn_decode_kernel<T, D, 2>), grid, dim3(256), 0, st, q, Kc, Vc, h_kv, T_max, B, pos, idx, cnt, kmax, sl2, S, ws); break;
    case 4: hipLaunchKernelGGL((attn_decode_kernel<T, D, 4>), grid, dim3(256), 0, st, q, Kc, Vc, h_kv, T_max, B, pos, idx, cnt, kmax, sl2, S, ws); break;
    default: hipLaunchKernelGGL((attn_decode_kernel<T, D, 8>), grid, dim3(256), 0, st, q, Kc, Vc, h_kv, T_max, B, pos, idx, cnt, kmax, sl2, S, ws); break;
  }
}

hipError_t launch_attn_decode(int dtype, const void* q, const void* Kc, const void* Vc, int batch,
                              int h_q, int h_kv, int d, int T_max, int B, const int32_t* pos,
                              const int32_t* idx, const int32_t* cnt, int kmax, float scale,
                              void* O, float* ws, hipStream_t st) {
  const int G = h_q / h_kv;
  const int S = decode_attn_splits(batch, h_kv);
  const dim3 grid((unsigned)(batch * h_kv * S));
  const float sl2 = scale * kLog2eD;
  const long long n_hu = (long long)batch * h_q;
  if (dtype == SW_BF16) {
    auto qq = reinterpret_cast<const uint16_t*>(q);
    auto kk = reinterpret_cast<const uint16_t*>(Kc);
    auto vv = reinterpret_cast<const uint16_t*>(Vc);
    if (d == 128) launch_attn_decode_t<uint16_t, 128>(G, grid, st, qq, kk, vv, h_kv, T_max, B, pos, idx, cnt, kmax, sl2, S, ws);
    else launch_attn_decode_t<uint16_t, 64>(G, grid, st, qq, kk, vv, h_kv, T_max, B, pos, idx, cnt, kmax, sl2, S, ws);
    hipLaunchKernelGGL(attn_merge_kernel<uint16_t>, dim3((unsigned)n_hu), dim3(128), 0, st, ws, S, d,
                       n_hu, reinterpret_cast<uint16_t*>(O));
  } else {
    auto qq = reinterpret_cast<const float*>(q);
    auto kk = reinterpret_cast<const float*>(Kc);
    auto vv = reinterpret_cast<const float*>(Vc);
    if (d == 128) launch_attn_decode_t<float, 128>(G, grid, st, qq, kk, vv, h_kv, T_max, B, pos, idx, cnt, kmax, sl2, S, ws);
    else launch_attn_decode_t<float, 64>(G, grid, st, qq, kk, vv, h_kv, T_max, B, pos, idx, cnt, kmax, sl2, S, ws);
    hipLaunchKernelGGL(attn_merge_kernel<float>, dim3((unsigned)n_hu), dim3(128), 0, st, ws, S, d, n_hu,
                       reinterpret_cast<float*>(O));
  }
  return hipGetLastError();
}

}  // namespace sw
