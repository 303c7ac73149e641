// Decode attention (paper Alg. 2 step 7): single-token softmax attention over
// the tokens of the selected key blocks, split-K over those tokens.
//
//  attn_decode_mfma_kernel  bf16: one workgroup per (sequence, KV head, split);
//                           the split's selected-block list is staged in LDS,
//                           K/V groups of 16 tokens are streamed with raw buffer
//                           loads and the G query heads of the KV group are
//                           scored and accumulated on MFMA
//  attn_decode_kernel       fp32: each workgroup streams an equal share of the
//                           selected tokens of one (sequence, KV head) for all
//                           G query heads of the group with 16-byte loads and
//                           keeps an online softmax per (key lane group, head)
//  attn_merge_kernel        log-sum-exp merge of the splits
#include <mutex>

#include "sw_common.h"
#include "sw_internal.h"

namespace sw {

constexpr float kLog2eD = 1.4426950408889634f;

// Combine a lane's value with that of lane ^ 16 / lane ^ 32 through the
// permlane swaps (VALU moves; each returns the lane's own value and its
// partner's in some order).
__device__ __forceinline__ float fmax_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float fmax_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
constexpr int kDecodeSelCache = 512;   // selected-block entries cached per workgroup

// Tuning constants (overridable at build time).
#ifndef SW_DEC_GPS
#define SW_DEC_GPS 2          // 16-token groups per wavefront step in decode attention
#endif
#ifndef SW_DEC_WGS
#define SW_DEC_WGS 512        // target decode-attention workgroups per launch
#endif
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

  // this workgroup's slice of the selected-block list, cached in LDS
  __shared__ int sel_sh[kDecodeSelCache];
  const int jj0 = (int)(f0 / B);
  const int nsh = (f1 > f0) ? (int)((f1 - 1) / B) - jj0 + 1 : 0;
  const bool cached = nsh <= kDecodeSelCache;
  if (cached)
    for (int x = tid; x < nsh; x += 256) sel_sh[x] = sel[jj0 + x];
  __syncthreads();

  constexpr int U = 4;                           // tokens per key group per step
  for (long long fb = f0 + (long long)grp * U; fb < f1; fb += (long long)NG * U) {
    uint4 kraw[U], vraw[U];
    bool valid[U];
#pragma unroll
    for (int x = 0; x < U; ++x) {
      const long long f = fb + x;
      bool ok2 = f < f1;
      int tok = 0;
      if (ok2) {
        const int jj = (int)(f / B);
        const int off = (int)(f - (long long)jj * B);
        const int j = cached ? sel_sh[jj - jj0] : sel[jj];
        tok = j * B + off;
        ok2 = (j >= 0 && j <= bc && tok <= p);
      }
      valid[x] = ok2;
      kraw[x] = make_uint4(0, 0, 0, 0);
      vraw[x] = make_uint4(0, 0, 0, 0);
      if (ok2) {
        kraw[x] = *reinterpret_cast<const uint4*>(Kb + (long long)tok * D);
        vraw[x] = *reinterpret_cast<const uint4*>(Vb + (long long)tok * D);
      }
    }
    float sc[U][G];
#pragma unroll
    for (int x = 0; x < U; ++x) {
      float kf[EPL];
      if constexpr (sizeof(T) == 2) {
        const uint32_t kw[4] = {kraw[x].x, kraw[x].y, kraw[x].z, kraw[x].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          kf[2 * e] = __uint_as_float(kw[e] << 16);
          kf[2 * e + 1] = __uint_as_float(kw[e] & 0xffff0000u);
        }
      } else {
        kf[0] = __uint_as_float(kraw[x].x); kf[1] = __uint_as_float(kraw[x].y);
        kf[2] = __uint_as_float(kraw[x].z); kf[3] = __uint_as_float(kraw[x].w);
      }
#pragma unroll
      for (int u = 0; u < G; ++u) {
        float a = 0.0f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) a += qv[u][e] * kf[e];
#pragma unroll
        for (int off2 = LPK / 2; off2 > 0; off2 >>= 1) a += __shfl_xor(a, off2);
        sc[x][u] = valid[x] ? a : -INFINITY;
      }
    }
    float vf[U][EPL];
#pragma unroll
    for (int x = 0; x < U; ++x) {
      if constexpr (sizeof(T) == 2) {
        const uint32_t vw[4] = {vraw[x].x, vraw[x].y, vraw[x].z, vraw[x].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          vf[x][2 * e] = __uint_as_float(vw[e] << 16);
          vf[x][2 * e + 1] = __uint_as_float(vw[e] & 0xffff0000u);
        }
      } else {
        vf[x][0] = __uint_as_float(vraw[x].x); vf[x][1] = __uint_as_float(vraw[x].y);
        vf[x][2] = __uint_as_float(vraw[x].z); vf[x][3] = __uint_as_float(vraw[x].w);
      }
    }
#pragma unroll
    for (int u = 0; u < G; ++u) {
      float mx = sc[0][u];
#pragma unroll
      for (int x = 1; x < U; ++x) mx = fmaxf(mx, sc[x][u]);
      if (mx == -INFINITY) continue;               // no valid token in this step
      const float mnew = fmaxf(mrun[u], mx);
      const float alpha = exp2f(mrun[u] - mnew);
      float pv[U];
      float ps = 0.0f;
#pragma unroll
      for (int x = 0; x < U; ++x) {
        pv[x] = exp2f(sc[x][u] - mnew);
        ps += pv[x];
      }
      mrun[u] = mnew;
      lrun[u] = lrun[u] * alpha + ps;
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        float acc = o[u][e] * alpha;
#pragma unroll
        for (int x = 0; x < U; ++x) acc += pv[x] * vf[x][e];
        o[u][e] = acc;
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

// bf16 split-K decode attention on MFMA. Workgroup = (sequence, KV head,
// split), 4 wavefronts; a wavefront takes groups of 16 consecutive selected
// tokens, GPS groups per step, loading the groups of step it+1 while it
// computes step it (two register sets, the step loop unrolled by two so
// neither set is copied).
//   S = K q^T   v_mfma_f32_16x16x32_bf16: A = 16 key rows x 32 dims read
//               straight from the cache (16 bytes per lane), B = the G query
//               heads (zero-padded to 16 columns). Lane n + 16 (m / 4) holds
//               key m of head n, so the online-softmax state of a head stays
//               in the lane (plus two exchanges for the max).
//   O^T += V^T P^T  v_mfma_f32_16x16x16bf16_1k: A = V^T from a per-wave LDS
//               slice written transposed (4 keys x 8 dims per lane), B = P in
//               the accumulator layout of S.
// The split's block indices are staged in LDS once, and the K/V loads go
// through buffer descriptors that end at the last valid token (lanes past it
// read zero), so the loop has no global index loads and no per-lane branches
// around loads: the loads of the next step stay in flight during the math.
typedef __bf16 bf16x8d __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4d __attribute__((ext_vector_type(4)));

constexpr int kDecBufWord3 = 0x00020000;   // raw buffer descriptor word 3 (gfx9 family)

template <int D>
__global__ __launch_bounds__(256) void attn_decode_mfma_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ Kc, const uint16_t* __restrict__ Vc,
    int h_kv, int G, int T_max, int B, const int32_t* __restrict__ pos,
    const int32_t* __restrict__ idx, const int32_t* __restrict__ cnt, int kmax, float sl2, int S,
    float* __restrict__ ws) {
  constexpr int VTS = 16 + 4;                      // V^T row stride (keys + pad)
  constexpr int GPS = SW_DEC_GPS;                  // 16-token groups per wave step
  // LDS: per-wave V^T slices during the loop; the epilogue's partials reuse it
  constexpr int VT_BYTES = 4 * GPS * D * VTS * 2;
  constexpr int EP_BYTES = (4 * 16 * D + 2 * 4 * 16) * 4;
  __shared__ __attribute__((aligned(16))) char smem[VT_BYTES > EP_BYTES ? VT_BYTES : EP_BYTES];
  __shared__ int16_t ssel[SW_MAX_BLOCKS + 2];      // this split's block indices
  auto vt_slice = [&](int wv, int x) {
    return reinterpret_cast<uint16_t*>(smem) + (wv * GPS + x) * D * VTS;
  };
  float (*sm_o)[16][D] = reinterpret_cast<float (*)[16][D]>(smem);
  float (*sm_m)[16] = reinterpret_cast<float (*)[16]>(smem + 4 * 16 * D * 4);
  float (*sm_l)[16] = reinterpret_cast<float (*)[16]>(smem + 4 * 16 * D * 4 + 4 * 16 * 4);
  const int sp = blockIdx.x % S;
  const int bg = blockIdx.x / S;                   // (sequence, kv head)
  const int bi = bg / h_kv;
  const int g = bg % h_kv;
  const int h_q = h_kv * G;
  const int tid = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6), l = tid & 63;
  const int ln = l & 15, lg = l >> 4;
  const int p = pos[bi];
  const bool ok = p >= 0 && p < T_max;
  const int bc = ok ? p / B : 0;
  // a valid selection has at most SW_MAX_BLOCKS distinct blocks
  const int tau = ok ? max(0, min(min(cnt[bi], kmax), SW_MAX_BLOCKS)) : 0;
  const int gpb = B / 16;                          // 16-token groups per block
  const int ngroups = tau * gpb;
  const int g0 = (int)((long long)ngroups * sp / S), g1 = (int)((long long)ngroups * (sp + 1) / S);
  const int jlo = g0 / gpb;
  const int nj = (g1 > g0) ? (g1 - 1) / gpb - jlo + 1 : 0;
  {
    const int32_t* sel = idx + (long long)bi * kmax + jlo;
    for (int e = tid; e < nj; e += 256) ssel[e] = (int16_t)max(-1, min(sel[e], 32767));
  }

  // query fragments (B operand of S = K q^T): head ln, dims 32c + 8 lg .. +7
  bf16x8d qf[D / 32];
  {
    const bool hv = ln < G;
    const uint16_t* qp = q + ((long long)bi * h_q + g * G + (hv ? ln : 0)) * D + lg * 8;
#pragma unroll
    for (int c = 0; c < D / 32; ++c) {
      uint4 v = hv ? *reinterpret_cast<const uint4*>(qp + 32 * c) : make_uint4(0, 0, 0, 0);
      qf[c] = *reinterpret_cast<bf16x8d*>(&v);
    }
  }
  f32x4d oacc[D / 16];
#pragma unroll
  for (int t = 0; t < D / 16; ++t) oacc[t] = f32x4d{0.f, 0.f, 0.f, 0.f};
  float mrun = -INFINITY, lrun = 0.0f;
  const uint16_t* Kb = Kc + (long long)bg * T_max * D;
  const uint16_t* Vb = Vc + (long long)bg * T_max * D;
  // V staging: lane takes keys 4 kq .. 4 kq + 3 and dims 8 dq .. 8 dq + 7
  const int kq = l & 3, dq = l >> 2;
  const bool vthr = dq < D / 8;
  // per-lane byte offsets inside a 16-token group (tile invariant)
  const int koff = ln * D * 2 + lg * 16;
  const int voff = vthr ? (kq * 4 * D * 2 + dq * 16) : 0x40000000;   // idle lanes read past the end
  __syncthreads();                                 // ssel visible

  const int nsteps = (g1 - g0 + 4 * GPS - 1) / (4 * GPS);
  // token of the first key of group gi, or -1 when the group holds no valid key
  auto group_t0 = [&](int gi) {
    const int f = gi * 16;
    const int jj = f / B;
    const int j = __builtin_amdgcn_readfirstlane((int)ssel[jj - jlo]);
    const int t0 = j * B + (f - jj * B);
    return __builtin_amdgcn_readfirstlane((j >= 0 && j <= bc && t0 <= p) ? t0 : -1);
  };
  auto issue = [&](int step, uint4 (&kr)[GPS][D / 32], uint4 (&vr)[GPS][4], int (&t0s)[GPS]) {
#pragma unroll
    for (int x = 0; x < GPS; ++x) {
      const int gi = g0 + (step * 4 + w) * GPS + x;
      const int t0 = (step < nsteps && gi < g1) ? group_t0(gi) : -1;
      t0s[x] = t0;
      // No branch around the loads (the wait counts stay exact): a group
      // without valid keys gets an empty descriptor and reads zeros. The
      // loads are non-temporal (cache policy 2): each selected K/V byte is
      // read once per step, and the streaming hint lifts the read rate.
      const int tb = max(t0, 0);
      const int bytes = (t0 >= 0) ? (p + 1 - t0) * D * 2 : 0;   // keys past p read as zero
      const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
          (void*)(Kb + (long long)tb * D), (short)0, bytes, kDecBufWord3);
      const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
          (void*)(Vb + (long long)tb * D), (short)0, bytes, kDecBufWord3);
#pragma unroll
      for (int c = 0; c < D / 32; ++c) {
        auto a = __builtin_amdgcn_raw_buffer_load_b128(rk, koff + c * 64, 0, 2);
        kr[x][c] = __builtin_bit_cast(uint4, a);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        auto b = __builtin_amdgcn_raw_buffer_load_b128(rv, voff + r * D * 2, 0, 2);
        vr[x][r] = __builtin_bit_cast(uint4, b);
      }
    }
  };
  // one step on the register set (kraw, vraw, tok0)
  auto compute = [&](const uint4 (&kraw)[GPS][D / 32], const uint4 (&vraw)[GPS][4],
                     const int (&tok0)[GPS]) {
    // V^T into this wave's LDS slice
#pragma unroll
    for (int x = 0; x < GPS; ++x) {
      if (vthr && tok0[x] >= 0) {
        uint16_t* vt = vt_slice(w, x);
        const uint32_t a[4] = {vraw[x][0].x, vraw[x][0].y, vraw[x][0].z, vraw[x][0].w};
        const uint32_t b[4] = {vraw[x][1].x, vraw[x][1].y, vraw[x][1].z, vraw[x][1].w};
        const uint32_t c[4] = {vraw[x][2].x, vraw[x][2].y, vraw[x][2].z, vraw[x][2].w};
        const uint32_t d[4] = {vraw[x][3].x, vraw[x][3].y, vraw[x][3].z, vraw[x][3].w};
#pragma unroll
        for (int wd = 0; wd < 4; ++wd) {
          uint2 lo, hi;
          lo.x = (a[wd] & 0xffffu) | (b[wd] << 16);
          lo.y = (c[wd] & 0xffffu) | (d[wd] << 16);
          hi.x = (a[wd] >> 16) | (b[wd] & 0xffff0000u);
          hi.y = (c[wd] >> 16) | (d[wd] & 0xffff0000u);
          *reinterpret_cast<uint2*>(vt + (dq * 8 + 2 * wd) * VTS + kq * 4) = lo;
          *reinterpret_cast<uint2*>(vt + (dq * 8 + 2 * wd + 1) * VTS + kq * 4) = hi;
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int x = 0; x < GPS; ++x) {
      if (tok0[x] < 0) continue;                   // uniform across the wavefront
      f32x4d sacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < D / 32; ++c)
        sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8d, kraw[x][c]),
                                                       qf[c], sacc, 0, 0, 0);
      float sv[4];
      float mx = -INFINITY;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int key = tok0[x] + 4 * lg + v;
        sv[v] = (key <= p) ? sacc[v] * sl2 : -INFINITY;
        mx = fmaxf(mx, sv[v]);
      }
      mx = fmax_xor16(mx);
      mx = fmax_xor32(mx);
      const float mnew = fmaxf(mrun, mx);          // finite: key tok0 <= p is valid
      const float alpha = exp2f(mrun - mnew);
      mrun = mnew;
      float pv[4];
      float ps = 0.0f;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        pv[v] = exp2f(sv[v] - mnew);
        ps += pv[v];
      }
      lrun = lrun * alpha + ps;
      s16x4 pb;
      pb[0] = (short)f32_to_bf16(pv[0]);
      pb[1] = (short)f32_to_bf16(pv[1]);
      pb[2] = (short)f32_to_bf16(pv[2]);
      pb[3] = (short)f32_to_bf16(pv[3]);
      const uint16_t* vt = vt_slice(w, x);
#pragma unroll
      for (int t = 0; t < D / 16; ++t) {
        oacc[t] *= alpha;
        const uint2 va = *reinterpret_cast<const uint2*>(vt + (t * 16 + ln) * VTS + lg * 4);
        oacc[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(*reinterpret_cast<const s16x4*>(&va),
                                                            pb, oacc[t], 0, 0, 0);
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };
  uint4 kA[GPS][D / 32], vA[GPS][4], kB[GPS][D / 32], vB[GPS][4];
  int tA[GPS], tB[GPS];
  issue(0, kA, vA, tA);
  for (int it = 0; it < nsteps; it += 2) {
    issue(it + 1, kB, vB, tB);
    compute(kA, vA, tA);
    if (it + 1 >= nsteps) break;
    issue(it + 2, kA, vA, tA);
    compute(kB, vB, tB);
  }
  __syncthreads();                                 // V^T slices are dead from here
  // per-wave partials: head ln; lane groups hold disjoint keys (sum l) and
  // disjoint output dims
  float lsum = sum_xor16(lrun);
  lsum = sum_xor32(lsum);
  if (lg == 0) {
    sm_m[w][ln] = mrun;
    sm_l[w][ln] = lsum;
  }
#pragma unroll
  for (int t = 0; t < D / 16; ++t)
#pragma unroll
    for (int v = 0; v < 4; ++v) sm_o[w][ln][t * 16 + 4 * lg + v] = oacc[t][v];
  __syncthreads();
  const int nsp = S;
  float* ws_ml = ws;
  float* ws_o = ws + (long long)gridDim.x / S * G * nsp * 2;
  for (int xx = tid; xx < G * D; xx += 256) {
    const int u = xx / D, dim = xx % D;
    float M = -INFINITY;
    for (int k = 0; k < 4; ++k) M = fmaxf(M, sm_m[k][u]);
    float Lsum = 0.0f, Osum = 0.0f;
    if (M != -INFINITY) {
      for (int k = 0; k < 4; ++k) {
        const float sc = exp2f(sm_m[k][u] - M);
        Lsum += sm_l[k][u] * sc;
        Osum += sm_o[k][u][dim] * sc;
      }
    }
    const long long hu = (long long)bi * h_q + g * G + u;
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

// Splits per (sequence, KV head): about SW_DEC_WGS workgroups; 512 fills
// every CU once at the bf16 kernel's occupancy (2 workgroups of 4 waves).
int decode_attn_splits(int batch, int h_kv) {
  const int pairs = batch * h_kv;
  int S = (SW_DEC_WGS + pairs - 1) / pairs;
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

// ---------------------------------------------------------------------------
// fixed scratch for the allocation-free entry point
// ---------------------------------------------------------------------------

// The split-K partials of sw_sparse_attn_decode_noalloc: a fixed device array
// (each GPU the library runs on holds its own copy until the process ends).
// Host code never passes the array's name to a kernel; it passes the device
// address looked up below, once per device.
static __device__ __align__(256) __attribute__((used)) float scratch[SW_NOALLOC_SCRATCH_BYTES / 4];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];        // device address of `scratch`, per device
}  // namespace

hipError_t noalloc_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
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
    if (d == 128)
      hipLaunchKernelGGL(attn_decode_mfma_kernel<128>, grid, dim3(256), 0, st, qq, kk, vv, h_kv, G,
                         T_max, B, pos, idx, cnt, kmax, sl2, S, ws);
    else
      hipLaunchKernelGGL(attn_decode_mfma_kernel<64>, grid, dim3(256), 0, st, qq, kk, vv, h_kv, G,
                         T_max, B, pos, idx, cnt, kmax, sl2, S, ws);
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
