// Block-sparse causal flash attention over the selected key blocks
// (paper Alg. 1 step 8): for each query head and query block, softmax over
// the tokens of the selected blocks that precede each query, renormalised
// over those keys only.
//
// Work item = (query block, KV head g, query-head slice). A 256-thread
// workgroup has 4 wavefronts of 32 query rows each: with B = 128 they are the
// 128 rows of one query head; with B = 64 they are two query heads of the same
// KV group. All waves share the K/V tiles staged in LDS.
//
// Per wavefront and 64-key tile the scores are computed transposed,
// S^T = K Q^T, so that each lane owns one query column: the running max and
// sum stay in the lane plus one exchange with the other half-wave. P then
// feeds the B operand of O^T = V^T P^T directly from the accumulator layout;
// V is staged transposed in LDS so that the A operand is two 8-byte reads.
//   bf16:  v_mfma_f32_32x32x16_bf16, fp32 accumulate, P rounded to bf16.
//   fp32:  v_mfma_f32_32x32x2f32, P kept in fp32.
// Tiles are double-buffered in LDS; the next tile's global loads are issued
// before the current tile's math. Work items run longest-first (query blocks
// in descending order, the selection budget grows with the block index) and
// the workgroups of one (query block, KV head) are placed on one XCD so they
// share the K/V blocks through that XCD's L2.
#include "sw_common.h"
#include "sw_internal.h"

namespace sw {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int KT = 64;                 // keys per LDS tile
constexpr float kLog2e = 1.4426950408889634f;

// ---------------------------------------------------------------------------
// work mapping
// ---------------------------------------------------------------------------

// Number of block rows with local index >= x over all sequences.
__device__ __forceinline__ int rows_at_or_after(const SeqMeta& m, int x) {
  int c = 0;
  for (int s = 0; s < m.n_seqs; ++s) c += max(0, (m.blk_start[s + 1] - m.blk_start[s]) - x);
  return c;
}

// rho-th block row in longest-first order (local index descending, then
// sequence ascending). Returns the global row and the local index.
__device__ __forceinline__ void lpt_row(const SeqMeta& m, int rho, int* row, int* s_out,
                                        int* i_out) {
  int lo = 0, hi = m.max_b - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (rows_at_or_after(m, mid) > rho) lo = mid; else hi = mid - 1;
  }
  const int i = lo;
  int k = rho - rows_at_or_after(m, i + 1);
  int s = 0;
  for (; s < m.n_seqs; ++s) {
    if (m.blk_start[s + 1] - m.blk_start[s] > i) {
      if (k == 0) break;
      --k;
    }
  }
  *row = m.blk_start[s] + i;
  *s_out = s;
  *i_out = i;
}

// ---------------------------------------------------------------------------
// bf16 kernel
// ---------------------------------------------------------------------------

template <int D>
struct BfLds {
  static constexpr int KS = D + 8;     // K row stride (elements): 16-byte pad
  static constexpr int VS = KT + 8;    // V^T row stride (elements): 16-byte pad
  static constexpr int K_ELEMS = KT * KS;
  static constexpr int V_ELEMS = D * VS;
  static constexpr int STAGE = K_ELEMS + V_ELEMS;
};

// Raw buffer descriptor word 3 for gfx9-family untyped loads (32-bit data format).
constexpr int kBufWord3 = 0x00020000;

template <int D, int BLK>
__global__ __launch_bounds__(256, 2) void attn_prefill_bf16_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, int h_q, int h_kv, long long N, SeqMeta m,
    const int32_t* __restrict__ idx, const int32_t* __restrict__ cnt, int kmax, float sl2,
    uint16_t* __restrict__ O, float* __restrict__ lse, int groups, int sg) {
  using L = BfLds<D>;
  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * L::STAGE];

  // ---- work item ----
  const int x = blockIdx.x;
  const int xcd = x & 7;
  const int slot = x >> 3;
  const int mu = slot % sg;
  const int gamma = (slot / sg) * 8 + xcd;
  if (gamma >= groups) return;
  const int rho = gamma / h_kv;
  const int g = gamma % h_kv;
  int row, s, i;
  lpt_row(m, rho, &row, &s, &i);
  constexpr int B = BLK;
  const int G = h_q / h_kv;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int l = tid & 63;
  const int hl = l >> 5;            // half-wave
  const int ln = l & 31;            // lane within half
  constexpr int hpw = (B == 64) ? 2 : 1;  // query heads per workgroup
  const int u = g * G + mu * hpw + (hpw == 2 ? (w >> 1) : 0);
  const int rw = (hpw == 2) ? (w & 1) : w;   // 32-row slice within the block
  const int seq0 = m.tok_start[s];
  const int seq1 = m.tok_start[s + 1];
  const int q0 = seq0 + i * B + rw * 32;     // first query token of this wave
  const bool active = (u < (g + 1) * G) && (q0 < seq1);

  // ---- Q fragments: lane holds query q0+ln, dims kk*16 + hl*8 .. +7 ----
  bf16x8 qf[D / 16];
  {
    const int qp = q0 + ln;
    const bool ok = active && qp < seq1;
    const uint16_t* qrow = Q + ((long long)u * N + (ok ? qp : 0)) * D;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      uint4 v = ok ? *reinterpret_cast<const uint4*>(qrow + kk * 16 + hl * 8) : make_uint4(0, 0, 0, 0);
      qf[kk] = *reinterpret_cast<bf16x8*>(&v);
    }
  }

  // ---- selected block list ----
  const int nsel = min(cnt[row], kmax);
  const int32_t* sel = idx + (long long)row * kmax;
  constexpr int tpb = B / KT;              // key tiles per block
  const int ntiles = nsel * tpb;

  // global -> register staging for one tile
  constexpr int KCH = D / 8;               // 16-byte chunks per key row
  constexpr int KPASS = (KT * KCH) / 256;  // K loads per thread
  uint4 kreg[KPASS];
  uint4 vreg[4];
  const int vkg = tid & 15;                // V: keys vkg*4 .. +3
  const int vdg = tid >> 4;                // V: dims vdg*8 .. +7
  const bool vthr = vdg < D / 8;

  auto tile_key0 = [&](int t, int* k0, bool* valid) {
    const int jj = t / tpb;
    const int kt = t % tpb;
    const int j = sel[jj];
    *valid = (j >= 0 && j <= i);
    *k0 = seq0 + (*valid ? j : 0) * B + kt * KT;
  };
  // One uniform branch per tile. The loads are raw buffer loads through a
  // descriptor based at the tile's first key and sized to the end of the
  // sequence, so keys past the end read as zero without any per-lane test
  // (they are masked in the softmax); per-lane offsets are tile invariant.
  const uint16_t* Kg = K + (long long)g * N * D;
  const uint16_t* Vg = V + (long long)g * N * D;
  int koff[KPASS];
#pragma unroll
  for (int p = 0; p < KPASS; ++p) {
    const int e = tid + p * 256;
    koff[p] = (e / KCH) * D * 2 + (e % KCH) * 16;
  }
  const int voff = (vkg * 4 * D + vdg * 8) * 2;
  auto load_tile = [&](int t) {
    int k0;
    bool valid;
    tile_key0(t, &k0, &valid);
    if (valid) {
      const int bytes = max(0, (seq1 - k0) * D * 2);   // 0: every load returns zero
      const __amdgpu_buffer_rsrc_t rk =
          __builtin_amdgcn_make_buffer_rsrc((void*)(Kg + (long long)k0 * D), (short)0, bytes, kBufWord3);
      const __amdgpu_buffer_rsrc_t rv =
          __builtin_amdgcn_make_buffer_rsrc((void*)(Vg + (long long)k0 * D), (short)0, bytes, kBufWord3);
#pragma unroll
      for (int p = 0; p < KPASS; ++p) {
        auto v = __builtin_amdgcn_raw_buffer_load_b128(rk, koff[p], 0, 0);
        kreg[p] = *reinterpret_cast<uint4*>(&v);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        auto v = __builtin_amdgcn_raw_buffer_load_b128(rv, voff + r * D * 2, 0, 0);
        vreg[r] = vthr ? *reinterpret_cast<uint4*>(&v) : make_uint4(0, 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int p = 0; p < KPASS; ++p) kreg[p] = make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int r = 0; r < 4; ++r) vreg[r] = make_uint4(0, 0, 0, 0);
    }
  };
  auto store_tile = [&](int buf) {
    uint16_t* ks = lds + buf * L::STAGE;
    uint16_t* vt = ks + L::K_ELEMS;
#pragma unroll
    for (int p = 0; p < KPASS; ++p) {
      const int e = tid + p * 256;
      const int key = e / KCH, ch = e % KCH;
      *reinterpret_cast<uint4*>(ks + key * L::KS + ch * 8) = kreg[p];
    }
    if (vthr) {
      const uint32_t a[4] = {vreg[0].x, vreg[0].y, vreg[0].z, vreg[0].w};
      const uint32_t b[4] = {vreg[1].x, vreg[1].y, vreg[1].z, vreg[1].w};
      const uint32_t c[4] = {vreg[2].x, vreg[2].y, vreg[2].z, vreg[2].w};
      const uint32_t d[4] = {vreg[3].x, vreg[3].y, vreg[3].z, vreg[3].w};
      // keys vkg*4 .. +3 go to position perm(vkg*4): bits 2 and 3 of the key
      // swapped, so that the 8 keys one lane feeds to the P.V MFMA
      // (c*16 + hl*4 + {0..3} and c*16 + 8 + hl*4 + {0..3}) are contiguous
      const int kb = vkg * 4;
      const int kpos = (kb & ~12) | ((kb & 4) << 1) | ((kb & 8) >> 1);
#pragma unroll
      for (int wd = 0; wd < 4; ++wd) {
        uint2 lo, hi;
        lo.x = (a[wd] & 0xffffu) | (b[wd] << 16);
        lo.y = (c[wd] & 0xffffu) | (d[wd] << 16);
        hi.x = (a[wd] >> 16) | (b[wd] & 0xffff0000u);
        hi.y = (c[wd] >> 16) | (d[wd] & 0xffff0000u);
        *reinterpret_cast<uint2*>(vt + (vdg * 8 + 2 * wd) * L::VS + kpos) = lo;
        *reinterpret_cast<uint2*>(vt + (vdg * 8 + 2 * wd + 1) * L::VS + kpos) = hi;
      }
    }
  };

  // ---- running state ----
  f32x16 oacc[D / 32];
#pragma unroll
  for (int t = 0; t < D / 32; ++t)
#pragma unroll
    for (int j = 0; j < 16; ++j) oacc[t][j] = 0.0f;
  float mrun = -INFINITY;
  float lrun = 0.0f;
  const int qpos = q0 + ln;

  if (ntiles > 0) {
    load_tile(0);
    store_tile(0);
  }
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    if (t + 1 < ntiles) load_tile(t + 1);
    int k0;
    bool valid;
    tile_key0(t, &k0, &valid);
    if (active && valid && k0 <= q0 + 31 && k0 < seq1) {
      const uint16_t* ks = lds + (t & 1) * L::STAGE;
      const uint16_t* vt = ks + L::K_ELEMS;
      f32x16 sacc[2];
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
#pragma unroll
        for (int j = 0; j < 16; ++j) sacc[h2][j] = 0.0f;
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) {
          const bf16x8 a =
              *reinterpret_cast<const bf16x8*>(ks + (h2 * 32 + ln) * L::KS + kk * 16 + hl * 8);
          sacc[h2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], sacc[h2], 0, 0, 0);
        }
      }
      // running max on the raw scores (the scale is positive), masking
      // only where the tile can reach past the query or the sequence end
      const bool need_mask = (k0 + KT - 1 > q0) || (k0 + KT > seq1);
      float mx = -INFINITY;
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          float v = sacc[h2][j];
          if (need_mask) {
            const int kp = k0 + h2 * 32 + (j >> 2) * 8 + hl * 4 + (j & 3);
            if (kp > qpos || kp >= seq1) v = -INFINITY;
          }
          sacc[h2][j] = v;
          mx = fmaxf(mx, v);
        }
      }
      mx = fmaxf(mx, __shfl_xor(mx, 32)) * sl2;
      const float mnew = fmaxf(mrun, mx);
      const float mref = (mnew == -INFINITY) ? 0.0f : mnew;
      const float alpha = __builtin_amdgcn_exp2f(mrun - mref);
      const bool rescale = __any(mnew != mrun);   // skip the O rescale when no max moved
      mrun = mnew;
      float psum = 0.0f;
      bf16x8 pb[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        float pv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          pv[e] = __builtin_amdgcn_exp2f(fmaf(sacc[c >> 1][(c & 1) * 8 + e], sl2, -mref));
          psum += pv[e];
        }
        uint32_t wds[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) wds[e] = pack_bf16x2(pv[2 * e], pv[2 * e + 1]);
        pb[c] = *reinterpret_cast<bf16x8*>(wds);
      }
      lrun = lrun * alpha + psum;
      if (rescale) {
#pragma unroll
        for (int td = 0; td < D / 32; ++td)
#pragma unroll
          for (int j = 0; j < 16; ++j) oacc[td][j] *= alpha;
      }
#pragma unroll
      for (int td = 0; td < D / 32; ++td) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const bf16x8 av =
              *reinterpret_cast<const bf16x8*>(vt + (td * 32 + ln) * L::VS + c * 16 + hl * 8);
          oacc[td] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pb[c], oacc[td], 0, 0, 0);
        }
      }
    }
    if (t + 1 < ntiles) store_tile((t + 1) & 1);
    __syncthreads();
  }

  // ---- epilogue ----
  if (!active || qpos >= seq1) return;
  const float ltot = lrun + __shfl_xor(lrun, 32);
  const float inv = ltot > 0.0f ? 1.0f / ltot : 0.0f;
  uint16_t* orow = O + ((long long)u * N + qpos) * D;
#pragma unroll
  for (int td = 0; td < D / 32; ++td) {
#pragma unroll
    for (int jb = 0; jb < 4; ++jb) {
      const int dv = td * 32 + jb * 8 + hl * 4;
      uint2 st;
      st.x = pack_bf16x2(oacc[td][jb * 4 + 0] * inv, oacc[td][jb * 4 + 1] * inv);
      st.y = pack_bf16x2(oacc[td][jb * 4 + 2] * inv, oacc[td][jb * 4 + 3] * inv);
      *reinterpret_cast<uint2*>(orow + dv) = st;
    }
  }
  if (lse && hl == 0)
    lse[(long long)u * N + qpos] = (ltot > 0.0f) ? (mrun + log2f(ltot)) / kLog2e : -INFINITY;
}

// ---------------------------------------------------------------------------
// fp32 kernel
// ---------------------------------------------------------------------------

template <int D>
struct F32Lds {
  static constexpr int KS = D + 4;     // K row stride (floats)
  static constexpr int VS = D + 4;     // V row stride (floats), not transposed
  static constexpr int K_ELEMS = KT * KS;
  static constexpr int STAGE = 2 * K_ELEMS;
};

template <int D>
__global__ __launch_bounds__(256, 1) void attn_prefill_f32_kernel(
    const float* __restrict__ Q, const float* __restrict__ K, const float* __restrict__ V,
    int h_q, int h_kv, long long N, SeqMeta m, const int32_t* __restrict__ idx,
    const int32_t* __restrict__ cnt, int kmax, float sl2, float* __restrict__ O,
    float* __restrict__ lse, int groups, int sg) {
  using L = F32Lds<D>;
  __shared__ __attribute__((aligned(16))) float lds[L::STAGE];
  const int x = blockIdx.x;
  const int xcd = x & 7;
  const int slot = x >> 3;
  const int mu = slot % sg;
  const int gamma = (slot / sg) * 8 + xcd;
  if (gamma >= groups) return;
  const int rho = gamma / h_kv;
  const int g = gamma % h_kv;
  int row, s, i;
  lpt_row(m, rho, &row, &s, &i);
  const int B = m.B;
  const int G = h_q / h_kv;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int l = tid & 63;
  const int hl = l >> 5;
  const int ln = l & 31;
  const int hpw = (B == 64) ? 2 : 1;
  const int u = g * G + mu * hpw + (hpw == 2 ? (w >> 1) : 0);
  const int rw = (hpw == 2) ? (w & 1) : w;
  const int seq0 = m.tok_start[s];
  const int seq1 = m.tok_start[s + 1];
  const int q0 = seq0 + i * B + rw * 32;
  const bool active = (u < (g + 1) * G) && (q0 < seq1);
  const int qpos = q0 + ln;

  float qf[D / 2];
  {
    const bool ok = active && qpos < seq1;
    const float* qrow = Q + ((long long)u * N + (ok ? qpos : 0)) * D;
#pragma unroll
    for (int kk = 0; kk < D / 2; ++kk) qf[kk] = ok ? qrow[kk * 2 + hl] : 0.0f;
  }
  const int nsel = min(cnt[row], kmax);
  const int32_t* sel = idx + (long long)row * kmax;
  const int tpb = B / KT;
  const int ntiles = nsel * tpb;

  f32x16 oacc[D / 32];
#pragma unroll
  for (int t = 0; t < D / 32; ++t)
#pragma unroll
    for (int j = 0; j < 16; ++j) oacc[t][j] = 0.0f;
  float mrun = -INFINITY, lrun = 0.0f;
  float* ks = lds;
  float* vs = lds + L::K_ELEMS;

  for (int t = 0; t < ntiles; ++t) {
    const int jj = t / tpb, kt = t % tpb;
    const int j = sel[jj];
    const bool valid = (j >= 0 && j <= i);
    const int k0 = seq0 + (valid ? j : 0) * B + kt * KT;
    __syncthreads();
    for (int e = tid; e < KT * (D / 4); e += 256) {
      const int key = e / (D / 4), ch = e % (D / 4);
      const int kp = k0 + key;
      float4 kv = make_float4(0.f, 0.f, 0.f, 0.f), vv = kv;
      if (valid && kp < seq1) {
        kv = *reinterpret_cast<const float4*>(K + ((long long)g * N + kp) * D + ch * 4);
        vv = *reinterpret_cast<const float4*>(V + ((long long)g * N + kp) * D + ch * 4);
      }
      *reinterpret_cast<float4*>(ks + key * L::KS + ch * 4) = kv;
      *reinterpret_cast<float4*>(vs + key * L::VS + ch * 4) = vv;
    }
    __syncthreads();
    if (!(active && valid && k0 <= q0 + 31)) continue;
    f32x16 sacc[2];
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
#pragma unroll
      for (int jx = 0; jx < 16; ++jx) sacc[h2][jx] = 0.0f;
#pragma unroll
      for (int kk = 0; kk < D / 2; ++kk)
        sacc[h2] = __builtin_amdgcn_mfma_f32_32x32x2f32(ks[(h2 * 32 + ln) * L::KS + kk * 2 + hl],
                                                        qf[kk], sacc[h2], 0, 0, 0);
    }
    float mx = -INFINITY;
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
      for (int jx = 0; jx < 16; ++jx) {
        float v = sacc[h2][jx] * sl2;
        const int kp = k0 + h2 * 32 + (jx >> 2) * 8 + hl * 4 + (jx & 3);
        if (kp > qpos || kp >= seq1) v = -INFINITY;
        sacc[h2][jx] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mnew = fmaxf(mrun, mx);
    const float mref = (mnew == -INFINITY) ? 0.0f : mnew;
    const float alpha = exp2f(mrun - mref);
    mrun = mnew;
    float psum = 0.0f;
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
      for (int jx = 0; jx < 16; ++jx) {
        const float p = exp2f(sacc[h2][jx] - mref);
        sacc[h2][jx] = p;
        psum += p;
      }
    lrun = lrun * alpha + psum;
#pragma unroll
    for (int td = 0; td < D / 32; ++td) {
#pragma unroll
      for (int jx = 0; jx < 16; ++jx) oacc[td][jx] *= alpha;
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
        for (int jx = 0; jx < 16; ++jx) {
          const int key = h2 * 32 + (jx >> 2) * 8 + hl * 4 + (jx & 3);
          oacc[td] = __builtin_amdgcn_mfma_f32_32x32x2f32(vs[key * L::VS + td * 32 + ln],
                                                          sacc[h2][jx], oacc[td], 0, 0, 0);
        }
    }
  }
  if (!active || qpos >= seq1) return;
  const float ltot = lrun + __shfl_xor(lrun, 32);
  const float inv = ltot > 0.0f ? 1.0f / ltot : 0.0f;
  float* orow = O + ((long long)u * N + qpos) * D;
#pragma unroll
  for (int td = 0; td < D / 32; ++td)
#pragma unroll
    for (int jb = 0; jb < 4; ++jb) {
      const int dv = td * 32 + jb * 8 + hl * 4;
      float4 st = make_float4(oacc[td][jb * 4 + 0] * inv, oacc[td][jb * 4 + 1] * inv,
                              oacc[td][jb * 4 + 2] * inv, oacc[td][jb * 4 + 3] * inv);
      *reinterpret_cast<float4*>(orow + dv) = st;
    }
  if (lse && hl == 0)
    lse[(long long)u * N + qpos] = (ltot > 0.0f) ? (mrun + log2f(ltot)) / kLog2e : -INFINITY;
}

hipError_t launch_attn_prefill(int dtype, const void* Q, const void* K, const void* V, int h_q,
                               int h_kv, int d, long long N, const SeqMeta& meta, int64_t nb,
                               const int32_t* idx, const int32_t* cnt, int kmax, float scale,
                               void* O, float* lse, hipStream_t st) {
  const int G = h_q / h_kv;
  const int hpw = (meta.B == 64) ? 2 : 1;
  const int sg = (G + hpw - 1) / hpw;
  const int groups = (int)(nb * h_kv);
  const unsigned grid = (unsigned)(((groups + 7) / 8) * 8 * sg);
  const float sl2 = scale * kLog2e;
  if (dtype == SW_BF16) {
    auto q = reinterpret_cast<const uint16_t*>(Q);
    auto k = reinterpret_cast<const uint16_t*>(K);
    auto v = reinterpret_cast<const uint16_t*>(V);
    auto o = reinterpret_cast<uint16_t*>(O);
#define SW_LAUNCH_BF16(DD, BB)                                                                  \
  hipLaunchKernelGGL((attn_prefill_bf16_kernel<DD, BB>), dim3(grid), dim3(256), 0, st, q, k, v, h_q, \
                     h_kv, N, meta, idx, cnt, kmax, sl2, o, lse, groups, sg)
    if (d == 128 && meta.B == 128) SW_LAUNCH_BF16(128, 128);
    else if (d == 128) SW_LAUNCH_BF16(128, 64);
    else if (meta.B == 128) SW_LAUNCH_BF16(64, 128);
    else SW_LAUNCH_BF16(64, 64);
#undef SW_LAUNCH_BF16
  } else {
    auto q = reinterpret_cast<const float*>(Q);
    auto k = reinterpret_cast<const float*>(K);
    auto v = reinterpret_cast<const float*>(V);
    auto o = reinterpret_cast<float*>(O);
    if (d == 128)
      hipLaunchKernelGGL(attn_prefill_f32_kernel<128>, dim3(grid), dim3(256), 0, st, q, k, v, h_q,
                         h_kv, N, meta, idx, cnt, kmax, sl2, o, lse, groups, sg);
    else
      hipLaunchKernelGGL(attn_prefill_f32_kernel<64>, dim3(grid), dim3(256), 0, st, q, k, v, h_q,
                         h_kv, N, meta, idx, cnt, kmax, sl2, o, lse, groups, sg);
  }
  return hipGetLastError();
}

}  // namespace sw
