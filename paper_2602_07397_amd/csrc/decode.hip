// Decode path (paper Alg. 2) except the attention: one new token per sequence
// per layer.
//
//  decode_init_kernel     state of one sequence from its prompt's prefill sketch
//  kv_append_kernel       step 1: K_t, V_t into the caches at pos[b]
//  decode_sketch_kernel   steps 2-4 over (sequence, 64-row chunk) workgroups:
//                         every workgroup forms the running means of the open
//                         query/key block and the SRHT of the token query and
//                         of both open representatives (wavefront-level
//                         Walsh-Hadamard transforms); chunk 0 stores them (and
//                         appends K_t, V_t in the one-call step); then each
//                         workgroup writes its rows' entries of (i) the new
//                         score row and (ii) the new last column, 4 lanes per
//                         sketch row
//  walk_strip_kernel      step 5 on the query row only, for the score entries
//                         the step leaves unchanged (rows and columns before
//                         the open block): r_prev W with W = (A/c)^s (or the
//                         clipped power) taken while streaming the fp32 score
//                         cache; one workgroup per (sequence, pair of
//                         32-column strips), the pairs balanced so that every
//                         workgroup reads about as many rows, 32 row groups
//                         reduced in a fixed order (lane exchanges within a
//                         wavefront, then the wavefronts); the rows above a
//                         strip, which hold only its decode-filled columns,
//                         are shared by every thread of the workgroup
//  decode_sketch_walk_kernel  the one-call step's launch of both: the walk
//                         workgroups and the sketch workgroups of a layer
//                         side by side (they touch disjoint state)
//  walk_row_norm_kernel   adds the open block's row and column terms to the
//                         walk row and divides it by its largest magnitude
//                         (the one-call step does this in
//                         select_decode_norm_kernel before selecting, step 6)
#include "select_row.h"
#include "sw_common.h"
#include "sw_internal.h"

namespace sw {

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
  float* As = reinterpret_cast<float*>(state + L.a) + (long long)seq * b_max * L.lda;
  for (int j = threadIdx.x; j < L.lda; j += 256)
    As[cache_at(b_max, m, j)] = (m < b && j < b) ? (float)A[(long long)m * b + j] : 0.0f;
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
    double* bar = reinterpret_cast<double*>(state + L.bar) + (long long)seq * 4 * d;
    for (int t = threadIdx.x; t < d; t += 256) {
#pragma unroll
      for (int c = 0; c < 2; ++c) {      // both position-parity copies
        bar[(2 * c) * d + t] = Qbar[(long long)(b - 1) * d + t];
        bar[(2 * c + 1) * d + t] = Kbar[(long long)(b - 1) * d + t];
      }
    }
    if (threadIdx.x == 0) {
      reinterpret_cast<double*>(state + L.scale)[seq] = A_scale[0];
      reinterpret_cast<int32_t*>(state + L.col0)[seq] = n / B;
      int32_t* cnt = reinterpret_cast<int32_t*>(state + L.cnt) + seq * 4;
      cnt[0] = cnt[1] = cnt[2] = cnt[3] = last;
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
// incremental sketch and score updates
// ---------------------------------------------------------------------------

template <typename T>
__device__ __forceinline__ float load_f32(const T* p, long long i) {
  if constexpr (sizeof(T) == 2) {
    return bf16_to_f32(reinterpret_cast<const uint16_t*>(p)[i]);
  } else {
    return p[i];
  }
}

constexpr int kScoreChunk = 64;

// Steps 2-4 of the token at pos[b] (one workgroup per (sequence, chunk of 64
// score rows); every workgroup of a sequence forms the same representatives):
//   - head sums of the new query and key (thread (group, 16-byte chunk)
//     adds the heads u = group, group + P, ...; the P groups are then added
//     per dimension in a fixed order);
//   - running means of the open query/key block from the previous step's copy
//     (restarted when pos % B == 0); chunk 0 stores the new copy;
//   - SRHT of the token query and of both open representatives (three
//     wavefronts, one transform each); chunk 0 stores them;
//   - rows j of the chunk: (i) A[b_cur][j] = q~_t . Ks[j] / sqrt(r) for
//     j < b_cur, (ii) A[j][b_cur] = Qs[j] . Ks[b_cur] / sqrt(r) for j <= b_cur,
//     four threads per row (coordinates k = 4 i + lane % 4, then two lane
//     exchanges).
// APPEND (the one-call step): chunk 0 also writes k_new and v_new into the
// caches Kc, Vc [batch][h_kv][T_max][d] at pos (Alg. 2 step 1).
// LDS of one sketch workgroup (doubles): per head group partial sums of the
// token's query and key, then six vectors of 256.
template <typename T>
constexpr int sketch_lds_doubles() {
  return 2 * 256 * (16 / (int)sizeof(T)) + 6 * 256;
}

template <typename T, bool APPEND>
__device__ __forceinline__ void decode_sketch_body(const T* __restrict__ q_new,
                                                   const T* __restrict__ k_new, int h_q, int h_kv,
                                                   int d, int B, const int32_t* __restrict__ pos,
                                                   const int8_t* __restrict__ signs,
                                                   const int32_t* __restrict__ cols, int r,
                                                   int batch, int b_max, char* __restrict__ state,
                                                   const T* __restrict__ v_new, T* __restrict__ Kc,
                                                   T* __restrict__ Vc, int T_max, int bi, int chunk,
                                                   double* lds) {
  constexpr int V = 16 / (int)sizeof(T);             // elements per 16-byte load
  double* pq = lds;
  double* pk = pq + 256 * V;
  double* xq = pk + 256 * V;
  double* xb = xq + 256;
  double* xk = xb + 256;
  double* sqt = xk + 256;
  double* sqb = sqt + 256;
  double* skb = sqb + 256;
  const DecodeLayout L = decode_layout(batch, d, r, b_max);
  const int t = threadIdx.x;
  // the new token's query/key chunks do not depend on the position: their
  // loads go out first (clamped head indices: no condition; extra ones unused)
  const int dpc = d / V;                           // chunks per head row
  const int P = 256 / dpc;                         // head groups
  const int ch = t % dpc, grp = t / dpc;
  constexpr int kChunks = 4;                       // head chunks loaded up front
  uint4 rq[kChunks], rk[kChunks];
#pragma unroll
  for (int i = 0; i < kChunks; ++i) {
    const int u = min(grp + i * P, h_q - 1), g = min(grp + i * P, h_kv - 1);
    rq[i] = *reinterpret_cast<const uint4*>(q_new + ((long long)bi * h_q + u) * d + ch * V);
    rk[i] = *reinterpret_cast<const uint4*>(k_new + ((long long)bi * h_kv + g) * d + ch * V);
  }
  const int p = pos[bi];
  const int bc = p / B;                  // open key block == query block
  if constexpr (APPEND) {
    if (chunk == 0 && p >= 0 && p < T_max) {
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
  const int r0 = chunk * kScoreChunk;
  if (r0 > bc) return;
  const bool store = chunk == 0;
  double* Qs = reinterpret_cast<double*>(state + L.qs) + (long long)bi * b_max * r;
  double* Ks = reinterpret_cast<double*>(state + L.ks) + (long long)bi * b_max * r;
  const int rd = (p + 1) & 1, wr = p & 1;          // previous / new copy of the open means
  const int32_t* cnt_rd = reinterpret_cast<const int32_t*>(state + L.cnt) + (bi * 2 + rd) * 2;
  int32_t* cnt_wr = reinterpret_cast<int32_t*>(state + L.cnt) + (bi * 2 + wr) * 2;
  const double* bar_rd = reinterpret_cast<const double*>(state + L.bar) + (long long)(bi * 2 + rd) * 2 * d;
  double* bar_wr = reinterpret_cast<double*>(state + L.bar) + (long long)(bi * 2 + wr) * 2 * d;

  // Then, in the order the values are needed (vector loads complete in
  // order): the previous open means and counts, the transform's signs and
  // columns, and last this thread's score row j of the earlier blocks'
  // sketches (coordinates k = 4 i + q4), which stay in flight while the
  // representatives are formed.
  const int td = min(t, d - 1), tr = min(t, r - 1);   // clamped: no load behind a branch
  const double bq_old = bar_rd[td], bk_old = bar_rd[d + td];
  const int8_t sgn = signs[td];
  const int colv = cols[tr] & (d - 1);
  const int qc = cnt_rd[0], kc = cnt_rd[1];
  const int q4 = t & 3;
  const int j = r0 + (t >> 2);
  constexpr int kPre = 16;
  double pre_q[kPre], pre_k[kPre];
#pragma unroll
  for (int i = 0; i < kPre; ++i) {
    const int k = q4 + 4 * i;
    // clamped (the load carries no condition); rows j >= b_cur are not used
    const int jj = min(j, max(bc - 1, 0)), kk = min(k, r - 1);
    pre_q[i] = Qs[(long long)jj * r + kk];
    pre_k[i] = Ks[(long long)jj * r + kk];
  }

  double sq[V], sk[V];
#pragma unroll
  for (int e = 0; e < V; ++e) sq[e] = sk[e] = 0.0;
  auto add_raw = [&](const uint4& raw, double (&acc)[V]) {
    const T* v = reinterpret_cast<const T*>(&raw);
#pragma unroll
    for (int e = 0; e < V; ++e) acc[e] += (double)load_f32(v, e);
  };
#pragma unroll
  for (int i = 0; i < kChunks; ++i) {
    if (grp + i * P < h_q) add_raw(rq[i], sq);
    if (grp + i * P < h_kv) add_raw(rk[i], sk);
  }
  for (int u = grp + kChunks * P; u < h_q; u += P)
    add_raw(*reinterpret_cast<const uint4*>(q_new + ((long long)bi * h_q + u) * d + ch * V), sq);
  for (int g = grp + kChunks * P; g < h_kv; g += P)
    add_raw(*reinterpret_cast<const uint4*>(k_new + ((long long)bi * h_kv + g) * d + ch * V), sk);
#pragma unroll
  for (int e = 0; e < V; ++e) {
    pq[grp * d + ch * V + e] = sq[e];
    pk[grp * d + ch * V + e] = sk[e];
  }
  const bool fresh = (p % B) == 0;
  __syncthreads();
  if (t < d) {
    double qa = 0.0, ka = 0.0;
    for (int x = 0; x < P; ++x) {
      qa += pq[x * d + t];
      ka += pk[x * d + t];
    }
    qa /= (double)h_q;
    ka /= (double)h_kv;
    const double qbn = fresh ? qa : ((double)qc * bq_old + qa) / (double)(qc + 1);
    const double kbn = fresh ? ka : ((double)kc * bk_old + ka) / (double)(kc + 1);
    if (store) {
      bar_wr[t] = qbn;
      bar_wr[d + t] = kbn;
    }
    const double sg = (double)sgn;
    xq[t] = qa * sg;
    xb[t] = qbn * sg;
    xk[t] = kbn * sg;
  }
  if (store && t == 0) {
    cnt_wr[0] = fresh ? 1 : qc + 1;
    cnt_wr[1] = fresh ? 1 : kc + 1;
  }
  __syncthreads();
  const int wave = t >> 6;
  if (wave == 0) wave_fwht(xq, d);
  else if (wave == 1) wave_fwht(xb, d);
  else if (wave == 2) wave_fwht(xk, d);
  __syncthreads();
  const double rs = 1.0 / sqrt((double)r);
  if (t < r) {
    sqt[t] = xq[colv] * rs;
    sqb[t] = xb[colv] * rs;
    skb[t] = xk[colv] * rs;
    if (store) {
      reinterpret_cast<double*>(state + L.qt)[(long long)bi * r + t] = sqt[t];
      Qs[(long long)bc * r + t] = sqb[t];
      Ks[(long long)bc * r + t] = skb[t];
    }
  }
  __syncthreads();
  // Qs[b_cur] and Ks[b_cur] are taken from LDS: chunk 0 may be storing them
  double accr = 0.0, accc = 0.0;
  if (j < bc) {
#pragma unroll
    for (int i = 0; i < kPre; ++i) {
      const int k = q4 + 4 * i;
      if (k < r) {
        accc += pre_q[i] * skb[k];
        accr += sqt[k] * pre_k[i];
      }
    }
    const double* qsj = Qs + (long long)j * r;
    const double* ksj = Ks + (long long)j * r;
    for (int k = q4 + 4 * kPre; k < r; k += 4) {
      accc += qsj[k] * skb[k];
      accr += sqt[k] * ksj[k];
    }
  } else if (j == bc) {
#pragma unroll 16
    for (int k = q4; k < r; k += 4) accc += sqb[k] * skb[k];
  }
  accr += __shfl_xor(accr, 1);
  accc += __shfl_xor(accc, 1);
  accr += __shfl_xor(accr, 2);
  accc += __shfl_xor(accc, 2);
  float* A = reinterpret_cast<float*>(state + L.a) + (long long)bi * b_max * L.lda;
  float* rowc = reinterpret_cast<float*>(state + L.rowc) + (long long)bi * b_max;
  float* colc = reinterpret_cast<float*>(state + L.colc) + (long long)bi * b_max;
  if (q4 == 0 && j <= bc) {
    const float vr = (float)(accr * rs), vc = (float)(accc * rs);
    if (j < bc) A[cache_at(b_max, bc, j)] = vr;
    A[cache_at(b_max, j, bc)] = vc;
    rowc[j] = j < bc ? vr : vc;          // the diagonal entry comes from the column
    colc[j] = vc;
  }
}

template <typename T, bool APPEND>
__global__ __launch_bounds__(256) void decode_sketch_kernel(const T* __restrict__ q_new,
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
  __shared__ double lds[sketch_lds_doubles<T>()];
  decode_sketch_body<T, APPEND>(q_new, k_new, h_q, h_kv, d, B, pos, signs, cols, r, batch, b_max,
                                state, v_new, Kc, Vc, T_max, blockIdx.x, blockIdx.y, lds);
}

// ---------------------------------------------------------------------------
// walk row
// ---------------------------------------------------------------------------

constexpr int kStripCols = 32;           // columns per strip: one 128-byte piece of a row
constexpr int kStripQuads = kStripCols / 4;
constexpr int kStripGroups = 32;         // row groups per workgroup, 8 per wavefront
constexpr int kStripThreads = kStripQuads * kStripGroups;
#ifndef SW_STRIP_ROWS
#define SW_STRIP_ROWS 4                  // rows each thread loads before adding
#endif
constexpr int kStripBufWord3 = 0x00020000;   // raw buffer descriptor word 3 (gfx9 family)

template <bool S8, bool RELU>
__device__ __forceinline__ double walk_weight(float a, double inv_c, int s_exp) {
  double x = (double)a * inv_c;
  if constexpr (RELU) x = fmax(x, 0.0);
  if constexpr (S8) {
    const double x2 = x * x, x4 = x2 * x2;
    return x4 * x4;
  } else {
    return pow_int_d(x, s_exp);
  }
}

__device__ __forceinline__ uint4 load_quad(__amdgpu_buffer_rsrc_t ra, int off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(ra, off, 0, 0));
}

// The walk row splits into the part the step's sketch does not change and the
// open block's row and column, which it rewrites (Alg. 2 step 4):
//   r[j] = sum_{m != b_cur} r_prev[m] W[m][j]                 (j < b_cur)
//          + r_prev[b_cur] W[b_cur][j]
//   r[b_cur] = sum_{m <= b_cur} r_prev[m] W[m][b_cur]
// walk_old_body computes the first sum from the score cache as the previous
// steps left it (it reads no entry of row or column b_cur, so it may run
// while the sketch of the same step writes them); walk_finish adds the rest.
//
// walk_old_body: one workgroup per (sequence, strip pair): strips k and
// S-1-k of 32 columns (S = lda / 32; the cache stores a strip's rows
// contiguously, 128 bytes each, so a strip is read as one contiguous range).
// Strip x's rows m = 32 x .. b_cur - 1 hold its causal entries, so a pair
// holds about b_cur rows in all. Its row groups are shared between the two
// strips in proportion to their row counts; thread (row group g, column quad
// q) takes every n-th row of its strip (n = the strip's group count) with
// 16-byte loads of 4 columns. The columns decode filled before the open
// block (col0 .. b_cur - 1) are non-zero in the rows above the strip as well
// (m < 32 x): those rows hold nothing else in the strip, so every thread of
// the workgroup takes a share of them, for those columns only.
// r_out[j] = (sum over the strip's rows: per group ascending, then over the
// 8 groups of a wavefront by a butterfly of lane exchanges, then over the
// four wavefronts in order) + (sum over the rows above: per thread
// ascending, then a butterfly over the 64 lanes, then the four wavefronts in
// order) of r_prev[m] W[m][j] for j < b_cur. Entries the cache
// holds as zero (above the diagonal outside the decode-filled columns) give
// zero terms; quads that are wholly zero are not loaded.
// LDS of one walk workgroup (doubles): the staged previous walk row, then
// per wavefront and strip the strip-row sums and the rows-above sums of the
// 32 columns.
constexpr int kWalkSmem = SW_MAX_BLOCKS;
constexpr int kWalkLdsDoubles = kWalkSmem + 2 * (kStripThreads / 64) * 2 * kStripCols;
static_assert(kStripThreads == 256 && kStripQuads == 8, "8 row groups x 8 quads per wavefront");

template <bool S8, bool RELU>
__device__ __forceinline__ void walk_old_body(const char* __restrict__ state, int batch, int d,
                                              int r, int b_max, int B,
                                              const int32_t* __restrict__ pos, int s_exp,
                                              const double* __restrict__ r_prev,
                                              double* __restrict__ r_out, int bi, int k,
                                              double* lds) {
  double* smem = lds;
  // wsum[w][strip][c]: wavefront w's strip-row sums; xw[w][strip][c]: its
  // rows-above sums (zero outside the decode-filled quads)
  double (*wsum)[2][kStripCols] = reinterpret_cast<double (*)[2][kStripCols]>(smem + kWalkSmem);
  double (*xw)[2][kStripCols] = wsum + kStripThreads / 64;
  const DecodeLayout L = decode_layout(batch, d, r, b_max);
  const int lda = L.lda;
  const int t = threadIdx.x;
  // the loads that do not need the position go out with it: the scale, the
  // first decode-filled column and the whole previous walk row (clamped
  // indices, no condition), which is then staged in LDS
  const int p = pos[bi];
  const double c0 = reinterpret_cast<const double*>(state + L.scale)[bi];
  const int col0 = reinterpret_cast<const int32_t*>(state + L.col0)[bi];
  constexpr int kStage = (SW_MAX_BLOCKS + kStripThreads - 1) / kStripThreads;
  {
    double rs[kStage];
#pragma unroll
    for (int i = 0; i < kStage; ++i)
      rs[i] = r_prev[(long long)bi * b_max + min(t + i * kStripThreads, b_max - 1)];
#pragma unroll
    for (int i = 0; i < kStage; ++i)
      if (t + i * kStripThreads < b_max) smem[t + i * kStripThreads] = rs[i];
  }
  const int bc = p / B;
  if (p < 0 || bc >= b_max) return;
  const int S = lda / kStripCols;
  const int sa = k, sb = S - 1 - k;                 // sb == sa: a single strip
  const double inv_c = 1.0 / (c0 > 0.0 ? c0 : 1.0);
  const float* A = reinterpret_cast<const float*>(state + L.a) + (long long)bi * b_max * lda;
  const int q = t % kStripQuads, g = t / kStripQuads;
  const int na = (sa * kStripCols < bc) ? bc - sa * kStripCols : 0;
  const int nbr = (sb != sa && sb * kStripCols < bc) ? bc - sb * kStripCols : 0;
  const int total = na + nbr;
  // row groups of strip a: about kStripGroups * na / total (each strip with
  // rows gets at least one)
  int ga = (nbr == 0) ? kStripGroups : (na == 0 ? 0 : (kStripGroups * na + total / 2) / total);
  if (na > 0 && nbr > 0) ga = min(max(ga, 1), kStripGroups - 1);
  const bool in_a = g < ga;
  const int x = in_a ? sa : sb;
  const int gi = in_a ? g : g - ga;                 // group index within the strip
  const int ng = in_a ? ga : kStripGroups - ga;     // groups of the strip
  const int m0 = x * kStripCols;
  const int nrows = in_a ? na : nbr;
  const int j = x * kStripCols + 4 * q;             // this thread's 4 columns
  const bool okj = j < bc;                          // the quad holds an old column
  const int ebc = bc - j;                           // element of column b_cur (if 0..3)
  // the sequence's score cache as a buffer: 32-bit offsets, and a load whose
  // quad holds nothing is sent past the end (it reads zeros)
  const int bytes = b_max * lda * 4;
  const __amdgpu_buffer_rsrc_t ra =
      __builtin_amdgcn_make_buffer_rsrc((void*)A, (short)0, bytes, kStripBufWord3);
  // The decode-filled columns before b_cur of strip sb over the rows above
  // it (rows < 32 sb): the loads of the first such quad over the first 2048
  // rows go out before the strip's own rows, so their latency is hidden.
  const int xjb = sb * kStripCols;
  const int jlo_b = max(col0, xjb), jhi_b = min(bc - 1, xjb + kStripCols - 1);
  const bool pre_b = sb != sa && xjb > 0 && jlo_b <= jhi_b;
  const int jd_b = xjb + 4 * ((jlo_b - xjb) / 4);
  uint4 pa[8];
#pragma unroll
  for (int v = 0; v < 8; ++v) {
    const int m = t + v * kStripThreads;
    pa[v] = load_quad(ra, (pre_b && m < xjb) ? cache_at(b_max, m, jd_b) * 4 : bytes);
  }
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  __syncthreads();                       // the staged row is visible
  const double* rp = smem;
  {
    constexpr int NR = S8 ? SW_STRIP_ROWS : SW_STRIP_ROWS / 2;   // the general power needs more registers
    for (int i0 = gi; i0 < nrows; i0 += NR * ng) {
      // every load of the pass is issued before any is used
      uint4 a[NR];
#pragma unroll
      for (int v = 0; v < NR; ++v) {
        const int i = i0 + v * ng;
        const bool ok = i < nrows && okj;
        a[v] = load_quad(ra, ok ? cache_at(b_max, m0 + i, j) * 4 : bytes);
      }
#pragma unroll
      for (int v = 0; v < NR; ++v) {
        const double rv = rp[m0 + min(i0 + v * ng, nrows - 1)];
        const float av[4] = {__uint_as_float(a[v].x), __uint_as_float(a[v].y),
                             __uint_as_float(a[v].z), __uint_as_float(a[v].w)};
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (e != ebc) acc[e] += rv * walk_weight<S8, RELU>(av[e], inv_c, s_exp);
      }
    }
  }
  // Both sums are reduced in a fixed order behind one barrier: per wavefront
  // by lane exchanges (a butterfly), then over the four wavefronts in order.
  const int wv = t >> 6, lane = t & 63;
  xw[wv][lane >> 5][lane & 31] = 0.0;
  // the decode-filled columns before b_cur of each strip over the rows above
  // it (rows 0 .. 32 x - 1), one quad at a time, every thread a share of rows
#pragma unroll 1
  for (int which = 0; which < 2; ++which) {
    const int xs = which ? sb : sa;
    if (which == 1 && sb == sa) break;
    const int xj0 = xs * kStripCols;
    const int jlo = max(col0, xj0), jhi = min(bc - 1, xj0 + kStripCols - 1);
    if (xj0 == 0 || jlo > jhi) continue;
#pragma unroll 1
    for (int qd = (jlo - xj0) / 4; qd <= (jhi - xj0) / 4; ++qd) {
      const int jd = xj0 + 4 * qd;
      double xa[4] = {0.0, 0.0, 0.0, 0.0};
      for (int m1 = t; m1 < xj0; m1 += 8 * kStripThreads) {
        uint4 a[8];
        if (which == 1 && jd == jd_b && m1 == t) {   // loaded before the strip's rows
#pragma unroll
          for (int v = 0; v < 8; ++v) a[v] = pa[v];
        } else {
#pragma unroll
          for (int v = 0; v < 8; ++v) {
            const int m = m1 + v * kStripThreads;
            a[v] = load_quad(ra, m < xj0 ? cache_at(b_max, m, jd) * 4 : bytes);
          }
        }
#pragma unroll
        for (int v = 0; v < 8; ++v) {
          const double rv = rp[min(m1 + v * kStripThreads, xj0 - 1)];
          const float av[4] = {__uint_as_float(a[v].x), __uint_as_float(a[v].y),
                               __uint_as_float(a[v].z), __uint_as_float(a[v].w)};
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (jd + e != bc) xa[e] += rv * walk_weight<S8, RELU>(av[e], inv_c, s_exp);
        }
      }
      for (int off = 1; off < 64; off <<= 1)
#pragma unroll
        for (int e = 0; e < 4; ++e) xa[e] += __shfl_xor(xa[e], off);
      if (lane == 0)
#pragma unroll
        for (int e = 0; e < 4; ++e) xw[wv][which][4 * qd + e] = xa[e];
    }
  }
  // the strip rows: the 8 row groups of a wavefront (lanes q, q + 8, ...,
  // q + 56 hold column quad q), per strip
  {
    double s0[4], s1[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      s0[e] = in_a ? acc[e] : 0.0;
      s1[e] = in_a ? 0.0 : acc[e];
    }
    for (int off = kStripQuads; off < 64; off <<= 1)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        s0[e] += __shfl_xor(s0[e], off);
        s1[e] += __shfl_xor(s1[e], off);
      }
    if (lane < kStripQuads)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        wsum[wv][0][4 * lane + e] = s0[e];
        wsum[wv][1][4 * lane + e] = s1[e];
      }
  }
  __syncthreads();
  if (t < 2 * kStripCols) {
    const int which = t / kStripCols, c = t % kStripCols;
    if (which == 0 || sb != sa) {
      const int xs = which ? sb : sa;
      double v = ((wsum[0][which][c] + wsum[1][which][c]) + wsum[2][which][c]) + wsum[3][which][c];
      const int jj = xs * kStripCols + c;
      if (jj >= col0 && xs * kStripCols > 0)
        v += ((xw[0][which][c] + xw[1][which][c]) + xw[2][which][c]) + xw[3][which][c];
      if (jj < bc) r_out[(long long)bi * b_max + jj] = v;
    }
  }
}

// Per-layer form: the unchanged part of the walk row into r_out[j], j < b_cur
// (walk_row_norm_kernel completes it).
template <bool S8, bool RELU>
__global__ __launch_bounds__(kStripThreads) void walk_strip_kernel(const char* __restrict__ state,
                                                                   int batch, int d, int r,
                                                                   int b_max, int B,
                                                                   const int32_t* __restrict__ pos,
                                                                   int s_exp,
                                                                   const double* __restrict__ r_prev,
                                                                   double* __restrict__ r_out) {
  __shared__ double lds[kWalkLdsDoubles];
  walk_old_body<S8, RELU>(state, batch, d, r, b_max, B, pos, s_exp, r_prev, r_out, blockIdx.x,
                          blockIdx.y, lds);
}

// The one-call step: the workgroups with blockIdx.y < pairs compute the
// unchanged part of this layer's walk row (none at the first walked layer),
// the others run the incremental sketch (with the KV append). The two read
// and write disjoint parts of the state, so they run side by side.
template <typename T, bool S8, bool RELU>
__global__ __launch_bounds__(256) void decode_sketch_walk_kernel(
    const T* __restrict__ q_new, const T* __restrict__ k_new, int h_q, int h_kv, int d, int B,
    const int32_t* __restrict__ pos, const int8_t* __restrict__ signs,
    const int32_t* __restrict__ cols, int r, int batch, int b_max, char* __restrict__ state,
    const T* __restrict__ v_new, T* __restrict__ Kc, T* __restrict__ Vc, int T_max, int pairs,
    int s_exp, const double* __restrict__ r_prev, double* __restrict__ rows) {
  static_assert(kStripThreads == 256, "both roles run 256 threads");
  constexpr int kLds = sketch_lds_doubles<T>() > kWalkLdsDoubles ? sketch_lds_doubles<T>()
                                                                 : kWalkLdsDoubles;
  __shared__ double lds[kLds];
  if ((int)blockIdx.y < pairs)
    walk_old_body<S8, RELU>(state, batch, d, r, b_max, B, pos, s_exp, r_prev, rows, blockIdx.x,
                            blockIdx.y, lds);
  else
    decode_sketch_body<T, true>(q_new, k_new, h_q, h_kv, d, B, pos, signs, cols, r, batch, b_max,
                                state, v_new, Kc, Vc, T_max, blockIdx.x, blockIdx.y - pairs, lds);
}

// walk_finish: thread t's values v[e] of the finished (unnormalised) walk row
// for blocks j = t*E + e <= b_cur (E = ceil((b_cur + 1) / 256)), from the
// unchanged part in old[j] (j < b_cur; not read when r_prev is NULL) and the
// open block's row and column of the score cache. At the first walked layer
// (r_prev NULL) the row is W[b_cur][j] itself. The column sum runs per
// thread over m = t, t + 256, ... ascending, then over the lanes of a
// wavefront by exchanges and over the four wavefronts in order.
template <bool S8, bool RELU, int MAXE>
__device__ __forceinline__ void walk_finish(const char* __restrict__ state, int batch, int d, int r,
                                            int b_max, int bi, int bc, int s_exp,
                                            const double* __restrict__ r_prev,
                                            const double* __restrict__ old, double (&v)[MAXE],
                                            double* tmp) {
  const DecodeLayout L = decode_layout(batch, d, r, b_max);
  const int t = threadIdx.x;
  const int avail = bc + 1;
  const int E = (avail + 255) / 256;
  const double c0 = reinterpret_cast<const double*>(state + L.scale)[bi];
  const double inv_c = 1.0 / (c0 > 0.0 ? c0 : 1.0);
  const float* rowc = reinterpret_cast<const float*>(state + L.rowc) + (long long)bi * b_max;
  const float* colc = reinterpret_cast<const float*>(state + L.colc) + (long long)bi * b_max;
  // every load goes out before any value is used (indices clamped into range)
  float wrow[MAXE];
#pragma unroll
  for (int e = 0; e < MAXE; ++e) wrow[e] = rowc[min(t * E + e, bc)];
  if (r_prev == nullptr) {
#pragma unroll
    for (int e = 0; e < MAXE; ++e) v[e] = walk_weight<S8, RELU>(wrow[e], inv_c, s_exp);
    return;
  }
  const double* rp = r_prev + (long long)bi * b_max;
  double ov[MAXE];
#pragma unroll
  for (int e = 0; e < MAXE; ++e) ov[e] = old[min(t * E + e, max(bc - 1, 0))];
  float wcol[MAXE];
  double rcol[MAXE];
#pragma unroll
  for (int e = 0; e < MAXE; ++e) {
    const int m = min(t + 256 * e, bc);
    wcol[e] = colc[m];
    rcol[e] = rp[m];
  }
  const double rb = rp[bc];
  double cs = 0.0;
#pragma unroll
  for (int e = 0; e < MAXE; ++e)
    if (t + 256 * e <= bc) cs += rcol[e] * walk_weight<S8, RELU>(wcol[e], inv_c, s_exp);
  for (int off = 1; off < 64; off <<= 1) cs += __shfl_xor(cs, off);
  if ((t & 63) == 0) tmp[t >> 6] = cs;
  __syncthreads();
  cs = ((tmp[0] + tmp[1]) + tmp[2]) + tmp[3];
  __syncthreads();
#pragma unroll
  for (int e = 0; e < MAXE; ++e) {
    const int j = t * E + e;
    v[e] = (j < bc) ? ov[e] + rb * walk_weight<S8, RELU>(wrow[e], inv_c, s_exp) : cs;
  }
}

// Per-layer form of the walk's completion: r_out[j] (j <= b_cur) finished
// from its unchanged part and divided by its largest magnitude; entries past
// b_cur are zeroed.
template <bool S8, bool RELU, int MAXE>
__global__ __launch_bounds__(256) void walk_row_norm_kernel(const char* __restrict__ state,
                                                            int batch, int d, int r, int b_max,
                                                            int B, const int32_t* __restrict__ pos,
                                                            int s_exp,
                                                            const double* __restrict__ r_prev,
                                                            double* __restrict__ r_out) {
  __shared__ double tmp[4];
  const int bi = blockIdx.x;
  const int p = pos[bi];
  const int bc = p / B;
  if (p < 0 || bc >= b_max) return;
  double* out = r_out + (long long)bi * b_max;
  const int t = threadIdx.x;
  const int avail = bc + 1;
  const int E = (avail + 255) / 256;
  double v[MAXE];
  walk_finish<S8, RELU, MAXE>(state, batch, d, r, b_max, bi, bc, s_exp, r_prev, out, v, tmp);
  double mx = 0.0;
#pragma unroll
  for (int e = 0; e < MAXE; ++e)
    if (e < E && t * E + e < avail) mx = fmax(mx, fabs(v[e]));
  for (int off = 32; off > 0; off >>= 1) mx = fmax(mx, __shfl_xor(mx, off));
  if ((t & 63) == 0) tmp[t >> 6] = mx;
  __syncthreads();
  mx = fmax(fmax(tmp[0], tmp[1]), fmax(tmp[2], tmp[3]));
  const double inv = mx > 0.0 ? 1.0 / mx : 1.0;
#pragma unroll
  for (int e = 0; e < MAXE; ++e) {
    const int j = t * E + e;
    if (e < E && j < avail) out[j] = v[e] * inv;
  }
  for (int j = avail + t; j < b_max; j += 256) out[j] = 0.0;
}

// The one-call step: the walk row of each sequence finished from its
// unchanged part in rows, divided in place by its largest magnitude over
// blocks 0..b_cur (entries past b_cur zeroed), then its selection (Alg. 2
// step 6, forced set {0, b_cur}) from the rescaled values the threads still
// hold in registers.
template <bool S8, bool RELU, int MAXE>
__global__ __launch_bounds__(256) void select_decode_norm_kernel(
    const char* __restrict__ state, int batch, int d, int r, int b_max, int B,
    const int32_t* __restrict__ pos, int s_exp, const double* __restrict__ r_prev,
    double* __restrict__ rows, int k, int pct, uint32_t flags, int32_t* __restrict__ idx,
    int32_t* __restrict__ cnt, int kmax) {
  __shared__ double tmp[4];
  const int bi = blockIdx.x;
  const int p = pos[bi];
  const int bc = p / B;
  if (p < 0 || bc >= b_max) return;
  double* row = rows + (long long)bi * b_max;
  const int avail = bc + 1;
  const int E = (avail + 255) / 256;
  const int t = threadIdx.x;
  double v[MAXE];
  walk_finish<S8, RELU, MAXE>(state, batch, d, r, b_max, bi, bc, s_exp, r_prev, row, v, tmp);
  double mx = 0.0;
#pragma unroll
  for (int e = 0; e < MAXE; ++e)
    if (e < E && t * E + e < avail) mx = fmax(mx, fabs(v[e]));
  for (int off = 32; off > 0; off >>= 1) mx = fmax(mx, __shfl_xor(mx, off));
  if ((t & 63) == 0) tmp[t >> 6] = mx;
  __syncthreads();
  mx = fmax(fmax(tmp[0], tmp[1]), fmax(tmp[2], tmp[3]));
  const double inv = mx > 0.0 ? 1.0 / mx : 1.0;
#pragma unroll
  for (int e = 0; e < MAXE; ++e) {
    const int j = t * E + e;
    if (e < E && j < avail) {
      v[e] = v[e] * inv;
      row[j] = v[e];
    }
  }
  for (int j = avail + t; j < b_max; j += 256) row[j] = 0.0;
  const int first = (flags & SW_FORCE_FIRST) ? 0 : -1;
  const int last = (flags & SW_FORCE_LAST) ? bc : -1;
  select_row_vals<MAXE>(v, avail, first, last, k, pct, idx + (long long)bi * kmax, cnt + bi, kmax);
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
void launch_sketch_t(const void* q_new, const void* k_new, int batch, int h_q, int h_kv, int d,
                     int B, const int32_t* pos, const int8_t* signs, const int32_t* cols, int r,
                     int b_max, char* state, const void* v_new, void* Kc, void* Vc, int T_max,
                     hipStream_t st) {
  const T* q = reinterpret_cast<const T*>(q_new);
  const T* k = reinterpret_cast<const T*>(k_new);
  const T* v = reinterpret_cast<const T*>(v_new);
  const dim3 grid((unsigned)batch, (unsigned)((b_max + kScoreChunk - 1) / kScoreChunk));
  if (Kc != nullptr)
    hipLaunchKernelGGL((decode_sketch_kernel<T, true>), grid, dim3(256), 0, st, q, k, h_q, h_kv, d,
                       B, pos, signs, cols, r, batch, b_max, state, v, reinterpret_cast<T*>(Kc),
                       reinterpret_cast<T*>(Vc), T_max);
  else
    hipLaunchKernelGGL((decode_sketch_kernel<T, false>), grid, dim3(256), 0, st, q, k, h_q, h_kv, d,
                       B, pos, signs, cols, r, batch, b_max, state, v, static_cast<T*>(nullptr),
                       static_cast<T*>(nullptr), T_max);
}

int strip_pairs(int batch, int d, int r, int b_max) {
  return (decode_layout(batch, d, r, b_max).lda / kStripCols + 1) / 2;
}

}  // namespace

hipError_t launch_decode_sketch(int dtype, const void* q_new, const void* k_new, int batch, int h_q,
                                int h_kv, int d, int B, const int32_t* pos, const int8_t* signs,
                                const int32_t* cols, int r, int b_max, char* state,
                                hipStream_t st, const void* v_new, void* Kc, void* Vc, int T_max) {
  if (dtype == SW_BF16)
    launch_sketch_t<uint16_t>(q_new, k_new, batch, h_q, h_kv, d, B, pos, signs, cols, r, b_max,
                              state, v_new, Kc, Vc, T_max, st);
  else
    launch_sketch_t<float>(q_new, k_new, batch, h_q, h_kv, d, B, pos, signs, cols, r, b_max, state,
                           v_new, Kc, Vc, T_max, st);
  return hipGetLastError();
}

hipError_t launch_decode_walk(const char* state, int batch, int d, int r, int b_max, int B,
                              const int32_t* pos, int s_exp, bool relu, const double* r_prev,
                              double* r_out, hipStream_t st) {
  const dim3 grid((unsigned)batch, (unsigned)strip_pairs(batch, d, r, b_max));
#define SW_NORM_LAUNCH(S8, RELU, E)                                                              \
  hipLaunchKernelGGL((walk_row_norm_kernel<S8, RELU, E>), dim3((unsigned)batch), dim3(256), 0, st, \
                     state, batch, d, r, b_max, B, pos, s_exp, r_prev, r_out)
#define SW_WALK_LAUNCH(S8, RELU)                                                                   \
  do {                                                                                            \
    if (r_prev != nullptr)                                                                        \
      hipLaunchKernelGGL((walk_strip_kernel<S8, RELU>), grid, dim3(kStripThreads), 0, st, state,  \
                         batch, d, r, b_max, B, pos, s_exp, r_prev, r_out);                       \
    switch (row_maxe(b_max)) {                                                                    \
      case 2: SW_NORM_LAUNCH(S8, RELU, 2); break;                                                 \
      case 4: SW_NORM_LAUNCH(S8, RELU, 4); break;                                                 \
      case 8: SW_NORM_LAUNCH(S8, RELU, 8); break;                                                 \
      default: SW_NORM_LAUNCH(S8, RELU, 16); break;                                               \
    }                                                                                             \
  } while (0)
  if (s_exp == 8 && !relu) SW_WALK_LAUNCH(true, false);
  else if (s_exp == 8) SW_WALK_LAUNCH(true, true);
  else if (!relu) SW_WALK_LAUNCH(false, false);
  else SW_WALK_LAUNCH(false, true);
#undef SW_WALK_LAUNCH
#undef SW_NORM_LAUNCH
  return hipGetLastError();
}

namespace {

template <typename T, bool S8, bool RELU>
void launch_layer_t(const void* q_new, const void* k_new, const void* v_new, void* Kc, void* Vc,
                    int T_max, int batch, int h_q, int h_kv, int d, int B, const int32_t* pos,
                    const int8_t* signs, const int32_t* cols, int r, int b_max, char* state,
                    int s_exp, const double* r_prev, double* rows, int k, int pct, uint32_t flags,
                    int32_t* idx, int32_t* cnt, int kmax, hipStream_t st) {
  const int pairs = r_prev != nullptr ? strip_pairs(batch, d, r, b_max) : 0;
  const int chunks = (b_max + kScoreChunk - 1) / kScoreChunk;
  hipLaunchKernelGGL((decode_sketch_walk_kernel<T, S8, RELU>),
                     dim3((unsigned)batch, (unsigned)(pairs + chunks)), dim3(256), 0, st,
                     reinterpret_cast<const T*>(q_new), reinterpret_cast<const T*>(k_new), h_q,
                     h_kv, d, B, pos, signs, cols, r, batch, b_max, state,
                     reinterpret_cast<const T*>(v_new), reinterpret_cast<T*>(Kc),
                     reinterpret_cast<T*>(Vc), T_max, pairs, s_exp, r_prev, rows);
#define SW_SEL_LAUNCH(E)                                                                        \
  hipLaunchKernelGGL((select_decode_norm_kernel<S8, RELU, E>), dim3((unsigned)batch), dim3(256), 0, \
                     st, state, batch, d, r, b_max, B, pos, s_exp, r_prev, rows, k, pct, flags,    \
                     idx, cnt, kmax)
  switch (row_maxe(b_max)) {
    case 2: SW_SEL_LAUNCH(2); break;
    case 4: SW_SEL_LAUNCH(4); break;
    case 8: SW_SEL_LAUNCH(8); break;
    default: SW_SEL_LAUNCH(16); break;
  }
#undef SW_SEL_LAUNCH
}

template <typename T>
void launch_layer_w(bool relu, const void* q_new, const void* k_new, const void* v_new, void* Kc,
                    void* Vc, int T_max, int batch, int h_q, int h_kv, int d, int B,
                    const int32_t* pos, const int8_t* signs, const int32_t* cols, int r, int b_max,
                    char* state, int s_exp, const double* r_prev, double* rows, int k, int pct,
                    uint32_t flags, int32_t* idx, int32_t* cnt, int kmax, hipStream_t st) {
#define SW_LAYER(S8, RELU)                                                                     \
  launch_layer_t<T, S8, RELU>(q_new, k_new, v_new, Kc, Vc, T_max, batch, h_q, h_kv, d, B, pos, \
                              signs, cols, r, b_max, state, s_exp, r_prev, rows, k, pct, flags, \
                              idx, cnt, kmax, st)
  if (s_exp == 8 && !relu) SW_LAYER(true, false);
  else if (s_exp == 8) SW_LAYER(true, true);
  else if (!relu) SW_LAYER(false, false);
  else SW_LAYER(false, true);
#undef SW_LAYER
}

}  // namespace

hipError_t launch_decode_layer(int dtype, const void* q_new, const void* k_new, const void* v_new,
                               void* Kc, void* Vc, int T_max, int batch, int h_q, int h_kv, int d,
                               int B, const int32_t* pos, const int8_t* signs, const int32_t* cols,
                               int r, int b_max, char* state, int s_exp, bool relu,
                               const double* r_prev, double* rows, int k, int pct, uint32_t flags,
                               int32_t* idx, int32_t* cnt, int kmax, hipStream_t st) {
  if (dtype == SW_BF16)
    launch_layer_w<uint16_t>(relu, q_new, k_new, v_new, Kc, Vc, T_max, batch, h_q, h_kv, d, B, pos,
                             signs, cols, r, b_max, state, s_exp, r_prev, rows, k, pct, flags, idx,
                             cnt, kmax, st);
  else
    launch_layer_w<float>(relu, q_new, k_new, v_new, Kc, Vc, T_max, batch, h_q, h_kv, d, B, pos,
                          signs, cols, r, b_max, state, s_exp, r_prev, rows, k, pct, flags, idx,
                          cnt, kmax, st);
  return hipGetLastError();
}

}  // namespace sw
