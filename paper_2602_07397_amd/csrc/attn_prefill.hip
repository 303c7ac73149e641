// Block-sparse causal flash attention over the selected key blocks
// (paper Alg. 1 step 8): for each query head and query block, softmax over
// the tokens of the selected blocks that precede each query, renormalised
// over those keys only.
//
// bf16 kernel. Work item = (query block, KV head g, slice of the group's query
// heads). A 512-thread workgroup has 8 wavefronts, two per SIMD; each owns 32
// query rows of one head (a B = 128 block takes four wavefronts per head, a
// B = 64 block two), so a workgroup serves two (B = 128) or four (B = 64)
// query heads of the same KV group from one copy of each K/V tile in LDS.
// The two wavefronts of a SIMD cover each other's LDS and barrier waits.
//
// Per wavefront and 32-key sub-tile the scores are computed transposed,
// S^T = K Q^T (v_mfma_f32_32x32x16_bf16, fp32 accumulate), so a lane owns one
// query column and its partial row sum; the other half-wave holds the rest of
// the row (one v_permlane32_swap combines them). P (rounded to bf16) feeds the
// B operand of O^T = V^T P^T straight from the accumulator layout. V stays in
// its natural row layout in LDS and the V^T operand is read with
// ds_read_b64_tr_b16, which hands each lane four consecutive keys of one
// dimension.
//
// Software pipeline over 32-key sub-tiles u, in a fixed issue order:
//   phase A: the score MFMAs of u+1, interleaved with the exponentials of
//            keys 16..31 of P(u);
//   phase B: the P.V MFMAs of u, interleaved with the exponentials of keys
//            0..15 of P(u+1).
// The exponent reference of a row does not track the row max on this path:
// between the phases, a row whose partial sum over P(u) exceeds kSumLimit
// (which bounds every element) takes the exact max of the sub-tile, rescales
// O and its sum and recomputes P(u) (rare, wave-uniform branch). Since
// O = sum(P V) / sum(P) for any common reference, the result does not depend
// on which reference was used.
//
// K/V tiles of 64 keys go through three LDS stages from registers loaded one
// tile ahead. The selected blocks are compacted in LDS at the start: valid
// blocks j < i first (never masked: only a sequence's last block can be
// partial), then the diagonal block i. The pipeline runs on into the
// diagonal block up to the sub-tile a wavefront's rows cross, which alone is
// masked (causal and sequence end); the sub-tiles after it are skipped. Work
// items run longest-first (query blocks in descending order, the selection
// budget grows with the block index) and the workgroups of one (query block,
// KV head) are placed on one XCD so they share the K/V blocks through that
// XCD's L2.
#include <type_traits>

#include "sw_common.h"
#include "sw_internal.h"

namespace sw {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int KT = 64;                 // keys per LDS tile
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNoRef = -1.0e30f;     // exponent reference before any key
constexpr float kSumLimit = 65536.0f;  // bound on a pipelined P sub-tile's partial row sum
constexpr int kPfWaves = 8;            // wavefronts per bf16 workgroup

// ---------------------------------------------------------------------------
// work mapping
// ---------------------------------------------------------------------------

// Rows with local block index >= x over all sequences (x may differ per
// lane); lane j of bl holds the block count of sequence j.
__device__ __forceinline__ int rows_from(int bl, int n_seqs, int x) {
  int c = 0;
  for (int j = 0; j < n_seqs; ++j) c += max(0, __builtin_amdgcn_readlane(bl, j) - x);
  return c;
}

// rho-th block row in longest-first order (local index descending, then
// sequence ascending). Returns the global row and the local index. Called by
// whole wavefronts: the block counts are spread over the lanes (at most 64
// sequences) and the local index is found by a 64-way search, each round
// testing 64 candidate indices at once.
__device__ __forceinline__ void lpt_row(const SeqMeta& m, int rho, int* row, int* s_out,
                                        int* i_out) {
  static_assert(SW_MAX_SEQS <= 64, "one sequence per lane");
  const int lane = threadIdx.x & 63;
  int bl = 0;
#pragma unroll
  for (int j = 0; j < SW_MAX_SEQS; ++j) {
    const int bj = m.blk_start[j + 1] - m.blk_start[j];
    bl = (lane == j && j < m.n_seqs) ? bj : bl;
  }
  // invariant: the answer (largest x with rows_from(x) > rho) lies in [lo, hi]
  int lo = 0, hi = m.max_b - 1;
  while (lo < hi) {
    const int step = (hi - lo + 63) >> 6;
    const int x = min(hi, lo + (lane + 1) * step);
    // rows_from decreases in x, so the passing candidates are a lane prefix
    const int pass = __popcll(__ballot(rows_from(bl, m.n_seqs, x) > rho));
    const int nlo = (pass == 0) ? lo : min(hi, lo + pass * step);
    hi = (pass == 64) ? hi : min(hi, lo + (pass + 1) * step) - 1;
    lo = nlo;
  }
  const int i = lo;
  const int k = rho - rows_from(bl, m.n_seqs, i + 1);   // rank among sequences longer than i
  const unsigned long long longer = __ballot(bl > i);
  const bool mine = ((longer >> lane) & 1ull) && (int)__popcll(longer & ((1ull << lane) - 1ull)) == k;
  const int s = __ffsll((unsigned long long)__ballot(mine)) - 1;
  *row = m.blk_start[s] + i;
  *s_out = s;
  *i_out = i;
}

// ---------------------------------------------------------------------------
// bf16 kernel
// ---------------------------------------------------------------------------

template <int D>
struct BfLds {
  static constexpr int KS = D + 8;     // K row stride (elements): rows 16 bytes apart in bank space
  static constexpr int VS = D + 32;    // V row stride (elements): rows 64 bytes apart in bank space
  static constexpr int K_ELEMS = KT * KS;
  static constexpr int V_ELEMS = KT * VS;
  static constexpr int STAGE = K_ELEMS + V_ELEMS;
  static constexpr int NST = 3;
};

// Raw buffer descriptor word 3 for gfx9-family untyped loads (32-bit data format).
constexpr int kBufWord3 = 0x00020000;

__device__ __forceinline__ float max_other_half(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_other_half(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

#define SW_INL __attribute__((always_inline))

template <int D, int BLK>
__global__ __launch_bounds__(kPfWaves * 64, 1) void attn_prefill_bf16_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, int h_q, int h_kv, long long N, SeqMeta m,
    const int32_t* __restrict__ idx, const int32_t* __restrict__ cnt, int kmax, float sl2,
    uint16_t* __restrict__ O, float* __restrict__ lse, int groups, int sg) {
  using L = BfLds<D>;
  constexpr int NT = kPfWaves * 64;        // threads
  __shared__ __attribute__((aligned(16))) uint16_t lds[L::NST * L::STAGE];
  __shared__ int blist[SW_MAX_BLOCKS];
  __shared__ int wtot[kPfWaves];

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
  constexpr int WPB = BLK / 32;            // wavefronts per (query head, block)
  constexpr int TPB = BLK / KT;            // key tiles per block
  const int G = h_q / h_kv;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int l = tid & 63;
  const int hl = l >> 5;                   // half-wave
  const int ln = l & 31;                   // lane within half
  const int task = mu * kPfWaves + w;
  const int u = g * G + task / WPB;        // query head (meaningful only when active)
  const int seq0 = m.tok_start[s];
  const int seq1 = m.tok_start[s + 1];
  // 32-row group of the block owned by this wavefront. Wavefronts w and
  // w + 4 share a SIMD; the upper half takes the groups in reverse order so
  // the two hold complementary groups (g and WPB-1-g) and every SIMD has the
  // same number of unmasked diagonal sub-tiles.
  const int rgrp = (w >= kPfWaves / 2) ? WPB - 1 - task % WPB : task % WPB;
  const int q0 = seq0 + i * BLK + rgrp * 32;   // first query row of this wavefront
  const bool active = (task < G * WPB) && (q0 < seq1);
  const int qpos = q0 + ln;                // this lane's query row

  // The selection count and the first chunk of the selection list are
  // loaded first, then Q: the list is needed first. The chunk lies within the
  // row's kmax entries whatever cnt holds.
  const int32_t* sel = idx + (long long)row * kmax;
  const int nsel = min(cnt[row], kmax);
  int jnext = (tid < kmax) ? sel[tid] : -1;

  // ---- Q fragments: lane holds query qpos, dims kk*16 + hl*8 .. +7 ----
  bf16x8 qf[D / 16];
  {
    const bool ok = active && qpos < seq1;
    const uint16_t* qrow = Q + ((long long)(ok ? u : 0) * N + (ok ? qpos : 0)) * D;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      uint4 v = ok ? *reinterpret_cast<const uint4*>(qrow + kk * 16 + hl * 8) : make_uint4(0, 0, 0, 0);
      qf[kk] = __builtin_bit_cast(bf16x8, v);
    }
  }

  // ---- selected blocks, compacted: valid j < i in list order, then i ----
  // Per chunk of NT entries each wavefront publishes its count of blocks
  // j < i (low 16 bits) and whether it saw the diagonal block (bit 16).
  int n_off = 0, sdiag = 0;
  for (int base = 0; base < nsel; base += NT) {
    const int e = base + tid;
    const int j = (e < nsel) ? jnext : -1;
    jnext = (e + NT < nsel) ? sel[e + NT] : -1;
    const bool off = (j >= 0 && j < i);
    const unsigned long long bal = __ballot(off);
    const bool dg = __ballot(j == i) != 0ull;
    const int pre = __popcll(bal & ((1ull << l) - 1ull));
    if (l == 0) wtot[w] = __popcll(bal) | (dg ? 0x10000 : 0);
    __syncthreads();
    int woff = 0, tot = 0;
#pragma unroll
    for (int q = 0; q < kPfWaves; ++q) {
      const int c = wtot[q];
      woff += (q < w) ? (c & 0xffff) : 0;
      tot += c & 0xffff;
      sdiag |= c >> 16;
    }
    if (off && n_off + woff + pre < SW_MAX_BLOCKS) blist[n_off + woff + pre] = j;
    n_off = min(n_off + tot, SW_MAX_BLOCKS);
    __syncthreads();
  }
  const int n_blk = n_off + sdiag;
  const int ntiles = n_blk * TPB;
  const int nofft = n_off * TPB;           // tiles before the diagonal block

  // ---- K/V staging: global -> registers -> LDS, 16-byte chunks ----
  constexpr int KCH = D / 8;               // chunks per key row
  constexpr int KP = (KT * KCH) / NT;      // chunks per thread for K (and for V)
  static_assert(KP >= 1 && KP * NT == KT * KCH, "tile chunks must divide over the workgroup");
  uint4 kreg[KP], vreg[KP];
  int goff[KP], kloff[KP], vloff[KP];
#pragma unroll
  for (int p = 0; p < KP; ++p) {
    const int e = tid + p * NT;
    const int r = e / KCH, ch = e % KCH;
    goff[p] = (r * D + ch * 8) * 2;
    kloff[p] = r * L::KS + ch * 8;
    vloff[p] = r * L::VS + ch * 8;
  }
  const uint16_t* Kg = K + (long long)g * N * D;
  const uint16_t* Vg = V + (long long)g * N * D;
  // first key of tile t (wave-uniform)
  auto tile_k0 = [&](int t) SW_INL {
    const int jj = t / TPB;
    const int j = (jj < n_off) ? __builtin_amdgcn_readfirstlane(blist[jj]) : i;
    return seq0 + j * BLK + (t % TPB) * KT;
  };
  // Raw buffer loads through a descriptor based at the tile's first key k0
  // and sized to the end of the sequence: keys past the end read as zero
  // without per-lane tests (the diagonal-tile mask removes them).
  auto load_into = [&](int k0, uint4 (&kr)[KP], uint4 (&vr)[KP]) SW_INL {
    const int bytes = max(0, (seq1 - k0) * D * 2);
    const __amdgpu_buffer_rsrc_t rk =
        __builtin_amdgcn_make_buffer_rsrc((void*)(Kg + (long long)k0 * D), (short)0, bytes, kBufWord3);
    const __amdgpu_buffer_rsrc_t rv =
        __builtin_amdgcn_make_buffer_rsrc((void*)(Vg + (long long)k0 * D), (short)0, bytes, kBufWord3);
#pragma unroll
    for (int p = 0; p < KP; ++p) {
      auto a = __builtin_amdgcn_raw_buffer_load_b128(rk, goff[p], 0, 0);
      kr[p] = __builtin_bit_cast(uint4, a);
      auto b = __builtin_amdgcn_raw_buffer_load_b128(rv, goff[p], 0, 0);
      vr[p] = __builtin_bit_cast(uint4, b);
    }
  };
  auto load_tile_at = [&](int k0) SW_INL { load_into(k0, kreg, vreg); };
  auto load_tile = [&](int t) SW_INL { load_tile_at(tile_k0(t)); };
  auto store_from = [&](int st, const uint4 (&kr)[KP], const uint4 (&vr)[KP]) SW_INL {
    uint16_t* ks = lds + st * L::STAGE;
    uint16_t* vs = ks + L::K_ELEMS;
#pragma unroll
    for (int p = 0; p < KP; ++p) {
      *reinterpret_cast<uint4*>(ks + kloff[p]) = kr[p];
      *reinterpret_cast<uint4*>(vs + vloff[p]) = vr[p];
    }
  };
  auto store_tile = [&](int st) SW_INL { store_from(st, kreg, vreg); };

  // ---- running state ----
  f32x16 oacc[D / 32];
#pragma unroll
  for (int td = 0; td < D / 32; ++td)
#pragma unroll
    for (int j = 0; j < 16; ++j) oacc[td][j] = 0.0f;
  float mref = kNoRef;
  float lsum = 0.0f;
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  constexpr int NKK = D / 16;              // score MFMAs per sub-tile
  constexpr int NPV = 2 * (D / 32);        // P.V MFMAs per sub-tile: (chunk, dim block)
  constexpr int QK_PER_PAIR = NKK / 4;     // score MFMAs per element pair (phase A)
  constexpr int PV_PER_PAIR = NPV / 4;     // P.V MFMAs per element pair (phase B)
  constexpr int kAhead = 3;                // K and V^T operands are read this many MFMAs ahead
  // V^T operand lane offset: lane (ln, hl) reads with ds_read_b64_tr_b16 from
  // key row c*16 + 4*hl + (ln%16)/4 (+8) and dims td*32 + 16*(ln/16) + 4*(ln%4);
  // it receives dim td*32 + ln of keys c*16 + 4*hl + 0..3 and
  // c*16 + 8 + 4*hl + 0..3, the keys its P operand holds.
  const int vlane = (4 * hl + ((ln & 15) >> 2)) * L::VS + 16 * (ln >> 4) + 4 * (ln & 3);

  // Scores of 32 keys (half h2 of a 64-key tile) x 32 queries, transposed:
  // element j is key h2*32 + 8*(j/4) + 4*hl + j%4, query qpos.
  auto qk_sub = [&](const uint16_t* ks, int h2, f32x16& S) SW_INL {
#pragma unroll
    for (int j = 0; j < 16; ++j) S[j] = 0.0f;
    const uint16_t* kr = ks + (h2 * 32 + ln) * L::KS + hl * 8;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(kr + kk * 16);
      S = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], S, 0, 0, 0);
    }
  };
  // causal + sequence-end mask of a diagonal-block sub-tile (raw scores)
  auto mask_sub = [&](int t, int h2, f32x16& S) SW_INL {
    const int k0 = tile_k0(t) + h2 * 32;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int kp = k0 + (j >> 2) * 8 + hl * 4 + (j & 3);
      if (kp > qpos || kp >= seq1) S[j] = -INFINITY;
    }
  };
  // row max of a sub-tile (log2 units)
  auto row_max = [&](const f32x16& S) SW_INL {
    float a = -INFINITY;
#pragma unroll
    for (int j = 0; j < 16; ++j) a = fmaxf(a, S[j]);
    return max_other_half(a) * sl2;
  };
  auto rescale_to = [&](float nref) SW_INL {
    const float alpha = __builtin_amdgcn_exp2f(mref - nref);
    mref = nref;
    lsum *= alpha;
#pragma unroll
    for (int td = 0; td < D / 32; ++td)
#pragma unroll
      for (int j = 0; j < 16; ++j) oacc[td][j] *= alpha;
  };
  // element pair e (elements 2e, 2e+1): P word and partial row sum
  auto pair = [&](const f32x16& S, int e, uint32_t& word, float& ts) SW_INL {
    const float nr = -mref;
    const float p0 = __builtin_amdgcn_exp2f(fmaf(S[2 * e], sl2, nr));
    const float p1 = __builtin_amdgcn_exp2f(fmaf(S[2 * e + 1], sl2, nr));
    word = pack_bf16x2(p0, p1);
    ts = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, word), ones, ts, false);
  };
  auto vread = [&](const uint16_t* vr, int n) SW_INL {
    const uint16_t* pp = vr + (n / (D / 32)) * 16 * L::VS + (n % (D / 32)) * 32;
    const i16x4 r0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) i16x4*)(pp));
    const i16x4 r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) i16x4*)(pp + 8 * L::VS));
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(r0, r1, 0, 1, 2, 3, 4, 5, 6, 7));
  };
  // rare path: exact row max of S, new reference, rescale, recompute P(u)
  auto refix = [&](const f32x16& S, uint32_t (&w0)[4], uint32_t (&w1)[4], float& ts) SW_INL {
    rescale_to(fmaxf(mref, row_max(S)));
    ts = 0.0f;
#pragma unroll
    for (int e = 0; e < 4; ++e) pair(S, e, w0[e], ts);
#pragma unroll
    for (int e = 0; e < 4; ++e) pair(S, 4 + e, w1[e], ts);
  };
  auto check = [&](const f32x16& cur, uint32_t (&w0)[4], uint32_t (&w1)[4], float& ts) SW_INL {
    if (__any(ts > kSumLimit)) refix(cur, w0, w1, ts);
    lsum += ts;
  };
  // phase B: P.V of sub-tile u, with the chunk-0 exponentials of the next
  // sub-tile's scores when HAS_NEXT
  auto phase_b = [&](const uint16_t* vr, const uint32_t (&w0)[4], const uint32_t (&w1)[4],
                     bf16x8 (&vf)[NPV], const f32x16& nxt, uint32_t (&wn)[4], float& tn,
                     auto has_next) SW_INL {
    constexpr bool HAS_NEXT = decltype(has_next)::value;
    const bf16x8 pb[2] = {__builtin_bit_cast(bf16x8, w0), __builtin_bit_cast(bf16x8, w1)};
    tn = 0.0f;
#pragma unroll
    for (int n = 0; n < NPV; ++n) {
      if (n + kAhead < NPV) vf[n + kAhead] = vread(vr, n + kAhead);
      oacc[n % (D / 32)] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[n], pb[n / (D / 32)],
                                                                   oacc[n % (D / 32)], 0, 0, 0);
      if (HAS_NEXT && (n % PV_PER_PAIR) == PV_PER_PAIR - 1) {
        const int e = n / PV_PER_PAIR;               // 0..3
        pair(nxt, e, wn[e], tn);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // One pipeline sub-step (see the header): cur = S(u) with chunk-0 words wc
  // and their partial sum tc; produces nxt = S(u+1), its chunk-0 words wn and
  // partial sum tn.
  // tmask >= 0: S(u+1) is the wavefront's diagonal sub-tile, half h2n of
  // tile tmask, and is masked before its exponentials.
  auto sub = [&](f32x16& cur, uint32_t (&wc)[4], float& tc, f32x16& nxt, uint32_t (&wn)[4],
                 float& tn, const uint16_t* ksn, int h2n, const uint16_t* vs, int c0,
                 int tmask) SW_INL {
    const uint16_t* kr = ksn + (h2n * 32 + ln) * L::KS + hl * 8;
    const uint16_t* vr = vs + vlane + c0 * 16 * L::VS;
    uint32_t w1[4];
    bf16x8 kf[NKK];
    bf16x8 vf[NPV];
#pragma unroll
    for (int q = 0; q < kAhead; ++q) kf[q] = *reinterpret_cast<const bf16x8*>(kr + q * 16);
#pragma unroll
    for (int j = 0; j < 16; ++j) nxt[j] = 0.0f;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      if (kk + kAhead < NKK) kf[kk + kAhead] = *reinterpret_cast<const bf16x8*>(kr + (kk + kAhead) * 16);
      if (kk >= NKK - kAhead) vf[kk - (NKK - kAhead)] = vread(vr, kk - (NKK - kAhead));
      nxt = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk], qf[kk], nxt, 0, 0, 0);
      if ((kk % QK_PER_PAIR) == QK_PER_PAIR - 1) {
        const int e = kk / QK_PER_PAIR;              // 0..3
        pair(cur, 4 + e, w1[e], tc);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if (tmask >= 0) mask_sub(tmask, h2n, nxt);
    check(cur, wc, w1, tc);
    phase_b(vr, wc, w1, vf, nxt, wn, tn, std::true_type{});
  };
  // final sub-step of a wavefront's run: no scores ahead
  auto sub_last = [&](f32x16& cur, uint32_t (&wc)[4], float& tc, const uint16_t* vs, int c0) SW_INL {
    const uint16_t* vr = vs + vlane + c0 * 16 * L::VS;
    uint32_t w1[4];
    bf16x8 vf[NPV];
#pragma unroll
    for (int q = 0; q < kAhead; ++q) vf[q] = vread(vr, q);
#pragma unroll
    for (int e = 0; e < 4; ++e) pair(cur, 4 + e, w1[e], tc);
    check(cur, wc, w1, tc);
    uint32_t wdummy[4];
    float tdummy;
    phase_b(vr, wc, w1, vf, cur, wdummy, tdummy, std::false_type{});
  };

  // Stages: during tile step t, K/V(t) are in stv, K(t+1) in stk, and tile
  // t+2 is written to stw from the registers loaded during step t-1; tile
  // t+3 is loaded into those registers.
  // The first key of tile t+3 is looked up one step ahead (k0_ahead), so the
  // LDS read of the block list never stalls the loads.
  int stv = 0, stk = 1, stw = 2;
  int k0_ahead = 0;
  auto stage_io = [&](int t) SW_INL {
    if (t + 2 < ntiles) store_tile(stw);
    if (t + 3 < ntiles) load_tile_at(k0_ahead);
    if (t + 4 < ntiles) k0_ahead = tile_k0(t + 4);
  };
  auto next_stage = [&]() SW_INL {
    const int t0 = stv;
    stv = stk;
    stk = stw;
    stw = t0;
    __syncthreads();
  };
  f32x16 sX, sY;
  uint32_t wX[4], wY[4];
  float tX = 0.0f, tY = 0.0f;
  // Last 32-key sub-tile of this wavefront's run, counting two per tile:
  // the off-diagonal blocks, then in the diagonal block the sub-tiles up to
  // the one its rows cross (number rgrp; the later ones lie after all its
  // rows and are skipped, the earlier ones precede them and need no mask).
  // Wavefronts without rows stop after the off-diagonal blocks.
  const int uend = 2 * nofft - 1 + ((active && sdiag) ? rgrp + 1 : 0);
  // off-diagonal tile t < nofft-1: both halves, the second computing the
  // first half of tile t+1 (every wavefront's run goes past it)
  auto tile_step = [&](int t) SW_INL {
    stage_io(t);
    const uint16_t* kt = lds + stv * L::STAGE;
    const uint16_t* vs = kt + L::K_ELEMS;
    sub(sX, wX, tX, sY, wY, tY, kt, 1, vs, 0, -1);
    sub(sY, wY, tY, sX, wX, tX, lds + stk * L::STAGE, 0, vs, 2, -1);
    next_stage();
  };
  // any later tile: each half continues, ends or skips this wavefront's run
  auto tile_end = [&](int t) SW_INL {
    stage_io(t);
    const uint16_t* kt = lds + stv * L::STAGE;
    const uint16_t* vs = kt + L::K_ELEMS;
    const int v0 = 2 * t;
    if (v0 + 1 <= uend) sub(sX, wX, tX, sY, wY, tY, kt, 1, vs, 0, (v0 + 1 == uend) ? t : -1);
    else if (v0 == uend) sub_last(sX, wX, tX, vs, 0);
    if (v0 + 2 <= uend)
      sub(sY, wY, tY, sX, wX, tX, lds + stk * L::STAGE, 0, vs, 2, (v0 + 2 == uend) ? t + 1 : -1);
    else if (v0 + 1 == uend) sub_last(sY, wY, tY, vs, 2);
    next_stage();
  };

  if (ntiles > 0) {
    // tiles 0 and 1 are loaded together (a second register set), then tile 2
    uint4 k1reg[KP], v1reg[KP];
    load_tile(0);
    if (ntiles > 1) load_into(tile_k0(1), k1reg, v1reg);
    store_tile(0);
    if (ntiles > 1) store_from(1, k1reg, v1reg);
    if (ntiles > 2) load_tile(2);
    if (ntiles > 3) k0_ahead = tile_k0(3);
    __syncthreads();
    if (uend >= 0) {
      // scores of the first sub-tile; its chunk-0 words are left to the
      // first check (an infinite partial sum forces the exact reference)
      qk_sub(lds, 0, sX);
      if (uend == 0) mask_sub(0, 0, sX);
      tX = INFINITY;
#pragma unroll
      for (int e = 0; e < 4; ++e) wX[e] = 0u;
    }
    int t = 0;
    for (; t + 1 < nofft; ++t) tile_step(t);
    for (; t < ntiles; ++t) tile_end(t);
  }

  // ---- epilogue ----
  // The wavefront's 32 x D output rows are normalised into LDS (the K/V
  // stages are free once every wavefront has passed the barrier) and written
  // back row-contiguous: rows q0..q0+31 of head u are one contiguous run of
  // O, so each 16-byte-per-lane store covers 64 / (D / 8) whole rows.
  const float ltot = sum_other_half(lsum);
  const float inv = ltot > 0.0f ? 1.0f / ltot : 0.0f;
  constexpr int OS = D + 8;                // output row stride in LDS (elements)
  static_assert(kPfWaves * 32 * OS <= L::NST * L::STAGE, "output staging must fit the K/V stages");
  __syncthreads();
  uint16_t* ob = lds + w * 32 * OS;
#pragma unroll
  for (int td = 0; td < D / 32; ++td) {
#pragma unroll
    for (int jb = 0; jb < 4; ++jb) {
      uint2 st;
      st.x = pack_bf16x2(oacc[td][jb * 4 + 0] * inv, oacc[td][jb * 4 + 1] * inv);
      st.y = pack_bf16x2(oacc[td][jb * 4 + 2] * inv, oacc[td][jb * 4 + 3] * inv);
      *reinterpret_cast<uint2*>(ob + ln * OS + td * 32 + jb * 8 + hl * 4) = st;
    }
  }
  if (!active) return;
  constexpr int CPR = D / 8;               // 16-byte chunks per row
  constexpr int RPI = 64 / CPR;            // rows per store instruction
  const int rr = l / CPR, cc = l % CPR;
  uint16_t* obase = O + ((long long)u * N + q0) * D;
#pragma unroll
  for (int it = 0; it < 32 / RPI; ++it) {
    const int r = it * RPI + rr;
    const uint4 v = *reinterpret_cast<const uint4*>(ob + r * OS + cc * 8);
    if (q0 + r < seq1) *reinterpret_cast<uint4*>(obase + (long long)r * D + cc * 8) = v;
  }
  if (lse && hl == 0 && qpos < seq1)
    lse[(long long)u * N + qpos] = (ltot > 0.0f) ? (mref + log2f(ltot)) / kLog2e : -INFINITY;
}

#undef SW_INL

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
  const int groups = (int)(nb * h_kv);
  const float sl2 = scale * kLog2e;
  if (dtype == SW_BF16) {
    // 32 query rows per wavefront, kPfWaves wavefronts per workgroup
    const int sg = (G * (meta.B / 32) + kPfWaves - 1) / kPfWaves;
    const unsigned grid = (unsigned)(((groups + 7) / 8) * 8 * sg);
    auto q = reinterpret_cast<const uint16_t*>(Q);
    auto k = reinterpret_cast<const uint16_t*>(K);
    auto v = reinterpret_cast<const uint16_t*>(V);
    auto o = reinterpret_cast<uint16_t*>(O);
#define SW_LAUNCH_BF16(DD, BB)                                                                  \
  hipLaunchKernelGGL((attn_prefill_bf16_kernel<DD, BB>), dim3(grid), dim3(kPfWaves * 64), 0, st, q, k, v, h_q, \
                     h_kv, N, meta, idx, cnt, kmax, sl2, o, lse, groups, sg)
    if (d == 128 && meta.B == 128) SW_LAUNCH_BF16(128, 128);
    else if (d == 128) SW_LAUNCH_BF16(128, 64);
    else if (meta.B == 128) SW_LAUNCH_BF16(64, 128);
    else SW_LAUNCH_BF16(64, 64);
#undef SW_LAUNCH_BF16
  } else {
    const int hpw = (meta.B == 64) ? 2 : 1;
    const int sg = (G + hpw - 1) / hpw;
    const unsigned grid = (unsigned)(((groups + 7) / 8) * 8 * sg);
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
