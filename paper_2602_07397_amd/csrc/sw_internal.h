// Launchers shared between the kernel translation units and the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sw_common.h"

namespace sw {

// Byte layout of one layer's decode state (every section 256-byte aligned):
//   double A_scale[batch]        score scale c frozen at its prefill value
//   int32  col0[batch]           first key block whose column decode fills
//   int32  cnt[batch][2][2]      token counts of the open query / key block,
//                                two copies selected by the position's parity
//   double bar[batch][2][2][d]   running means of the open query / key block,
//                                two copies selected by the position's parity
//   double qt[batch][r]          sketch of the current token's query
//   double Qs[batch][b_max][r]   sketch of every query-block representative
//   double Ks[batch][b_max][r]   sketch of every key-block representative
//   float  rowc[batch][b_max]    the open block's score row A[b_cur][:] and
//   float  colc[batch][b_max]    column A[:][b_cur] as the last step wrote
//                                them (contiguous copies of cache entries)
//   float  A[batch][lda/32][b_max][32]  block-score cache in strips of 32
//                                columns (entry (m, j) at cache_at(b_max, m, j)
//                                within a sequence), lda = b_max rounded up
//                                to a multiple of 32
// The step at position p reads the open-block means and counts of copy
// (p + 1) % 2 (written by the step at p - 1) and writes copy p % 2, so every
// workgroup of a step reads the previous values while one of them writes
// the new ones.
struct DecodeLayout {
  int64_t scale, col0, cnt, bar, qt, qs, ks, rowc, colc, a, total;
  int lda;
};

__host__ __device__ inline DecodeLayout decode_layout(int batch, int d, int r, int b_max) {
  auto al = [](int64_t x) { return (x + 255) / 256 * 256; };
  DecodeLayout L;
  L.lda = (b_max + 31) & ~31;
  int64_t o = 0;
  L.scale = o;  o = al(o + 8LL * batch);
  L.col0 = o;   o = al(o + 4LL * batch);
  L.cnt = o;    o = al(o + 16LL * batch);
  L.bar = o;    o = al(o + 32LL * batch * d);
  L.qt = o;     o = al(o + 8LL * batch * r);
  L.qs = o;     o = al(o + 8LL * batch * b_max * r);
  L.ks = o;     o = al(o + 8LL * batch * b_max * r);
  L.rowc = o;   o = al(o + 4LL * batch * b_max);
  L.colc = o;   o = al(o + 4LL * batch * b_max);
  L.a = o;      o = al(o + 4LL * batch * b_max * L.lda);
  L.total = o;
  return L;
}

// Offset (in floats) of score (m, j) within one sequence's cache: the cache
// is stored as strips of 32 columns, each strip's rows contiguous (128 bytes
// per row), so a walk over one strip's rows reads one contiguous range.
__host__ __device__ inline int cache_at(int b_max, int m, int j) {
  return ((j >> 5) * b_max + m) * 32 + (j & 31);
}

constexpr int kDecodeMaxSplits = 32;

int64_t sketch_workspace_bytes(int h_q, int h_kv, int d, int64_t nb);

hipError_t launch_sketch(int dtype, const void* Q, const void* K, int h_q, int h_kv, int d,
                         const SeqMeta& meta, int64_t nb, long long N, const int8_t* signs,
                         const int32_t* cols, int r, double* Qs, double* Ks, double* A,
                         double* A_scale, double* Qbar, double* Kbar, void* ws, hipStream_t st);

int64_t walk_workspace_bytes(int variant, int64_t nm);

hipError_t launch_walk(int variant, const double* A, const double* A_scale, int s_exp,
                       double logit_scale, const SeqMeta& meta, int64_t nb, const double* R_prev,
                       double* R_out, double* ws, hipStream_t st);

hipError_t launch_select(const double* R, const SeqMeta& meta, int64_t nb, int k, int pct,
                         uint32_t flags, int32_t* idx, int32_t* cnt, int kmax, hipStream_t st);

hipError_t launch_attn_prefill(int dtype, const void* Q, const void* K, const void* V, int h_q,
                               int h_kv, int d, long long N, const SeqMeta& meta, int64_t nb,
                               const int32_t* idx, const int32_t* cnt, int kmax, float scale,
                               void* O, float* lse, hipStream_t st);

hipError_t launch_decode_init(char* state, int batch, int d, int r, int b_max, int seq, int n, int B,
                              const double* Qs, const double* Ks, const double* A,
                              const double* A_scale, const double* Qbar, const double* Kbar,
                              hipStream_t st);

hipError_t launch_kv_append(int dtype, const void* k_new, const void* v_new, void* Kc, void* Vc,
                            int batch, int h_kv, int d, int T_max, const int32_t* pos,
                            hipStream_t st);

hipError_t launch_decode_sketch(int dtype, const void* q_new, const void* k_new, int batch, int h_q,
                                int h_kv, int d, int B, const int32_t* pos, const int8_t* signs,
                                const int32_t* cols, int r, int b_max, char* state,
                                hipStream_t st, const void* v_new = nullptr, void* Kc = nullptr,
                                void* Vc = nullptr, int T_max = 0);

// Alg. 2 step 5 for the per-layer entry point: the walk row of every
// sequence, divided by its largest magnitude, into r_out [batch][b_max].
hipError_t launch_decode_walk(const char* state, int batch, int d, int r, int b_max, int B,
                              const int32_t* pos, int s_exp, bool relu, const double* r_prev,
                              double* r_out, hipStream_t st);

// Alg. 2 steps 1-6 of one layer for the one-call step: the incremental
// sketch with the KV append, side by side with the walk over the score
// entries the sketch leaves unchanged, then the walk row finished, normalised
// and written to rows [batch][b_max], and its selection.
hipError_t launch_decode_layer(int dtype, const void* q_new, const void* k_new, const void* v_new,
                               void* Kc, void* Vc, int T_max, int batch, int h_q, int h_kv, int d,
                               int B, const int32_t* pos, const int8_t* signs, const int32_t* cols,
                               int r, int b_max, char* state, int s_exp, bool relu,
                               const double* r_prev, double* rows, int k, int pct, uint32_t flags,
                               int32_t* idx, int32_t* cnt, int kmax, hipStream_t st);

hipError_t launch_select_decode(const double* rows, int batch, int b_max, int B,
                                const int32_t* pos, int k, int pct, uint32_t flags, int32_t* idx,
                                int32_t* cnt, int kmax, hipStream_t st);

int decode_attn_splits(int batch, int h_kv);

// Device address of this device's fixed scratch array
// (SW_NOALLOC_SCRATCH_BYTES), looked up on the first call on each device.
hipError_t noalloc_scratch(void** out);

hipError_t launch_attn_decode(int dtype, const void* q, const void* Kc, const void* Vc, int batch,
                              int h_q, int h_kv, int d, int T_max, int B, const int32_t* pos,
                              const int32_t* idx, const int32_t* cnt, int kmax, float scale,
                              void* O, float* ws, hipStream_t st);

}  // namespace sw
