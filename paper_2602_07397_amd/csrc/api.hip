// C ABI of the sketch-and-walk library: host-side validation, layout
// computation and dispatch to the kernel launchers. Nothing here touches the
// GPU before every argument has been checked.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <string>

#include "sw_common.h"
#include "sw_internal.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return SW_OK;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

bool is_pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }

int check_ptr(const void* p, size_t align, const char* name) {
  if (p == nullptr) return fail(SW_ERR_INVALID_ARG, "%s is NULL", name);
  if (!aligned(p, align)) return fail(SW_ERR_INVALID_ARG, "%s is not %zu-byte aligned", name, align);
  return SW_OK;
}

#define CHECK(x)              \
  do {                        \
    int rc_ = (x);            \
    if (rc_ != SW_OK) return rc_; \
  } while (0)

// Builds the per-call sequence layout from host cu_seqlens.
int build_meta(int n_seqs, const int32_t* cu, int B, sw::SeqMeta* m, int64_t* nb, int64_t* nm) {
  if (n_seqs < 1 || n_seqs > SW_MAX_SEQS)
    return fail(SW_ERR_INVALID_ARG, "n_seqs=%d outside [1, %d]", n_seqs, SW_MAX_SEQS);
  if (cu == nullptr) return fail(SW_ERR_INVALID_ARG, "cu_seqlens is NULL");
  if (B < 16 || B > 1024 || B % 16 != 0)
    return fail(SW_ERR_INVALID_ARG, "B=%d must be a multiple of 16 in [16, 1024]", B);
  if (cu[0] != 0) return fail(SW_ERR_INVALID_ARG, "cu_seqlens[0]=%d must be 0", cu[0]);
  memset(m, 0, sizeof(*m));
  m->n_seqs = n_seqs;
  m->B = B;
  int64_t blocks = 0, mat = 0;
  int max_b = 0;
  for (int s = 0; s < n_seqs; ++s) {
    const int64_t len = (int64_t)cu[s + 1] - cu[s];
    if (len < 1) return fail(SW_ERR_INVALID_ARG, "sequence %d has length %lld < 1", s, (long long)len);
    const int64_t b = (len + B - 1) / B;
    if (b > SW_MAX_BLOCKS)
      return fail(SW_ERR_UNSUPPORTED, "sequence %d has %lld blocks > %d", s, (long long)b, SW_MAX_BLOCKS);
    m->tok_start[s] = cu[s];
    m->blk_start[s] = (int)blocks;
    m->mat_start[s] = mat;
    blocks += b;
    mat += b * b;
    if (b > max_b) max_b = (int)b;
  }
  if ((int64_t)cu[n_seqs] >= (int64_t)1 << 31)
    return fail(SW_ERR_INVALID_ARG, "total tokens too large");
  m->tok_start[n_seqs] = cu[n_seqs];
  m->blk_start[n_seqs] = (int)blocks;
  m->mat_start[n_seqs] = mat;
  m->max_b = max_b;
  *nb = blocks;
  *nm = mat;
  return SW_OK;
}

int check_heads(int h_q, int h_kv) {
  if (h_q < 1 || h_kv < 1 || h_q % h_kv != 0)
    return fail(SW_ERR_INVALID_ARG, "h_q=%d must be a positive multiple of h_kv=%d", h_q, h_kv);
  if (h_q > 1024) return fail(SW_ERR_INVALID_ARG, "h_q=%d too large", h_q);
  return SW_OK;
}

int budget(int avail, int nf, int k, int pct) {
  int t = (k > 0) ? k : (avail * pct + 99) / 100;
  if (t < nf) t = nf;
  if (t > avail) t = avail;
  return t;
}

int max_count(const sw::SeqMeta& m, int k, int pct, uint32_t flags) {
  int best = 0;
  for (int s = 0; s < m.n_seqs; ++s) {
    const int b = m.blk_start[s + 1] - m.blk_start[s];
    for (int i = 0; i < b; ++i) {
      const int first = (flags & SW_FORCE_FIRST) ? 0 : -1;
      const int last = (flags & SW_FORCE_LAST) ? i : -1;
      const int nf = (first >= 0) + (last >= 0 && last != first);
      const int t = budget(i + 1, nf, k, pct);
      if (t > best) best = t;
    }
  }
  return best;
}

int check_budget_args(int k, int density_pct, uint32_t flags) {
  if (flags & ~(SW_FORCE_FIRST | SW_FORCE_LAST))
    return fail(SW_ERR_INVALID_ARG, "unknown flags 0x%x", flags);
  if (k <= 0 && (density_pct < 1 || density_pct > 100))
    return fail(SW_ERR_INVALID_ARG, "density_pct=%d outside [1, 100] (k=%d)", density_pct, k);
  return SW_OK;
}

int hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(SW_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

}  // namespace

extern "C" {

const char* sw_last_error(void) { return g_err.c_str(); }

int sw_abi_version(void) { return SW_ABI_VERSION; }

int sw_layout(int n_seqs, const int32_t* cu_seqlens, int B, int64_t* nb, int64_t* nm,
              int32_t* max_b) {
  sw::SeqMeta m;
  int64_t b = 0, mm = 0;
  CHECK(build_meta(n_seqs, cu_seqlens, B, &m, &b, &mm));
  if (nb) *nb = b;
  if (nm) *nm = mm;
  if (max_b) *max_b = m.max_b;
  return ok();
}

int64_t sw_sketch_workspace_bytes(int h_q, int h_kv, int d, int n_seqs, const int32_t* cu_seqlens,
                                  int B) {
  sw::SeqMeta m;
  int64_t nb = 0, nm = 0;
  if (build_meta(n_seqs, cu_seqlens, B, &m, &nb, &nm) != SW_OK) return -1;
  if (check_heads(h_q, h_kv) != SW_OK) return -1;
  if (!is_pow2(d) || d < 16 || d > 256) {
    fail(SW_ERR_INVALID_ARG, "d=%d must be a power of two in [16, 256]", d);
    return -1;
  }
  ok();
  return sw::sketch_workspace_bytes(h_q, h_kv, d, nb);
}

int sw_select_max_count(int n_seqs, const int32_t* cu_seqlens, int B, int k, int density_pct,
                        uint32_t flags, int32_t* kmax) {
  sw::SeqMeta m;
  int64_t nb = 0, nm = 0;
  CHECK(build_meta(n_seqs, cu_seqlens, B, &m, &nb, &nm));
  CHECK(check_budget_args(k, density_pct, flags));
  if (kmax == nullptr) return fail(SW_ERR_INVALID_ARG, "kmax is NULL");
  *kmax = max_count(m, k, density_pct, flags);
  return ok();
}

int sw_sketch_scores(int dtype, const void* Q, const void* K, int h_q, int h_kv, int d,
                     int n_seqs, const int32_t* cu_seqlens, int B, const int8_t* signs,
                     const int32_t* cols, int r, double* Qs, double* Ks, double* A,
                     double* A_scale, double* Qbar, double* Kbar, void* workspace,
                     int64_t workspace_bytes, void* stream) {
  if (dtype != SW_F32 && dtype != SW_BF16) return fail(SW_ERR_INVALID_ARG, "dtype=%d", dtype);
  CHECK(check_heads(h_q, h_kv));
  if (!is_pow2(d) || d < 16 || d > 256)
    return fail(SW_ERR_INVALID_ARG, "d=%d must be a power of two in [16, 256]", d);
  if (r < 1 || r > d) return fail(SW_ERR_INVALID_ARG, "r=%d outside [1, d=%d]", r, d);
  sw::SeqMeta m;
  int64_t nb = 0, nm = 0;
  CHECK(build_meta(n_seqs, cu_seqlens, B, &m, &nb, &nm));
  CHECK(check_ptr(Q, 16, "Q"));
  CHECK(check_ptr(K, 16, "K"));
  CHECK(check_ptr(signs, 1, "signs"));
  CHECK(check_ptr(cols, 4, "cols"));
  CHECK(check_ptr(Qs, 8, "Qs"));
  CHECK(check_ptr(Ks, 8, "Ks"));
  CHECK(check_ptr(A, 8, "A"));
  CHECK(check_ptr(A_scale, 8, "A_scale"));
  if (Qbar && !aligned(Qbar, 8)) return fail(SW_ERR_INVALID_ARG, "Qbar misaligned");
  if (Kbar && !aligned(Kbar, 8)) return fail(SW_ERR_INVALID_ARG, "Kbar misaligned");
  const int64_t need = sw::sketch_workspace_bytes(h_q, h_kv, d, nb);
  if (need > 0) CHECK(check_ptr(workspace, 256, "workspace"));
  if (workspace_bytes < need)
    return fail(SW_ERR_INVALID_ARG, "workspace_bytes=%lld < required %lld",
                (long long)workspace_bytes, (long long)need);
  hipError_t e = sw::launch_sketch(dtype, Q, K, h_q, h_kv, d, m, nb, (long long)cu_seqlens[n_seqs],
                                   signs, cols, r, Qs, Ks, A, A_scale, Qbar, Kbar, workspace,
                                   reinterpret_cast<hipStream_t>(stream));
  return hip_status(e, "sw_sketch_scores launch");
}

int64_t sw_walk_workspace_bytes(int variant, int n_seqs, const int32_t* cu_seqlens, int B) {
  if (variant < SW_WALK_POWER || variant > SW_WALK_MATPOW) return -1;
  sw::SeqMeta m;
  int64_t nb = 0, nm = 0;
  if (build_meta(n_seqs, cu_seqlens, B, &m, &nb, &nm) != SW_OK) return -1;
  return sw::walk_workspace_bytes(variant, nm);
}

int sw_walk_update_variant(int variant, const double* A, const double* A_scale, int s,
                           double logit_scale, int n_seqs, const int32_t* cu_seqlens, int B,
                           const double* R_prev, double* R_out, void* workspace,
                           int64_t workspace_bytes, void* stream) {
  if (variant < SW_WALK_POWER || variant > SW_WALK_MATPOW)
    return fail(SW_ERR_INVALID_ARG, "unknown walk variant %d", variant);
  if (s < 1 || s > 64) return fail(SW_ERR_INVALID_ARG, "s=%d outside [1, 64]", s);
  if (!isfinite(logit_scale)) return fail(SW_ERR_INVALID_ARG, "logit_scale is not finite");
  sw::SeqMeta m;
  int64_t nb = 0, nm = 0;
  CHECK(build_meta(n_seqs, cu_seqlens, B, &m, &nb, &nm));
  CHECK(check_ptr(A, 8, "A"));
  CHECK(check_ptr(A_scale, 8, "A_scale"));
  CHECK(check_ptr(R_out, 8, "R_out"));
  if (R_prev && !aligned(R_prev, 8)) return fail(SW_ERR_INVALID_ARG, "R_prev misaligned");
  if (R_out == R_prev || R_out == A) return fail(SW_ERR_INVALID_ARG, "R_out aliases an input");
  const int64_t need = sw::walk_workspace_bytes(variant, nm);
  if (need > 0) {
    CHECK(check_ptr(workspace, 8, "workspace"));
    if (workspace_bytes < need)
      return fail(SW_ERR_INVALID_ARG, "workspace_bytes=%lld < required %lld",
                  (long long)workspace_bytes, (long long)need);
  }
  hipError_t e = sw::launch_walk(variant, A, A_scale, s, logit_scale, m, nb, R_prev, R_out,
                                 static_cast<double*>(workspace),
                                 reinterpret_cast<hipStream_t>(stream));
  return hip_status(e, "sw_walk_update launch");
}

int sw_walk_update(const double* A, const double* A_scale, int s, int n_seqs,
                   const int32_t* cu_seqlens, int B, const double* R_prev, double* R_out,
                   void* stream) {
  return sw_walk_update_variant(SW_WALK_POWER, A, A_scale, s, 1.0, n_seqs, cu_seqlens, B, R_prev,
                                R_out, nullptr, 0, stream);
}

int sw_select_topk_blocks(const double* R, int n_seqs, const int32_t* cu_seqlens, int B, int k,
                          int density_pct, uint32_t flags, int32_t* idx, int32_t* cnt, int kmax,
                          void* stream) {
  sw::SeqMeta m;
  int64_t nb = 0, nm = 0;
  CHECK(build_meta(n_seqs, cu_seqlens, B, &m, &nb, &nm));
  CHECK(check_budget_args(k, density_pct, flags));
  CHECK(check_ptr(R, 8, "R"));
  CHECK(check_ptr(idx, 4, "idx"));
  CHECK(check_ptr(cnt, 4, "cnt"));
  const int need = max_count(m, k, density_pct, flags);
  if (kmax < need) return fail(SW_ERR_INVALID_ARG, "kmax=%d < largest budget %d", kmax, need);
  hipError_t e = sw::launch_select(R, m, nb, k, density_pct, flags, idx, cnt, kmax,
                                   reinterpret_cast<hipStream_t>(stream));
  return hip_status(e, "sw_select_topk_blocks launch");
}

int sw_sparse_attn_prefill(int dtype, const void* Q, const void* K, const void* V, int h_q,
                           int h_kv, int d, int n_seqs, const int32_t* cu_seqlens, int B,
                           const int32_t* idx, const int32_t* cnt, int kmax, float scale, void* O,
                           float* lse, void* stream) {
  if (dtype != SW_F32 && dtype != SW_BF16) return fail(SW_ERR_INVALID_ARG, "dtype=%d", dtype);
  CHECK(check_heads(h_q, h_kv));
  if (d != 64 && d != 128) return fail(SW_ERR_UNSUPPORTED, "attention head dim d=%d (64 or 128)", d);
  if (B != 64 && B != 128) return fail(SW_ERR_UNSUPPORTED, "attention block size B=%d (64 or 128)", B);
  sw::SeqMeta m;
  int64_t nb = 0, nm = 0;
  CHECK(build_meta(n_seqs, cu_seqlens, B, &m, &nb, &nm));
  CHECK(check_ptr(Q, 16, "Q"));
  CHECK(check_ptr(K, 16, "K"));
  CHECK(check_ptr(V, 16, "V"));
  CHECK(check_ptr(O, 16, "O"));
  CHECK(check_ptr(idx, 4, "idx"));
  CHECK(check_ptr(cnt, 4, "cnt"));
  if (lse && !aligned(lse, 4)) return fail(SW_ERR_INVALID_ARG, "lse misaligned");
  if (kmax < 1) return fail(SW_ERR_INVALID_ARG, "kmax=%d < 1", kmax);
  if (!(scale > 0.0f)) scale = 1.0f / sqrtf((float)d);
  hipError_t e = sw::launch_attn_prefill(dtype, Q, K, V, h_q, h_kv, d,
                                         (long long)cu_seqlens[n_seqs], m, nb, idx, cnt, kmax,
                                         scale, O, lse, reinterpret_cast<hipStream_t>(stream));
  return hip_status(e, "sw_sparse_attn_prefill launch");
}

// ---------------------------------------------------------------------------
// decode (Alg. 2)
// ---------------------------------------------------------------------------

static int check_decode_shape(int batch, int d, int r, int b_max, int B) {
  if (batch < 1 || batch > 65536) return fail(SW_ERR_INVALID_ARG, "batch=%d outside [1, 65536]", batch);
  if (!is_pow2(d) || d < 16 || d > 256)
    return fail(SW_ERR_INVALID_ARG, "d=%d must be a power of two in [16, 256]", d);
  if (r < 1 || r > d) return fail(SW_ERR_INVALID_ARG, "r=%d outside [1, d=%d]", r, d);
  if (b_max < 1 || b_max > SW_MAX_BLOCKS)
    return fail(SW_ERR_INVALID_ARG, "b_max=%d outside [1, %d]", b_max, SW_MAX_BLOCKS);
  if (B < 16 || B > 1024 || B % 16 != 0)
    return fail(SW_ERR_INVALID_ARG, "B=%d must be a multiple of 16 in [16, 1024]", B);
  return SW_OK;
}

static int max_count_decode(int b_max, int k, int pct, uint32_t flags) {
  int best = 0;
  for (int a = 1; a <= b_max; ++a) {
    const int first = (flags & SW_FORCE_FIRST) ? 0 : -1;
    const int last = (flags & SW_FORCE_LAST) ? a - 1 : -1;
    const int nf = (first >= 0) + (last >= 0 && last != first);
    const int t = budget(a, nf, k, pct);
    if (t > best) best = t;
  }
  return best;
}

int64_t sw_decode_state_bytes(int batch, int d, int r, int b_max) {
  if (check_decode_shape(batch, d, r, b_max, 64) != SW_OK) return -1;
  ok();
  return sw::decode_layout(batch, d, r, b_max).total;
}

int sw_decode_state_init(void* state, int batch, int d, int r, int b_max, int seq, int n, int B,
                         const double* Qs, const double* Ks, const double* A,
                         const double* A_scale, const double* Qbar, const double* Kbar,
                         void* stream) {
  CHECK(check_decode_shape(batch, d, r, b_max, B));
  if (seq < 0 || seq >= batch) return fail(SW_ERR_INVALID_ARG, "seq=%d outside [0, %d)", seq, batch);
  if (n < 1 || (n + B - 1) / B > b_max)
    return fail(SW_ERR_INVALID_ARG, "prompt length n=%d needs more than b_max=%d blocks", n, b_max);
  CHECK(check_ptr(state, 256, "state"));
  CHECK(check_ptr(Qs, 8, "Qs"));
  CHECK(check_ptr(Ks, 8, "Ks"));
  CHECK(check_ptr(A, 8, "A"));
  CHECK(check_ptr(A_scale, 8, "A_scale"));
  CHECK(check_ptr(Qbar, 8, "Qbar"));
  CHECK(check_ptr(Kbar, 8, "Kbar"));
  hipError_t e = sw::launch_decode_init(reinterpret_cast<char*>(state), batch, d, r, b_max, seq, n, B,
                                        Qs, Ks, A, A_scale, Qbar, Kbar,
                                        reinterpret_cast<hipStream_t>(stream));
  return hip_status(e, "sw_decode_state_init launch");
}

int sw_kv_append(int dtype, const void* k_new, const void* v_new, void* Kc, void* Vc, int batch,
                 int h_kv, int d, int T_max, const int32_t* pos, void* stream) {
  if (dtype != SW_F32 && dtype != SW_BF16) return fail(SW_ERR_INVALID_ARG, "dtype=%d", dtype);
  if (batch < 1 || h_kv < 1 || d < 1 || T_max < 1)
    return fail(SW_ERR_INVALID_ARG, "batch=%d h_kv=%d d=%d T_max=%d must be positive", batch, h_kv, d, T_max);
  CHECK(check_ptr(k_new, 4, "k_new"));
  CHECK(check_ptr(v_new, 4, "v_new"));
  CHECK(check_ptr(Kc, 4, "Kc"));
  CHECK(check_ptr(Vc, 4, "Vc"));
  CHECK(check_ptr(pos, 4, "pos"));
  hipError_t e = sw::launch_kv_append(dtype, k_new, v_new, Kc, Vc, batch, h_kv, d, T_max, pos,
                                      reinterpret_cast<hipStream_t>(stream));
  return hip_status(e, "sw_kv_append launch");
}

int sw_sketch_scores_decode(int dtype, const void* q_new, const void* k_new, int batch, int h_q,
                            int h_kv, int d, int B, const int32_t* pos, const int8_t* signs,
                            const int32_t* cols, int r, int b_max, void* state, void* stream) {
  if (dtype != SW_F32 && dtype != SW_BF16) return fail(SW_ERR_INVALID_ARG, "dtype=%d", dtype);
  CHECK(check_heads(h_q, h_kv));
  CHECK(check_decode_shape(batch, d, r, b_max, B));
  CHECK(check_ptr(q_new, 16, "q_new"));
  CHECK(check_ptr(k_new, 16, "k_new"));
  CHECK(check_ptr(pos, 4, "pos"));
  CHECK(check_ptr(signs, 1, "signs"));
  CHECK(check_ptr(cols, 4, "cols"));
  CHECK(check_ptr(state, 256, "state"));
  hipError_t e = sw::launch_decode_sketch(dtype, q_new, k_new, batch, h_q, h_kv, d, B, pos, signs,
                                          cols, r, b_max, reinterpret_cast<char*>(state),
                                          reinterpret_cast<hipStream_t>(stream));
  return hip_status(e, "sw_sketch_scores_decode launch");
}

int sw_walk_update_decode_variant(int variant, const void* state, int batch, int d, int r,
                                  int b_max, int B, const int32_t* pos, int s,
                                  const double* r_prev, double* r_out, void* stream) {
  if (variant == SW_WALK_SOFTMAX || variant == SW_WALK_MATPOW)
    return fail(SW_ERR_UNSUPPORTED, "walk variant %d is not available in decode", variant);
  if (variant != SW_WALK_POWER && variant != SW_WALK_RELU)
    return fail(SW_ERR_INVALID_ARG, "unknown walk variant %d", variant);
  if (s < 1 || s > 64) return fail(SW_ERR_INVALID_ARG, "s=%d outside [1, 64]", s);
  CHECK(check_decode_shape(batch, d, r, b_max, B));
  CHECK(check_ptr(state, 256, "state"));
  CHECK(check_ptr(pos, 4, "pos"));
  CHECK(check_ptr(r_out, 8, "r_out"));
  if (r_prev && !aligned(r_prev, 8)) return fail(SW_ERR_INVALID_ARG, "r_prev misaligned");
  if (r_prev == r_out) return fail(SW_ERR_INVALID_ARG, "r_out aliases r_prev");
  hipError_t e = sw::launch_decode_walk(static_cast<const char*>(state), batch, d, r, b_max, B,
                                        pos, s, variant == SW_WALK_RELU, r_prev, r_out,
                                        reinterpret_cast<hipStream_t>(stream));
  return hip_status(e, "sw_walk_update_decode launch");
}

int sw_walk_update_decode(const void* state, int batch, int d, int r, int b_max, int B,
                          const int32_t* pos, int s, const double* r_prev, double* r_out,
                          void* stream) {
  return sw_walk_update_decode_variant(SW_WALK_POWER, state, batch, d, r, b_max, B, pos, s, r_prev,
                                       r_out, stream);
}

int sw_select_max_count_decode(int b_max, int k, int density_pct, uint32_t flags, int32_t* kmax) {
  if (b_max < 1 || b_max > SW_MAX_BLOCKS)
    return fail(SW_ERR_INVALID_ARG, "b_max=%d outside [1, %d]", b_max, SW_MAX_BLOCKS);
  CHECK(check_budget_args(k, density_pct, flags));
  if (kmax == nullptr) return fail(SW_ERR_INVALID_ARG, "kmax is NULL");
  *kmax = max_count_decode(b_max, k, density_pct, flags);
  return ok();
}

int sw_select_topk_blocks_decode(const double* rows, int batch, int b_max, int B,
                                 const int32_t* pos, int k, int density_pct, uint32_t flags,
                                 int32_t* idx, int32_t* cnt, int kmax, void* stream) {
  CHECK(check_decode_shape(batch, 16, 1, b_max, B));
  CHECK(check_budget_args(k, density_pct, flags));
  CHECK(check_ptr(rows, 8, "rows"));
  CHECK(check_ptr(pos, 4, "pos"));
  CHECK(check_ptr(idx, 4, "idx"));
  CHECK(check_ptr(cnt, 4, "cnt"));
  const int need = max_count_decode(b_max, k, density_pct, flags);
  if (kmax < need) return fail(SW_ERR_INVALID_ARG, "kmax=%d < largest budget %d", kmax, need);
  hipError_t e = sw::launch_select_decode(rows, batch, b_max, B, pos, k, density_pct, flags, idx,
                                          cnt, kmax, reinterpret_cast<hipStream_t>(stream));
  return hip_status(e, "sw_select_topk_blocks_decode launch");
}

int64_t sw_decode_attn_workspace_bytes(int batch, int h_q, int h_kv, int d) {
  if (batch < 1 || h_kv < 1 || h_q < h_kv || d < 1) {
    fail(SW_ERR_INVALID_ARG, "batch=%d h_q=%d h_kv=%d d=%d", batch, h_q, h_kv, d);
    return -1;
  }
  ok();
  const int64_t S = sw::decode_attn_splits(batch, h_kv);
  return (int64_t)batch * h_q * S * (d + 2) * 4;
}

int sw_sparse_attn_decode(int dtype, const void* q, const void* Kc, const void* Vc, int batch,
                          int h_q, int h_kv, int d, int T_max, int B, const int32_t* pos,
                          const int32_t* idx, const int32_t* cnt, int kmax, float scale, void* O,
                          void* workspace, int64_t workspace_bytes, void* stream) {
  if (dtype != SW_F32 && dtype != SW_BF16) return fail(SW_ERR_INVALID_ARG, "dtype=%d", dtype);
  CHECK(check_heads(h_q, h_kv));
  const int G = h_q / h_kv;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return fail(SW_ERR_UNSUPPORTED, "decode attention needs h_q/h_kv in {1,2,4,8}, got %d", G);
  if (d != 64 && d != 128) return fail(SW_ERR_UNSUPPORTED, "decode attention head dim d=%d (64 or 128)", d);
  if (batch < 1 || batch > 65536) return fail(SW_ERR_INVALID_ARG, "batch=%d", batch);
  if (T_max < 1) return fail(SW_ERR_INVALID_ARG, "T_max=%d", T_max);
  // the kernels walk a selected block in 16-token groups
  if (B < 16 || B > 1024 || B % 16 != 0)
    return fail(SW_ERR_INVALID_ARG, "B=%d must be a multiple of 16 in [16, 1024]", B);
  if (kmax < 1) return fail(SW_ERR_INVALID_ARG, "kmax=%d < 1", kmax);
  CHECK(check_ptr(q, 16, "q"));
  CHECK(check_ptr(Kc, 16, "Kc"));
  CHECK(check_ptr(Vc, 16, "Vc"));
  CHECK(check_ptr(O, 4, "O"));
  CHECK(check_ptr(pos, 4, "pos"));
  CHECK(check_ptr(idx, 4, "idx"));
  CHECK(check_ptr(cnt, 4, "cnt"));
  const int64_t need = sw_decode_attn_workspace_bytes(batch, h_q, h_kv, d);
  CHECK(check_ptr(workspace, 256, "workspace"));
  if (workspace_bytes < need)
    return fail(SW_ERR_INVALID_ARG, "workspace_bytes=%lld < required %lld",
                (long long)workspace_bytes, (long long)need);
  if (!(scale > 0.0f)) scale = 1.0f / sqrtf((float)d);
  hipError_t e = sw::launch_attn_decode(dtype, q, Kc, Vc, batch, h_q, h_kv, d, T_max, B, pos, idx,
                                        cnt, kmax, scale, O, reinterpret_cast<float*>(workspace),
                                        reinterpret_cast<hipStream_t>(stream));
  return hip_status(e, "sw_sparse_attn_decode launch");
}

int sw_sparse_attn_decode_noalloc(int dtype, const void* q, const void* Kc, const void* Vc,
                                  int batch, int h_q, int h_kv, int d, int T_max, int B,
                                  const int32_t* pos, const int32_t* idx, const int32_t* cnt,
                                  int kmax, float scale, void* O, void* stream) {
  const int64_t need = sw_decode_attn_workspace_bytes(batch, h_q, h_kv, d);
  if (need < 0) return SW_ERR_INVALID_ARG;
  if (need > (int64_t)SW_NOALLOC_SCRATCH_BYTES)
    return fail(SW_ERR_INVALID_ARG,
                "batch=%d h_q=%d d=%d needs %lld bytes of split-K scratch, more than the %lld "
                "bytes the allocation-free entry point holds (use sw_sparse_attn_decode)",
                batch, h_q, d, (long long)need, (long long)SW_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  hipError_t e = sw::noalloc_scratch(&ws);
  if (e != hipSuccess) return hip_status(e, "sw_sparse_attn_decode_noalloc scratch lookup");
  return sw_sparse_attn_decode(dtype, q, Kc, Vc, batch, h_q, h_kv, d, T_max, B, pos, idx, cnt, kmax,
                               scale, O, ws, need, stream);
}

int64_t sw_decode_step_workspace_bytes(int batch, int h_q, int h_kv, int d) {
  return sw_decode_attn_workspace_bytes(batch, h_q, h_kv, d);
}

int sw_decode_step(int dtype, int layers, int batch, int h_q, int h_kv, int d, int r, int T_max,
                   int B, int b_max, const void* q_new, const void* k_new, const void* v_new,
                   void* Kc, void* Vc, void* state, const int32_t* pos, const int8_t* signs,
                   const int32_t* cols, int s, int walk_variant, int k, int density_pct,
                   uint32_t flags, int kmax, float scale, double* rows, int32_t* idx, int32_t* cnt,
                   void* O, void* workspace, int64_t workspace_bytes, void* stream) {
  if (dtype != SW_F32 && dtype != SW_BF16) return fail(SW_ERR_INVALID_ARG, "dtype=%d", dtype);
  if (layers < 1) return fail(SW_ERR_INVALID_ARG, "layers=%d < 1", layers);
  if (walk_variant == SW_WALK_SOFTMAX || walk_variant == SW_WALK_MATPOW)
    return fail(SW_ERR_UNSUPPORTED, "walk variant %d is not available in decode", walk_variant);
  if (walk_variant != SW_WALK_POWER && walk_variant != SW_WALK_RELU)
    return fail(SW_ERR_INVALID_ARG, "unknown walk variant %d", walk_variant);
  if (s < 1 || s > 64) return fail(SW_ERR_INVALID_ARG, "s=%d outside [1, 64]", s);
  CHECK(check_heads(h_q, h_kv));
  CHECK(check_decode_shape(batch, d, r, b_max, B));
  const int G = h_q / h_kv;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return fail(SW_ERR_UNSUPPORTED, "decode attention needs h_q/h_kv in {1,2,4,8}, got %d", G);
  if (d != 64 && d != 128) return fail(SW_ERR_UNSUPPORTED, "decode attention head dim d=%d (64 or 128)", d);
  if (T_max < 1 || (int64_t)b_max * B < T_max)
    return fail(SW_ERR_INVALID_ARG, "T_max=%d must be in [1, b_max * B = %lld]", T_max,
                (long long)b_max * B);
  CHECK(check_budget_args(k, density_pct, flags));
  const int need_k = max_count_decode(b_max, k, density_pct, flags);
  if (kmax < need_k) return fail(SW_ERR_INVALID_ARG, "kmax=%d < largest budget %d", kmax, need_k);
  CHECK(check_ptr(q_new, 16, "q_new"));
  CHECK(check_ptr(k_new, 16, "k_new"));
  CHECK(check_ptr(v_new, 16, "v_new"));
  CHECK(check_ptr(Kc, 16, "Kc"));
  CHECK(check_ptr(Vc, 16, "Vc"));
  CHECK(check_ptr(state, 256, "state"));
  CHECK(check_ptr(pos, 4, "pos"));
  CHECK(check_ptr(signs, 1, "signs"));
  CHECK(check_ptr(cols, 4, "cols"));
  CHECK(check_ptr(rows, 8, "rows"));
  CHECK(check_ptr(idx, 4, "idx"));
  CHECK(check_ptr(cnt, 4, "cnt"));
  CHECK(check_ptr(O, 16, "O"));
  const int64_t need = sw_decode_attn_workspace_bytes(batch, h_q, h_kv, d);
  CHECK(check_ptr(workspace, 256, "workspace"));
  if (workspace_bytes < need)
    return fail(SW_ERR_INVALID_ARG, "workspace_bytes=%lld < required %lld",
                (long long)workspace_bytes, (long long)need);
  if (!(scale > 0.0f)) scale = 1.0f / sqrtf((float)d);
  const size_t esz = dtype == SW_BF16 ? 2 : 4;
  const int64_t q_step = (int64_t)batch * h_q * d * esz;
  const int64_t kv_step = (int64_t)batch * h_kv * d * esz;
  const int64_t cache_step = (int64_t)batch * h_kv * T_max * d * esz;
  const int64_t state_step = sw::decode_layout(batch, d, r, b_max).total;
  const int64_t row_step = (int64_t)batch * b_max;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const char* qb = static_cast<const char*>(q_new);
  const char* kb = static_cast<const char*>(k_new);
  const char* vb = static_cast<const char*>(v_new);
  char* Kb = static_cast<char*>(Kc);
  char* Vb = static_cast<char*>(Vc);
  char* Sb = static_cast<char*>(state);
  char* Ob = static_cast<char*>(O);
  for (int l = 0; l < layers; ++l) {
    char* stl = Sb + l * state_step;
    void* Kl = Kb + l * cache_step;
    void* Vl = Vb + l * cache_step;
    double* rl = rows + l * row_step;
    int32_t* il = idx + (int64_t)l * batch * kmax;
    int32_t* cl = cnt + (int64_t)l * batch;
    hipError_t e = sw::launch_decode_layer(
        dtype, qb + l * q_step, kb + l * kv_step, vb + l * kv_step, Kl, Vl, T_max, batch, h_q,
        h_kv, d, B, pos, signs, cols, r, b_max, stl, s, walk_variant == SW_WALK_RELU,
        l == 0 ? nullptr : rl - row_step, rl, k, density_pct, flags, il, cl, kmax, st);
    if (e == hipSuccess)
      e = sw::launch_attn_decode(dtype, qb + l * q_step, Kl, Vl, batch, h_q, h_kv, d, T_max, B, pos,
                                 il, cl, kmax, scale, Ob + l * q_step,
                                 reinterpret_cast<float*>(workspace), st);
    if (e != hipSuccess) return hip_status(e, "sw_decode_step launch");
  }
  return ok();
}

}  // extern "C"
