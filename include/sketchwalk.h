/*
 * sketchwalk.h - C ABI of the MI355X (gfx950) Sketch&Walk attention library.
 *
 * Method: Le et al., "Scout Before You Attend: Sketch-and-Walk Sparse
 * Attention for Efficient LLM Inference". Each entry point below names the
 * passage of the paper that defines what it computes.
 *
 * Conventions shared by every call
 * --------------------------------
 * - Pointers are DEVICE pointers unless marked [host]. The caller owns every
 *   buffer; the library keeps no state between calls apart from a
 *   thread-local error string.
 * - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *   Work is enqueued asynchronously; results are ready when the stream is.
 * - Return value: SW_OK, or an error code with a message in
 *   sw_last_error(). Arguments are validated on the host before anything is
 *   enqueued; an invalid call enqueues nothing. SW_ERR_HIP reports a failed
 *   launch. Faults inside a kernel surface at the caller's next
 *   synchronisation.
 * - Tensor pointers must be 16-byte aligned and sizes in elements are given
 *   per argument. Element types: SW_F32 = float, SW_BF16 = bfloat16 stored as
 *   uint16.
 * - Sequences (prefill): `n_seqs` sequences are concatenated along the token
 *   axis; cu_seqlens [host, n_seqs+1] holds cumulative lengths (cu[0] = 0,
 *   every length >= 1, total N = cu[n_seqs]). Sequence s has
 *   b_s = ceil(n_s / B) blocks. Block rows are numbered globally: sequence s
 *   owns rows [bo_s, bo_s + b_s) with bo_s = sum_{t<s} b_t (nb = total).
 *   Per-sequence b_s x b_s matrices are stored row-major back to back,
 *   sequence s at element offset mo_s = sum_{t<s} b_t^2 (nm = total).
 * - Q is [h_q][N][d], K and V are [h_kv][N][d] (head-major, row-major,
 *   contiguous); h_q is a multiple of h_kv and query head u reads KV head
 *   u / (h_q / h_kv).
 * - Every output is deterministic: the same inputs give the same bits.
 */
#ifndef SKETCHWALK_H
#define SKETCHWALK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SW_ABI_VERSION 1

#define SW_OK 0
#define SW_ERR_INVALID_ARG 1
#define SW_ERR_UNSUPPORTED 2
#define SW_ERR_HIP 3

#define SW_F32 0
#define SW_BF16 1

/* Forced-block flags for selection (paper Sec. 4.1 keeps the first and the
   last key block of every query block). */
#define SW_FORCE_FIRST 1u
#define SW_FORCE_LAST 2u

/* Walk transitions (sw_walk_update_variant, sw_walk_update_decode_variant). */
#define SW_WALK_POWER 0   /* (A/c)^s element-wise: Alg. 1 step 6 */
#define SW_WALK_RELU 1    /* (max(A, 0)/c)^s element-wise */
#define SW_WALK_SOFTMAX 2 /* causal row softmax of logit_scale * A */
#define SW_WALK_MATPOW 3  /* (A/c)^s as a matrix power */

#define SW_MAX_SEQS 64          /* sequences per prefill call */
#define SW_MAX_BLOCKS 4096      /* blocks per sequence */

/* Message of the last failed call on this thread ("" if none). */
const char* sw_last_error(void);

/* SW_ABI_VERSION of the built library. */
int sw_abi_version(void);

/* Host-only layout query: nb (total block rows), nm (total matrix
   elements, sum of b_s^2) and the largest b_s. No GPU work. */
int sw_layout(int n_seqs, const int32_t* cu_seqlens /* [host] */, int B,
              int64_t* nb, int64_t* nm, int32_t* max_b);

/* Host-only: bytes of workspace sw_sketch_scores needs (>= 0), or -1 on
   invalid arguments. */
int64_t sw_sketch_workspace_bytes(int h_q, int h_kv, int d, int n_seqs,
                                  const int32_t* cu_seqlens /* [host] */, int B);

/* Host-only: the largest per-row budget tau_i a selection with these
   parameters produces (the minimum valid `kmax`). Budget rule: k > 0 gives
   tau_i = k, otherwise tau_i = ceil((i+1) * density_pct / 100) in integer
   arithmetic; then tau_i is clamped to [|F_i|, i+1], F_i the forced set. */
int sw_select_max_count(int n_seqs, const int32_t* cu_seqlens /* [host] */, int B,
                        int k, int density_pct, uint32_t flags, int32_t* kmax);

/*
 * sw_sketch_scores - Small-World Sketching of one layer: paper Alg. 1
 * steps 1-5 (Sec. 2.2; SRHT construction in the appendix lemma on the
 * Hadamard transform guarantee).
 *
 *   qbar_i = mean over the tokens of block i of the head-averaged queries
 *            (a partial last block averages the tokens it has); kbar likewise
 *            over the KV heads.
 *   Qs_i   = (1/sqrt(r)) * ((qbar_i * signs) H)[cols]   (H = +-1 Sylvester
 *            Walsh-Hadamard matrix, natural order); Ks likewise.
 *   A      = Qs Ks^T / sqrt(r) per sequence, with the entries whose key block
 *            follows the query block set to 0 (causal).
 *   A_scale[s] = max |A| over sequence s (0 when every score is 0; consumers
 *            then use 1).
 *
 * dtype: SW_F32 or SW_BF16 (Q, K). d: power of two in [16, 256]. B: block
 * size, multiple of 16, <= 1024. signs [d] int8 (+1/-1); cols [r] int32,
 * distinct, in [0, d) (device data: values are reduced modulo d, never
 * range-checked); 1 <= r <= d.
 * Outputs (float64): Qs, Ks [nb][r]; A [nm]; A_scale [n_seqs]; Qbar, Kbar
 * [nb][d] block means (optional, may be NULL).
 * workspace: >= sw_sketch_workspace_bytes(...) bytes, 256-byte aligned (the
 * current kernels need none: the query returns 0 and workspace may be NULL).
 */
int sw_sketch_scores(int dtype, const void* Q, const void* K, int h_q, int h_kv, int d,
                     int n_seqs, const int32_t* cu_seqlens /* [host] */, int B,
                     const int8_t* signs, const int32_t* cols, int r,
                     double* Qs, double* Ks, double* A, double* A_scale,
                     double* Qbar, double* Kbar,
                     void* workspace, int64_t workspace_bytes, void* stream);

/*
 * sw_walk_update - Sketch-Determined Walk: paper Sec. 2.3, Alg. 1 step 6,
 * appendix lemma on walk accumulation across layers.
 *
 *   W = (A / c)^s element-wise (c = A_scale[s], or 1 where it is 0);
 *   R_out = W if R_prev is NULL (first walked layer), else R_prev W;
 *   then every row of R_out is divided by its largest magnitude (rows of
 *   zeros stay zero). Both rescalings multiply rows by positive factors and
 *   leave every ranking unchanged.
 *
 * A [nm] float64 from sw_sketch_scores (lower triangular per sequence);
 * s: integer >= 1. R_prev, R_out [nm] float64; R_out must not alias R_prev
 * or A. Sequences are independent.
 */
int sw_walk_update(const double* A, const double* A_scale, int s,
                   int n_seqs, const int32_t* cu_seqlens /* [host] */, int B,
                   const double* R_prev, double* R_out, void* stream);

/*
 * sw_walk_update_variant - sw_walk_update with another transition in place
 * of the element-wise power (the walk step of Sec. 2.3 under the readings
 * that Sec. 1 / Fig. 2 and the appendix lemma on the walk's stationary
 * structure suggest):
 *   SW_WALK_POWER    W = (A/c)^s element-wise (identical to sw_walk_update);
 *   SW_WALK_RELU     W = (max(A, 0)/c)^s element-wise: negative scores give
 *                    zero weight instead of (-x)^s;
 *   SW_WALK_SOFTMAX  W[i][j] = exp(t A[i][j]) / sum_{j' <= i} exp(t A[i][j'])
 *                    for j <= i, 0 above the diagonal, t = logit_scale
 *                    (sqrt(r / d) rescales the sketched score to a block
 *                    attention logit); s is not used;
 *   SW_WALK_MATPOW   W = (A/c)^s as a matrix power (entry (i, j) sums the
 *                    score products along every s-hop block path), computed
 *                    by binary exponentiation in fp64.
 * Then R_out = W or R_prev W, rows divided by their largest magnitude, as in
 * sw_walk_update. Arguments as there, plus:
 * workspace: >= sw_walk_workspace_bytes(...) bytes of device memory, 8-byte
 * aligned (may be NULL when that is 0); its contents are scratch.
 * s in [1, 64] for every variant; logit_scale finite.
 */
int64_t sw_walk_workspace_bytes(int variant, int n_seqs, const int32_t* cu_seqlens /* [host] */,
                                int B);
int sw_walk_update_variant(int variant, const double* A, const double* A_scale, int s,
                           double logit_scale, int n_seqs, const int32_t* cu_seqlens /* [host] */,
                           int B, const double* R_prev, double* R_out, void* workspace,
                           int64_t workspace_bytes, void* stream);

/*
 * sw_select_topk_blocks - top-tau key blocks per query block: paper Alg. 1
 * step 7, first/last blocks kept as in Sec. 4.1.
 *
 * Row i of sequence s ranks key blocks 0..i (causal). F_i = {0 if
 * SW_FORCE_FIRST} U {i if SW_FORCE_LAST}; tau_i as in sw_select_max_count.
 * The row keeps F_i plus the tau_i - |F_i| best other blocks by (R value
 * descending, block index ascending).
 *
 * R [nm] float64. Outputs: idx [nb][kmax] int32 block indices ascending
 * (entries past cnt[row] are -1); cnt [nb] int32 = tau_i. kmax must be at
 * least sw_select_max_count(...). density_pct in [1, 100] (used when k <= 0).
 */
int sw_select_topk_blocks(const double* R, int n_seqs, const int32_t* cu_seqlens /* [host] */,
                          int B, int k, int density_pct, uint32_t flags,
                          int32_t* idx, int32_t* cnt, int kmax, void* stream);

/*
 * sw_sparse_attn_prefill - block-sparse causal attention on the original
 * per-head Q, K, V over the selected blocks: paper Alg. 1 step 8.
 *
 * For query head u at token p of block i (sequence s), with g = u / G:
 *   O[u][p] = sum_t softmax_t(scale * Q[u][p] . K[g][t]) V[g][t]
 * over the tokens t <= p of the blocks idx[row][0..cnt[row]) (softmax
 * renormalised over those keys only). scale <= 0 selects 1/sqrt(d).
 *
 * dtype SW_BF16 or SW_F32; d in {64, 128}; B in {64, 128} (other values
 * return SW_ERR_UNSUPPORTED). O [h_q][N][d] in the input dtype. lse [h_q][N] float32
 * natural-log sum-exp of the scaled logits (optional, may be NULL).
 * idx/cnt as written by sw_select_topk_blocks (block indices ascending,
 * each <= its row's block index; entries outside [0, i] are skipped and
 * cnt is clamped to kmax, so malformed selections cannot read out of
 * bounds).
 */
int sw_sparse_attn_prefill(int dtype, const void* Q, const void* K, const void* V,
                           int h_q, int h_kv, int d,
                           int n_seqs, const int32_t* cu_seqlens /* [host] */, int B,
                           const int32_t* idx, const int32_t* cnt, int kmax, float scale,
                           void* O, float* lse, void* stream);

/* ======================================================================
 * Decode (paper Alg. 2): one new token per sequence per layer.
 *
 * Per-layer decode state: one caller-owned device buffer of
 * sw_decode_state_bytes(batch, d, r, b_max) bytes (256-byte aligned), laid
 * out as consecutive 256-byte-aligned sections
 *   double A_scale[batch]         score scale c (frozen at its prefill value)
 *   int32  col0[batch]            first key block whose column decode fills
 *                                 (= prompt length / B)
 *   int32  cnt[batch][2][2]       token counts of the open query / key block,
 *                                 two copies: the step at position p reads
 *                                 copy (p + 1) % 2 and writes copy p % 2
 *   double bar[batch][2][2][d]    running means of the open query / key block,
 *                                 two copies as for cnt
 *   double qt[batch][r]           sketch of the latest token's query
 *   double Qs[batch][b_max][r]    sketch of every query-block representative
 *   double Ks[batch][b_max][r]    sketch of every key-block representative
 *   float  rowc[batch][b_max], colc[batch][b_max]  the open block's score
 *                                 row and column as the last step wrote them
 *   float  A[batch][lda/32][b_max][32]  block-score cache (fp32) in strips
 *                                 of 32 columns: score (m, j) of a sequence
 *                                 at float offset ((j/32) b_max + m) 32 + j%32,
 *                                 lda = b_max rounded up to a multiple of 32
 * Checkpointing a decode is a byte copy of this buffer (plus the caches)
 * taken between calls.
 * pos [batch] int32 (device): 0-based position of the new token of each
 * sequence; b_cur = pos / B is the open block. Sequences whose pos is
 * negative, >= T_max (attention, append) or beyond b_max blocks are skipped:
 * their state, cache entries, walk rows and selections are left untouched,
 * and sw_sparse_attn_decode writes zeros as their attention output.
 * ====================================================================== */

/* Host-only: bytes of one layer's decode state (-1 on invalid arguments). */
int64_t sw_decode_state_bytes(int batch, int d, int r, int b_max);

/* Fills sequence `seq` of a layer's decode state from the prefill sketch of
   its n-token prompt (one sequence's outputs of sw_sketch_scores: Qs, Ks
   [b][r], A [b][b], A_scale [1], Qbar, Kbar [b][d], b = ceil(n/B) <= b_max).
   The open block is the prompt's last block (with its token count); the
   score cache is zero outside the prompt's b x b corner. Alg. 2 inputs: the
   cached block reps and block-score estimate from prefill. */
int sw_decode_state_init(void* state, int batch, int d, int r, int b_max, int seq, int n, int B,
                         const double* Qs, const double* Ks, const double* A,
                         const double* A_scale, const double* Qbar, const double* Kbar,
                         void* stream);

/* Alg. 2 step 1: writes k_new, v_new [batch][h_kv][d] into the caches
   Kc, Vc [batch][h_kv][T_max][d] at token pos[b]. */
int sw_kv_append(int dtype, const void* k_new, const void* v_new, void* Kc, void* Vc, int batch,
                 int h_kv, int d, int T_max, const int32_t* pos, void* stream);

/*
 * sw_sketch_scores_decode - Alg. 2 steps 2-4 for the tokens q_new
 * [batch][h_q][d], k_new [batch][h_kv][d] at pos[b]:
 *   - running mean of the head-averaged key (and query) of the open block
 *     (restarted when pos % B == 0);
 *   - q~_t = SRHT(head-averaged query), and the sketches of both open
 *     representatives (stored in Qs[b_cur], Ks[b_cur]);
 *   - (i) new query row A[b_cur][j] = q~_t . Ks[j] / sqrt(r), j < b_cur;
 *     (ii) last column A[m][b_cur] = Qs[m] . Ks[b_cur] / sqrt(r), m <= b_cur
 *     (the diagonal entry comes from (ii)).
 * signs/cols/r as in sw_sketch_scores (same transform as the prompt).
 * q_new and k_new must be 16-byte aligned (SW_ERR_INVALID_ARG otherwise).
 */
int sw_sketch_scores_decode(int dtype, const void* q_new, const void* k_new, int batch, int h_q,
                            int h_kv, int d, int B, const int32_t* pos, const int8_t* signs,
                            const int32_t* cols, int r, int b_max, void* state, void* stream);

/*
 * sw_walk_update_decode - Alg. 2 step 5 on the current query row:
 *   r_out = W[b_cur, :] if r_prev is NULL (first walked layer), else
 *   r_prev W, with W = (A / c)^s element-wise over the layer's score cache;
 *   then divided by its largest magnitude. r_prev, r_out [batch][b_max]
 *   float64 (entries past b_cur are written as 0; r_out must not alias
 *   r_prev). Sums run in fp64 in a fixed order.
 */
int sw_walk_update_decode(const void* state, int batch, int d, int r, int b_max, int B,
                          const int32_t* pos, int s, const double* r_prev, double* r_out,
                          void* stream);

/*
 * sw_walk_update_decode_variant - sw_walk_update_decode with the transition
 * chosen as in sw_walk_update_variant. SW_WALK_POWER and SW_WALK_RELU only:
 * the other two need the whole weight matrix of every layer at every step
 * (softmax normalizers of rows whose last column decode rewrites, or s
 * matrix products) and return SW_ERR_UNSUPPORTED.
 */
int sw_walk_update_decode_variant(int variant, const void* state, int batch, int d, int r,
                                  int b_max, int B, const int32_t* pos, int s,
                                  const double* r_prev, double* r_out, void* stream);

/* Host-only: the largest decode budget over rows of up to b_max blocks. */
int sw_select_max_count_decode(int b_max, int k, int density_pct, uint32_t flags, int32_t* kmax);

/*
 * sw_select_topk_blocks_decode - Alg. 2 step 6: per sequence, key blocks
 * 0..b_cur ranked by the walk row rows[b] (from sw_walk_update_decode); the
 * forced set is {0 (SW_FORCE_FIRST), b_cur (SW_FORCE_LAST)} and counts
 * inside tau = ceil((b_cur+1) density_pct / 100) (or k). idx [batch][kmax]
 * ascending, -1 padded; cnt [batch].
 */
int sw_select_topk_blocks_decode(const double* rows, int batch, int b_max, int B,
                                 const int32_t* pos, int k, int density_pct, uint32_t flags,
                                 int32_t* idx, int32_t* cnt, int kmax, void* stream);

/* Host-only: workspace bytes of sw_sparse_attn_decode (-1 on bad input). */
int64_t sw_decode_attn_workspace_bytes(int batch, int h_q, int h_kv, int d);

/*
 * sw_sparse_attn_decode - Alg. 2 step 7: for each sequence b and query head
 * u (g = u / G), softmax(scale q[b][u] . Kc[b][g][t]) over the tokens
 * t <= pos[b] of the selected blocks, applied to Vc. Split-K over the
 * selected tokens with a log-sum-exp merge. q [batch][h_q][d]; Kc, Vc
 * [batch][h_kv][T_max][d]; O [batch][h_q][d] in the input dtype.
 * G = h_q / h_kv in {1, 2, 4, 8}; d in {64, 128}; B a multiple of 16 in
 * [16, 1024] (SW_ERR_INVALID_ARG otherwise); scale <= 0 -> 1/sqrt(d).
 */
int sw_sparse_attn_decode(int dtype, const void* q, const void* Kc, const void* Vc, int batch,
                          int h_q, int h_kv, int d, int T_max, int B, const int32_t* pos,
                          const int32_t* idx, const int32_t* cnt, int kmax, float scale, void* O,
                          void* workspace, int64_t workspace_bytes, void* stream);

/*
 * sw_sparse_attn_decode_noalloc - sw_sparse_attn_decode for callers that
 * cannot allocate device memory (code under HIP graph capture, serving loops
 * that forbid allocation): the same kernels and results, with the split-K
 * partials in a fixed device array of SW_NOALLOC_SCRATCH_BYTES that the
 * library holds on each GPU it runs on until the process ends, instead of a
 * caller workspace. The call allocates nothing. A call whose partials need
 * more than SW_NOALLOC_SCRATCH_BYTES (sw_decode_attn_workspace_bytes) returns
 * SW_ERR_INVALID_ARG. Every call on one GPU shares that GPU's array: calls
 * that overlap on one GPU (different streams or threads) race; calls in
 * stream order do not. The array needs no clearing: each call writes every
 * partial it reads. The first call on a device looks the array's address up
 * once. Other arguments as in sw_sparse_attn_decode.
 */
#define SW_NOALLOC_SCRATCH_BYTES (8 * 1024 * 1024)
int sw_sparse_attn_decode_noalloc(int dtype, const void* q, const void* Kc, const void* Vc,
                                  int batch, int h_q, int h_kv, int d, int T_max, int B,
                                  const int32_t* pos, const int32_t* idx, const int32_t* cnt,
                                  int kmax, float scale, void* O, void* stream);

/*
 * sw_decode_step - one decode step of every layer in one call: Alg. 2 steps
 * 1-7 for layer 0, 1, ..., layers-1 in order (the walk row of layer l starts
 * from that of layer l-1; layer 0 is the first walked layer). Per layer it
 * enqueues the same arithmetic as sw_kv_append + sw_sketch_scores_decode +
 * sw_walk_update_decode_variant + sw_select_topk_blocks_decode +
 * sw_sparse_attn_decode, with the KV append, the score updates and the walk
 * over the score entries the step leaves unchanged in one launch, and the
 * open block's walk terms and the normalisation in the selection's launch
 * (4 kernel launches per layer instead of 7); results are bit-identical to
 * those calls.
 *
 * Layer-stacked, contiguous buffers (device):
 *   q_new [layers][batch][h_q][d], k_new, v_new [layers][batch][h_kv][d]
 *   (input dtype, 16-byte aligned); Kc, Vc [layers][batch][h_kv][T_max][d]
 *   (updated at pos); state [layers][sw_decode_state_bytes(batch, d, r,
 *   b_max)] (updated); rows [layers][batch][b_max] float64 walk rows (out);
 *   idx [layers][batch][kmax], cnt [layers][batch] selections (out); O
 *   [layers][batch][h_q][d] attention outputs (out, input dtype).
 * T_max <= b_max * B; walk_variant SW_WALK_POWER or SW_WALK_RELU; other
 * arguments as in the per-layer calls. workspace: >=
 * sw_decode_step_workspace_bytes(...) bytes, 256-byte aligned, reused by
 * every layer in stream order. The call only enqueues work on `stream`; it
 * may be captured into a HIP graph.
 */
int64_t sw_decode_step_workspace_bytes(int batch, int h_q, int h_kv, int d);
int sw_decode_step(int dtype, int layers, int batch, int h_q, int h_kv, int d, int r, int T_max,
                   int B, int b_max, const void* q_new, const void* k_new, const void* v_new,
                   void* Kc, void* Vc, void* state, const int32_t* pos, const int8_t* signs,
                   const int32_t* cols, int s, int walk_variant, int k, int density_pct,
                   uint32_t flags, int kmax, float scale, double* rows, int32_t* idx, int32_t* cnt,
                   void* O, void* workspace, int64_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SKETCHWALK_H */
