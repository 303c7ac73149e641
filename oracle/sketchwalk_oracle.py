"""Plain fp64 CPU oracle for the Sketch&Walk attention hot path.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or
execute this module: only the tests, the smoke check and the benchmark's CPU
baseline leg use it. It shares no code with the GPU library and reads only
numpy arrays (inputs converted exactly to float64: bf16 and fp32 values are
representable).

Everything is written for legibility, not speed: one function per step of the
method, in the paper's order and notation, with numpy matmul as the only
library primitive. Paper references (Le et al., "Scout Before You Attend:
Sketch-and-Walk Sparse Attention for Efficient LLM Inference"):

  Def. Block Attention Score (Sec. 2.1)           -> block_score_true
  Alg. 1 step 1 (head averaging)                  -> head_mean
  Sec. 2.2 token-space sketch, Alg. 1 steps 2-3   -> block_means
  Sec. 2.2 feature-space sketch, Alg. 1 step 4,
    SRHT construction (appendix lemma on the
    Hadamard transform guarantee, step 1)         -> sylvester_hadamard, srht
  Sec. 2.2 estimate, Alg. 1 step 5                -> block_scores
  Sec. 2.3 walk, Alg. 1 step 6, lemma on walk
    accumulation across layers                    -> walk_weights, walk_step
  walk transition variants (Sec. 1 and Fig. 2;
    appendix lemma on stationary structure)       -> walk_weights_variant
  Alg. 1 step 7, Sec. 4.1 implementation details  -> row_budget, select_row,
                                                     select_blocks
  Alg. 1 step 8 (gather + softmax per head)       -> sparse_attention_prefill
  Alg. 2 (decode, steps 2-7)                      -> DecodeLayerState,
                                                     decode_layer_step,
                                                     decode_attention

Readings where the paper is silent or inconsistent (each is listed in the
design notes of the repository):

* SRHT scale: the Walsh-Hadamard factor is taken orthonormal, so
  H_d = (1/sqrt(r)) D W_syl S with W_syl the +-1 Sylvester matrix. Then the
  sketched inner product is an unbiased estimate of the block-mean inner
  product, and at r = d it is exact.
* Causality: block scores above the diagonal (key block after query block)
  are zero in prefill, so the walk state stays lower triangular.
* Walk power: element-wise integer power s >= 1, as Alg. 1 step 6 states.
  Three other transitions are kept as variants (walk_weights_variant): the
  power applied after clipping negative scores to zero; a causal row softmax
  (the transition matrix of the appendix lemma on the walk's stationary
  structure, with the sketched score rescaled to a block attention logit);
  and the matrix power that the introduction's multi-hop walk describes.
* Range: W is formed from A/c with c = max |A| of the layer, and every walk
  row is divided by its largest magnitude. Both rescale by positive factors
  and leave every row's ranking unchanged.
* Budget: tau_i = ceil((i+1) * pct / 100) in integer arithmetic, clamped to
  [|F_i|, i+1], where F_i is the forced set (first block and the query's own
  block). Forced blocks count inside tau_i and are not ranked.
* Ties: ordering is (score descending, block index ascending).
* Sparse attention: token-level causal mask inside the diagonal block, scale
  1/sqrt(d), softmax over the selected keys only, GQA head map g = u // G.
* Decode: a running mean is kept for the current query block as for the key
  block; Alg. 2 step 4 writes the new query row, then the whole last column
  (rows 0..b_q, overwriting the diagonal entry); the score scale c of each
  layer stays at its prefill value; the current block is forced and counts
  inside tau.
"""

from __future__ import annotations

import dataclasses
import functools
import math
from typing import List, Optional, Sequence, Tuple

import numpy as np

FORCE_FIRST = 1
FORCE_LAST = 2
FORCE_BOTH = FORCE_FIRST | FORCE_LAST


def f64(x) -> np.ndarray:
    """Exact conversion of an input array (numpy or torch, any float dtype)
    to float64."""
    if hasattr(x, "detach"):
        x = x.detach().to("cpu")
        import torch  # local: only needed when handed torch tensors
        x = x.to(torch.float64).numpy()
    return np.asarray(x, dtype=np.float64)


# ---------------------------------------------------------------------------
# Sec. 2.1: the quantity the sketch estimates
# ---------------------------------------------------------------------------

def block_score_true(Qa: np.ndarray, Ka: np.ndarray, B: int, i: int, j: int) -> float:
    """Def. Block Attention Score (Sec. 2.1): the mean of the B*B token dot
    products between query block i and key block j, divided by sqrt(d).
    Written as the literal double sum over token pairs."""
    d = Qa.shape[1]
    qi = Qa[i * B:(i + 1) * B]
    kj = Ka[j * B:(j + 1) * B]
    total = 0.0
    for s in range(qi.shape[0]):
        for t in range(kj.shape[0]):
            total += float(np.dot(qi[s], kj[t]))
    return total / (qi.shape[0] * kj.shape[0]) / math.sqrt(d)


# ---------------------------------------------------------------------------
# Small-World Sketching (Sec. 2.2, Alg. 1 steps 1-5)
# ---------------------------------------------------------------------------

def head_mean(X) -> np.ndarray:
    """Alg. 1 step 1: average over heads. X [h][n][d] -> [n][d].
    Under GQA the query average runs over the h_q query heads and the key
    average over the h_kv KV heads (each KV head stands for G query heads, so
    this equals the average over the expanded key heads)."""
    h, n, d = X.shape
    out = np.empty((n, d), dtype=np.float64)
    for a in range(0, n, 4096):          # token chunks (each token's sum is independent)
        out[a:a + 4096] = f64(X[:, a:a + 4096]).sum(axis=0) / h
    return out


def block_means(Xa: np.ndarray, B: int) -> np.ndarray:
    """Token-space sketch (Sec. 2.2; Alg. 1 steps 2-3): the mean of each
    block of B consecutive tokens. A partial last block is averaged over the
    tokens it holds. [n][d] -> [b][d], b = ceil(n / B)."""
    n, d = Xa.shape
    b = -(-n // B)
    out = np.zeros((b, d), dtype=np.float64)
    for i in range(b):
        seg = Xa[i * B:min(n, (i + 1) * B)]
        out[i] = seg.sum(axis=0) / seg.shape[0]
    return out


@functools.lru_cache(maxsize=None)
def sylvester_hadamard(d: int) -> np.ndarray:
    """The d x d Walsh-Hadamard matrix in natural (Sylvester) order:
    entry (a, m) is (-1) ** popcount(a & m). d must be a power of two.
    (Cached; the returned array is read-only.)"""
    if d < 1 or (d & (d - 1)) != 0:
        raise ValueError("d must be a power of two")
    H = np.empty((d, d), dtype=np.float64)
    for a in range(d):
        for m in range(d):
            H[a, m] = -1.0 if bin(a & m).count("1") % 2 else 1.0
    H.setflags(write=False)
    return H


def srht(Xbar: np.ndarray, signs, cols) -> np.ndarray:
    """Feature-space sketch (Sec. 2.2; Alg. 1 step 4): X~ = Xbar H_d with the
    subsampled randomized Hadamard transform H_d = sqrt(d/r) D W S (appendix,
    SRHT construction), W orthonormal (= W_syl / sqrt(d)), D = diag(signs),
    S = the r sampled columns ``cols``. [b][d] -> [b][r]."""
    signs = np.asarray(signs, dtype=np.float64)
    cols = np.asarray(cols, dtype=np.int64)
    d = Xbar.shape[1]
    r = cols.shape[0]
    W = sylvester_hadamard(d) / math.sqrt(d)
    DWS = (signs[:, None] * W)[:, cols]          # D W S, d x r
    return math.sqrt(d / r) * (Xbar @ DWS)


def block_scores(Qs: np.ndarray, Ks: np.ndarray, causal: bool = True) -> np.ndarray:
    """Sketched block attention (Sec. 2.2; Alg. 1 step 5):
    A = Q~ K~^T / sqrt(r). With ``causal`` the entries whose key block comes
    after the query block are zero."""
    r = Qs.shape[1]
    A = (Qs @ Ks.T) / math.sqrt(r)
    if causal:
        A = np.tril(A)
    return A


def score_scale(A: np.ndarray) -> float:
    """Largest |A| entry of one layer's score matrix (1 if all are zero).
    Dividing A by it before the power only multiplies W by the global
    factor c**-s, which no ranking sees."""
    c = float(np.max(np.abs(A))) if A.size else 0.0
    return c if c > 0.0 else 1.0


def sketch_scores(Q, K, B: int, signs, cols) -> dict:
    """Alg. 1 steps 1-5 for one sequence of one layer.
    Q [h_q][n][d], K [h_kv][n][d]. Returns block means, sketches, the causal
    score matrix and its scale."""
    Qa = head_mean(Q)
    Ka = head_mean(K)
    qbar = block_means(Qa, B)
    kbar = block_means(Ka, B)
    Qs = srht(qbar, signs, cols)
    Ks = srht(kbar, signs, cols)
    A = block_scores(Qs, Ks, causal=True)
    return dict(qbar=qbar, kbar=kbar, Qs=Qs, Ks=Ks, A=A, c=score_scale(A))


# ---------------------------------------------------------------------------
# Sketch-Determined Walk (Sec. 2.3; Alg. 1 step 6)
# ---------------------------------------------------------------------------

def walk_weights(A: np.ndarray, c: float, s: int) -> np.ndarray:
    """W = (A / c) raised element-wise to the integer power s (Alg. 1 step 6
    calls it element-wise exponentiation), by repeated multiplication."""
    if int(s) != s or s < 1:
        raise ValueError("s must be an integer >= 1")
    X = A / c
    W = X.copy()
    for _ in range(int(s) - 1):
        W = W * X
    return W


def normalize_rows(R: np.ndarray) -> np.ndarray:
    """Divide every row by its largest magnitude (rows of zeros stay zero).
    Row i of R_k is linear in row i of R_{k-1}, so this changes no ranking."""
    R = R.copy()
    for i in range(R.shape[0]):
        m = float(np.max(np.abs(R[i]))) if R.shape[1] else 0.0
        if m > 0.0:
            R[i] = R[i] / m
    return R


def walk_step(R_prev: Optional[np.ndarray], W: np.ndarray, normalize: bool = True) -> np.ndarray:
    """Walk state update (Sec. 2.3; Alg. 1 step 6; lemma on walk
    accumulation across layers): R = W at the first walked layer, otherwise
    the matrix product R_prev W."""
    R = W.copy() if R_prev is None else R_prev @ W
    return normalize_rows(R) if normalize else R


# ---------------------------------------------------------------------------
# Walk transition variants (readings of the walk step, see module header)
# ---------------------------------------------------------------------------

WALK_POWER = 0     # (A/c)^s element-wise: Alg. 1 step 6 as printed
WALK_RELU = 1      # (max(A, 0)/c)^s element-wise
WALK_SOFTMAX = 2   # causal row softmax of logit_scale * A (appendix lemma on
                   # the walk's stationary structure, step 1)
WALK_MATPOW = 3    # (A/c)^s as a matrix power: the s-hop walk inside one
                   # layer that Sec. 1 and Fig. 2 describe


def walk_weights_relu(A: np.ndarray, c: float, s: int) -> np.ndarray:
    """Negative block scores clipped to zero before the element-wise power, so
    that under even s a strongly negative score does not gain weight."""
    return walk_weights(np.maximum(A, 0.0), c, s)


def walk_weights_softmax(A: np.ndarray, logit_scale: float) -> np.ndarray:
    """Row-stochastic transition matrix: row i is the softmax over the causal
    key blocks j <= i of logit_scale * A[i, j]; entries above the diagonal are
    zero. logit_scale = sqrt(r / d) turns the sketched score (which estimates
    the block-mean inner product divided by sqrt(r)) into the block's mean
    attention logit."""
    b = A.shape[0]
    W = np.zeros_like(A, dtype=np.float64)
    for i in range(b):
        z = logit_scale * A[i, :i + 1]
        e = np.exp(z - np.max(z))
        W[i, :i + 1] = e / e.sum()
    return W


def walk_weights_matpow(A: np.ndarray, c: float, s: int) -> np.ndarray:
    """The s-th matrix power of A/c, by s - 1 successive products: entry
    (i, j) sums the products of scores along every s-hop block path from i
    to j."""
    if int(s) != s or s < 1:
        raise ValueError("s must be an integer >= 1")
    X = A / c
    W = X.copy()
    for _ in range(int(s) - 1):
        W = W @ X
    return W


def walk_weights_variant(variant: int, A: np.ndarray, c: float, s: int,
                         logit_scale: float = 1.0) -> np.ndarray:
    """W of one layer under the chosen transition (WALK_* constants)."""
    if variant == WALK_POWER:
        return walk_weights(A, c, s)
    if variant == WALK_RELU:
        return walk_weights_relu(A, c, s)
    if variant == WALK_SOFTMAX:
        return walk_weights_softmax(A, logit_scale)
    if variant == WALK_MATPOW:
        return walk_weights_matpow(A, c, s)
    raise ValueError(f"unknown walk variant {variant}")


# ---------------------------------------------------------------------------
# Top-tau selection (Alg. 1 step 7; Sec. 4.1 implementation details)
# ---------------------------------------------------------------------------

def forced_set(i: int, flags: int) -> List[int]:
    """Blocks always kept for query block i: the first key block and the
    last causal key block (block i itself)."""
    F = set()
    if flags & FORCE_FIRST:
        F.add(0)
    if flags & FORCE_LAST:
        F.add(i)
    return sorted(F)


def row_budget(avail: int, n_forced: int, pct: int = 0, k: int = 0) -> int:
    """Blocks kept in a row with ``avail`` causal key blocks: k when k > 0,
    else ceil(avail * pct / 100) computed in integers; clamped to
    [n_forced, avail]."""
    if k > 0:
        t = k
    else:
        t = (avail * pct + 99) // 100
    return min(max(t, n_forced), avail)


def select_row(values: np.ndarray, avail: int, forced: Sequence[int], tau: int):
    """Top-tau indices of one walk row over key blocks 0..avail-1: the forced
    blocks plus the best (tau - |F|) others by (value descending, index
    ascending); returned ascending. Also returns the relative gap between the
    last kept and the first dropped ranked value (inf when no boundary)."""
    fset = set(forced)
    cand = [j for j in range(avail) if j not in fset]
    order = sorted(cand, key=lambda j: (-float(values[j]), j))
    m = tau - len(fset)
    chosen = sorted(fset | set(order[:m]))
    if 0 < m < len(order):
        vk = float(values[order[m - 1]])
        vn = float(values[order[m]])
        gap = (vk - vn) / abs(vk) if vk != 0.0 else (0.0 if vn == vk else math.inf)
    else:
        gap = math.inf
    return chosen, gap


def select_blocks(R: np.ndarray, pct: int = 0, k: int = 0, flags: int = FORCE_BOTH):
    """Alg. 1 step 7 for every query block of one sequence (causal: row i
    ranks key blocks 0..i). Returns (list of index lists, gaps array)."""
    b = R.shape[0]
    sel, gaps = [], np.zeros(b)
    for i in range(b):
        F = forced_set(i, flags)
        tau = row_budget(i + 1, len(F), pct=pct, k=k)
        chosen, gap = select_row(R[i], i + 1, F, tau)
        sel.append(chosen)
        gaps[i] = gap
    return sel, gaps


# ---------------------------------------------------------------------------
# Block-sparse attention (Alg. 1 step 8)
# ---------------------------------------------------------------------------

def _softmax_rows(logits: np.ndarray) -> np.ndarray:
    m = np.max(logits, axis=1, keepdims=True)
    e = np.exp(logits - m)
    return e / e.sum(axis=1, keepdims=True)


def sparse_attention_block(Q, K, V, B: int, sel_i: Sequence[int], u: int, i: int,
                           scale: Optional[float] = None) -> np.ndarray:
    """Output rows of query block i for query head u (Alg. 1 step 8): gather
    the selected key/value blocks of KV head g = u // G, softmax over the
    gathered keys at or before each query position, weight the values.
    Q [h_q][n][d], K/V [h_kv][n][d] (float64). Returns [rows][d]."""
    h_q, n, d = Q.shape
    G = h_q // K.shape[0]
    g = u // G
    sc = (1.0 / math.sqrt(d)) if scale is None else scale
    rows = np.arange(i * B, min(n, (i + 1) * B))
    toks = np.concatenate([np.arange(j * B, min(n, (j + 1) * B)) for j in sorted(sel_i)])
    logits = (Q[u, rows] @ K[g, toks].T) * sc
    logits = np.where(toks[None, :] <= rows[:, None], logits, -np.inf)
    P = _softmax_rows(logits)
    return P @ V[g, toks]


def sparse_attention_prefill(Q, K, V, B: int, sel: Sequence[Sequence[int]],
                             scale: Optional[float] = None) -> np.ndarray:
    """Alg. 1 step 8 over every head and query block of one sequence."""
    Q, K, V = f64(Q), f64(K), f64(V)
    h_q, n, d = Q.shape
    O = np.zeros((h_q, n, d))
    for u in range(h_q):
        for i in range(len(sel)):
            O[u, i * B:min(n, (i + 1) * B)] = sparse_attention_block(Q, K, V, B, sel[i], u, i, scale)
    return O


def dense_causal_attention(Q, K, V, scale: Optional[float] = None) -> np.ndarray:
    """Ordinary causal softmax attention (GQA head map u -> u // G), written
    independently of the block-sparse path."""
    Q, K, V = f64(Q), f64(K), f64(V)
    h_q, n, d = Q.shape
    G = h_q // K.shape[0]
    sc = (1.0 / math.sqrt(d)) if scale is None else scale
    O = np.zeros_like(Q)
    mask = np.tril(np.ones((n, n), dtype=bool))
    for u in range(h_q):
        S = (Q[u] @ K[u // G].T) * sc
        S = np.where(mask, S, -np.inf)
        O[u] = _softmax_rows(S) @ V[u // G]
    return O


# ---------------------------------------------------------------------------
# Prefill, one walked layer end to end (Alg. 1)
# ---------------------------------------------------------------------------

def prefill_layer(Q, K, V, B: int, signs, cols, s: int, R_prev: Optional[np.ndarray],
                  pct: int = 0, k: int = 0, flags: int = FORCE_BOTH,
                  attention: bool = True) -> dict:
    """Alg. 1 for one sequence at one layer: sketch, walk, select, attend."""
    sk = sketch_scores(Q, K, B, signs, cols)
    W = walk_weights(sk["A"], sk["c"], s)
    R = walk_step(R_prev, W)
    sel, gaps = select_blocks(R, pct=pct, k=k, flags=flags)
    out = dict(sk, W=W, R=R, sel=sel, gaps=gaps)
    if attention:
        out["O"] = sparse_attention_prefill(Q, K, V, B, sel)
    return out


# ---------------------------------------------------------------------------
# Decode (Alg. 2)
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class DecodeLayerState:
    """Per-(sequence, layer) caches Alg. 2 carries between steps: the block
    representatives (means of closed blocks), the head-averaged query and key
    of every token of the open block so far, the score matrix A
    (b_max x b_max) and the prefill score scale c."""
    qbar: np.ndarray
    kbar: np.ndarray
    qtok: np.ndarray      # [tokens of the open block][d], head-averaged queries
    ktok: np.ndarray      # [tokens of the open block][d], head-averaged keys
    A: np.ndarray
    c: float

    def copy(self) -> "DecodeLayerState":
        return DecodeLayerState(self.qbar.copy(), self.kbar.copy(), self.qtok.copy(),
                                self.ktok.copy(), self.A.copy(), self.c)


def decode_state_from_prefill(Q, K, B: int, signs, cols, b_max: int) -> DecodeLayerState:
    """Caches Alg. 2 takes over from the prefill of an n-token prompt: block
    means, the head-averaged tokens of the last (possibly partial) block, the
    prefill score matrix and its scale."""
    sk = sketch_scores(Q, K, B, signs, cols)
    n = Q.shape[1]
    b = sk["qbar"].shape[0]
    d = sk["qbar"].shape[1]
    qbar = np.zeros((b_max, d))
    kbar = np.zeros((b_max, d))
    qbar[:b] = sk["qbar"]
    kbar[:b] = sk["kbar"]
    A = np.zeros((b_max, b_max))
    A[:b, :b] = sk["A"]
    first = (b - 1) * B                      # first token of the last block
    qtok = head_mean(Q[:, first:n])
    ktok = head_mean(K[:, first:n])
    return DecodeLayerState(qbar, kbar, qtok, ktok, A, sk["c"])


def decode_layer_step(st: DecodeLayerState, q_new, k_new, p: int, r_prev: Optional[np.ndarray],
                      B: int, signs, cols, s: int, pct: int = 0, k: int = 0,
                      flags: int = FORCE_BOTH, variant: int = WALK_POWER):
    """Alg. 2 steps 2-6 for the token at 0-based position p of one sequence
    at one layer. q_new [h_q][d], k_new [h_kv][d]. Updates ``st`` in place and
    returns (walk row over key blocks 0..b_cur, selected blocks, gap).

    The open block's representatives are the token-space sketch itself (the
    mean over the tokens the block holds so far, Sec. 2.2), recomputed from
    its tokens; Alg. 2's running-mean update gives the same value."""
    q_new, k_new = f64(q_new), f64(k_new)
    b_cur = p // B
    b_q = b_cur
    r = len(cols)
    # steps 2-3: the new token joins the open block (a block starts at p % B == 0)
    q_avg = head_mean(q_new[:, None, :])[0]
    k_avg = head_mean(k_new[:, None, :])[0]
    if p % B == 0:
        st.qtok = q_avg[None, :]
        st.ktok = k_avg[None, :]
    else:
        st.qtok = np.concatenate([st.qtok, q_avg[None, :]])
        st.ktok = np.concatenate([st.ktok, k_avg[None, :]])
    st.kbar[b_cur] = block_means(st.ktok, B)[0]
    st.qbar[b_q] = block_means(st.qtok, B)[0]
    q_t = srht(q_avg[None, :], signs, cols)[0]
    Ks = srht(st.kbar[:b_cur + 1], signs, cols)
    Qs = srht(st.qbar[:b_q + 1], signs, cols)
    # step 4 (i): new query row; (ii) last column (overwrites the diagonal)
    st.A[b_q, :b_cur + 1] = (Ks @ q_t) / math.sqrt(r)
    st.A[:b_q + 1, b_cur] = (Qs @ Ks[b_cur]) / math.sqrt(r)
    # step 5: walk, restricted to the row of the current query block
    W = walk_weights_variant(variant, st.A[:b_cur + 1, :b_cur + 1], st.c, s)
    row = W[b_q].copy() if r_prev is None else r_prev @ W
    m = float(np.max(np.abs(row)))
    if m > 0.0:
        row = row / m
    # step 6: top-tau with the current block (and the first block) kept
    F = forced_set(b_cur, flags)
    tau = row_budget(b_cur + 1, len(F), pct=pct, k=k)
    chosen, gap = select_row(row, b_cur + 1, F, tau)
    return row, chosen, gap


def decode_attention(q, Kc, Vc, sel: Sequence[int], p: int, B: int,
                     scale: Optional[float] = None) -> np.ndarray:
    """Alg. 2 step 7: per query head u, softmax over the tokens t <= p of the
    selected blocks of KV head u // G. q [h_q][d], Kc/Vc [h_kv][T][d]."""
    q = f64(q)
    h_q, d = q.shape
    G = h_q // Kc.shape[0]
    sc = (1.0 / math.sqrt(d)) if scale is None else scale
    toks = np.concatenate([np.arange(j * B, min(p + 1, (j + 1) * B)) for j in sorted(sel)])
    Ks = f64(Kc[:, toks.tolist()])          # the selected tokens only, [h_kv][tokens][d]
    Vs = f64(Vc[:, toks.tolist()])
    out = np.zeros((h_q, d))
    for u in range(h_q):
        g = u // G
        logits = (Ks[g] @ q[u]) * sc
        e = np.exp(logits - np.max(logits))
        out[u] = (e @ Vs[g]) / e.sum()
    return out


# ---------------------------------------------------------------------------
# Work counts used by the benchmark (definitions, not measurements)
# ---------------------------------------------------------------------------

def executed_attention_flops(seqlens: Sequence[int], B: int, h_q: int, d: int,
                             sel_per_seq: Sequence[Sequence[Sequence[int]]]) -> int:
    """2 matmuls x 2 flop per multiply-add over every unmasked (query, key)
    pair the sparse attention computes: 4 d per pair."""
    total = 0
    for n, sel in zip(seqlens, sel_per_seq):
        for i, row in enumerate(sel):
            ci = min(B, n - i * B)
            for j in row:
                cj = min(B, n - j * B)
                pairs = ci * (ci + 1) // 2 if j == i else ci * cj
                total += 4 * d * pairs * h_q
    return total
