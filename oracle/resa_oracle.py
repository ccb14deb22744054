"""Plain CPU oracle of Rectified Sparse Attention (ReSA) decoding.

TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's CPU
baseline may import this module; the library never calls it and never falls
back to it. It shares no code with the HIP path.

Everything is float64 on the exact values of bf16 inputs (bf16 -> float64 is
exact), one (batch, kv-head) group at a time, with no blocking, fusion or
reordering beyond what the paper's definitions state. Paper references are to
"Rectified Sparse Attention" (arXiv 2506.04108):

* Eq. 1   grouped-query attention  softmax(Q_ij K_i^T / sqrt(d)) V_i
* Eq. 2   group block sparse attention (softmax restricted to selected blocks)
* Eq. 3   block representation: element-wise min / max of the b keys of a block
* Eq. 4   Quest block score  sum_j max(q_j kmax_j, q_j kmin_j)
* Eq. 5   dynamic top-n  n = max(n_min, ceil(M * p)), with n_local forced blocks
* Sec. 2.1 "Block Selection" (local forcing), Fig. 3 (average pooling of the g
  query heads, one block set per GQA group)
* Sec. 2.2 "Rectification Algorithm" and Alg. 1 (dense re-encoding of the last
  f tokens every f steps, followed by a block-key refresh)
* App. A, Alg. 2 (split flash-decoding with a log-sum-exp combine)

Readings taken where the paper is silent or inconsistent (each is listed in
the design notes with its reason):

* p in Eq. 5 is the KEPT fraction; the API takes the sparsity s and keeps
  ceil(M * (1 - s)) blocks, computed exactly in decimal (``Fraction(str(s))``).
* n = min(M, max(n_min, n_local, ceil(M (1 - s)))); M = ceil(L / b) counts a
  partial last block, whose summary covers its valid tokens only.
* Ties in the top-n go to the lower block index; the selected ids are returned
  in ascending order.
* A masked logit in Eq. 2 is excluded from the softmax (weight exactly zero),
  not multiplied to zero.
* The block score uses the mean of the g query heads and no 1/sqrt(d) scale.
* The decode query sees its own key: the current token is appended first.
* Rectify takes the re-encoded rows (q_f, k_f, v_f) as inputs, writes k_f/v_f
  over cache rows [L - f, L), attends causally (row r sees t <= L - f + r) and
  recomputes the summaries of every block that holds a rewritten row.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np


# ----------------------------------------------------------------- conversions

def bf16_to_f64(u16) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float64, exactly."""
    u = np.asarray(u16, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def f64_to_bf16_exact(x: np.ndarray) -> np.ndarray:
    """float64 values that are exactly bf16-representable -> uint16 bits.

    Used for summaries, which are min/max of bf16 values and therefore bf16
    values themselves. Raises if a value would need rounding.
    """
    x = np.asarray(x, dtype=np.float64)
    f = x.astype(np.float32)
    if not np.array_equal(f.astype(np.float64), x, equal_nan=True):
        raise ValueError("value not representable in float32")
    u = f.view(np.uint32)
    if np.any(u & 0xFFFF):
        raise ValueError("value not representable in bf16")
    return (u >> 16).astype(np.uint16)


# ---------------------------------------------------------- Eq. 3: block summary

def num_blocks(seq_len: int, block_size: int) -> int:
    """M = ceil(L / b): the available blocks, a partial last block included."""
    return -(-int(seq_len) // int(block_size))


def block_summaries(K: np.ndarray, seq_len: int, block_size: int,
                    blocks: range | None = None):
    """Eq. 3: element-wise min and max of the keys of each block.

    K: ``[>= L, D]`` float64 keys of one (batch, kv-head) group.
    Returns ``(kmin, kmax)``, each ``[M, D]``; block m covers tokens
    ``[m*b, min((m+1)*b, L))``. ``blocks`` restricts the work to a range (the
    other rows are returned as NaN).
    """
    L, b = int(seq_len), int(block_size)
    M = num_blocks(L, b)
    D = K.shape[1]
    kmin = np.full((M, D), np.nan)
    kmax = np.full((M, D), np.nan)
    if blocks is None:
        # Every block: the full ones as one [blocks, b, D] view, then the
        # partial last one (the same element-wise min and max).
        full = L // b
        if full:
            rows = K[:full * b].reshape(full, b, D)
            kmin[:full] = rows.min(axis=1)
            kmax[:full] = rows.max(axis=1)
        blocks = range(full, M)
    for m in blocks:
        rows = K[m * b:min((m + 1) * b, L)]
        kmin[m] = rows.min(axis=0)
        kmax[m] = rows.max(axis=0)
    return kmin, kmax


def update_summary(kmin: np.ndarray, kmax: np.ndarray, pos: int, block_size: int,
                   k_new: np.ndarray):
    """Online update of the block statistics by the key written at ``pos``
    (Sec. 2.1, "Block Representation": new keys are folded into the running
    min/max; Alg. 1 updates the block-key cache after each token).

    A key that opens a new block initialises that block's min and max.
    Arrays are modified in place; they must have room for block ``pos // b``.
    """
    m = pos // block_size
    if pos % block_size == 0:
        kmin[m] = k_new
        kmax[m] = k_new
    else:
        kmin[m] = np.minimum(kmin[m], k_new)
        kmax[m] = np.maximum(kmax[m], k_new)


# ------------------------------------------------- Fig. 3 / Eq. 4: block scoring

def pooled_query(q_group: np.ndarray) -> np.ndarray:
    """Average pooling of the g query heads of one GQA group (Fig. 3)."""
    return np.asarray(q_group, dtype=np.float64).mean(axis=0)


def block_scores(qbar: np.ndarray, kmin: np.ndarray, kmax: np.ndarray) -> np.ndarray:
    """Eq. 4: score_m = sum_j max(q_j * kmax_mj, q_j * kmin_mj)."""
    return np.maximum(qbar[None, :] * kmax, qbar[None, :] * kmin).sum(axis=1)


# ----------------------------------------------------------- Eq. 5: block count

def num_selected(num_blocks_: int, sparsity: float, min_blocks: int, n_local: int) -> int:
    """Eq. 5 with p read as the kept fraction 1 - s, in exact decimal arithmetic.

    n = min(M, max(n_min, n_local, ceil(M * (1 - s)))).
    """
    M = int(num_blocks_)
    if M <= 0:
        return 0
    keep = 1 - Fraction(str(sparsity))
    n = max(int(min_blocks), int(n_local), math.ceil(M * keep))
    return min(M, n)


def select_blocks(scores: np.ndarray, n: int, n_local: int) -> np.ndarray:
    """Dynamic top-n of Sec. 2.1: the last ``n_local`` blocks get score +inf,
    then the n best blocks by (score descending, block id ascending) are kept.

    Returns the selected block ids in ascending order (int64).
    """
    s = np.array(scores, dtype=np.float64)
    M = s.shape[0]
    if n_local > 0:
        s[max(M - n_local, 0):] = np.inf
    order = sorted(range(M), key=lambda m: (-s[m], m))
    return np.array(sorted(order[:n]), dtype=np.int64)


# ------------------------------------------------ Eq. 1 / Eq. 2: the attention

def attend(q_heads: np.ndarray, K: np.ndarray, V: np.ndarray, tokens,
           sm_scale: float):
    """Softmax attention of each query row over the listed token positions.

    q_heads ``[g, D]``; K, V ``[>= max(tokens)+1, D]``. Returns ``(O [g, D],
    lse [g])`` with ``lse = log sum_t exp(q . K_t * sm_scale)``. With no token
    the output is zero and lse is -inf.
    """
    q_heads = np.atleast_2d(np.asarray(q_heads, dtype=np.float64))
    tokens = np.asarray(list(tokens), dtype=np.int64)
    g, D = q_heads.shape
    if tokens.size == 0:
        return np.zeros((g, V.shape[1])), np.full(g, -np.inf)
    z = (q_heads @ K[tokens].T) * sm_scale          # [g, T]
    zmax = z.max(axis=1, keepdims=True)
    w = np.exp(z - zmax)
    den = w.sum(axis=1)
    out = (w @ V[tokens]) / den[:, None]
    return out, zmax[:, 0] + np.log(den)


def block_tokens(block_ids, seq_len: int, block_size: int) -> np.ndarray:
    """Token positions covered by the given blocks, cut at L (Eq. 2's mask
    expanded per token, M_bar[k] = M[floor(k / b)])."""
    L, b = int(seq_len), int(block_size)
    toks = [t for m in block_ids for t in range(int(m) * b, min((int(m) + 1) * b, L))]
    return np.array(toks, dtype=np.int64)


def sparse_attend(q_heads, K, V, seq_len, block_ids, block_size, sm_scale):
    """Eq. 2 for one GQA group: every query head of the group attends to the
    tokens of the shared selected blocks only (masked tokens excluded)."""
    return attend(q_heads, K, V, block_tokens(block_ids, seq_len, block_size), sm_scale)


def dense_attend(q_heads, K, V, seq_len, sm_scale):
    """Eq. 1 for one decode query per head over all L cached tokens."""
    return attend(q_heads, K, V, range(int(seq_len)), sm_scale)


def merge_partials(outs, lses):
    """Alg. 2's combine: partial outputs over disjoint token sets merged by
    their log-sum-exp weights. ``outs [S, g, D]``, ``lses [S, g]``."""
    outs = np.asarray(outs, dtype=np.float64)
    lses = np.asarray(lses, dtype=np.float64)
    top = lses.max(axis=0)
    finite = np.isfinite(top)
    safe = np.where(finite, top, 0.0)
    w = np.where(np.isfinite(lses), np.exp(lses - safe[None, :]), 0.0)
    den = w.sum(axis=0)
    out = np.where(finite[:, None],
                   (w[:, :, None] * outs).sum(axis=0) / np.where(den > 0, den, 1.0)[:, None],
                   0.0)
    lse = np.where(finite, safe + np.log(np.where(den > 0, den, 1.0)), -np.inf)
    return out, lse


# --------------------------------------------------------- one decode step

def decode_group(q_group, K, V, seq_len, block_size, sparsity, min_blocks, n_local,
                 sm_scale):
    """Sparse decoding for one (batch, kv-head) group (Sec. 2.1, Eq. 2-5).

    q_group ``[g, D]`` float64; K, V ``[>= L, D]`` float64. Returns a dict with
    the summaries, scores, count n, selected ids, output ``[g, D]`` and lse.
    """
    kmin, kmax = block_summaries(K, seq_len, block_size)
    qbar = pooled_query(q_group)
    scores = block_scores(qbar, kmin, kmax)
    n = num_selected(kmin.shape[0], sparsity, min_blocks, n_local)
    idx = select_blocks(scores, n, n_local)
    out, lse = sparse_attend(q_group, K, V, seq_len, idx, block_size, sm_scale)
    return {"kmin": kmin, "kmax": kmax, "scores": scores, "n": n, "idx": idx,
            "out": out, "lse": lse}


# ------------------------------------------------------- Sec. 2.2: rectify

def rectify_group(q_f, K, V, kmin, kmax, seq_len, f, block_size, sm_scale,
                  k_f, v_f):
    """Dense rectification of the last f cache rows of one group.

    q_f ``[g, f, D]``; k_f, v_f ``[f, D]``; K, V ``[>= L, D]`` float64 and
    kmin/kmax ``[>= ceil(L/b), D]`` are updated in place. Row r of the window is
    cache position ``L - f + r`` and attends to positions ``t <= L - f + r``.
    Returns ``O [g, f, D]`` and ``lse [g, f]``.
    """
    L, f, b = int(seq_len), int(f), int(block_size)
    K[L - f:L] = k_f
    V[L - f:L] = v_f
    g = q_f.shape[0]
    out = np.zeros((g, f, V.shape[1]))
    lse = np.zeros((g, f))
    for r in range(f):
        o, s = attend(q_f[:, r, :], K, V, range(L - f + r + 1), sm_scale)
        out[:, r] = o
        lse[:, r] = s
    lo, hi = (L - f) // b, num_blocks(L, b)
    nmin, nmax = block_summaries(K, L, b, blocks=range(lo, hi))
    kmin[lo:hi] = nmin[lo:hi]
    kmax[lo:hi] = nmax[lo:hi]
    return out, lse


# ----------------------------------------------------- whole-batch helpers

def split_heads(q: np.ndarray, num_kv_heads: int) -> np.ndarray:
    """``[B, Hq, ...]`` -> ``[B, Hkv, g, ...]`` with query head h = i*g + j."""
    B, Hq = q.shape[:2]
    return q.reshape(B, num_kv_heads, Hq // num_kv_heads, *q.shape[2:])


class DecodeState:
    """Cache of one batch of sequences for the kernel-level decode loop of
    Alg. 1: caches, block-key cache and lengths, all float64 on the host."""

    def __init__(self, K, V, seq_lens, block_size):
        self.K = np.array(K, dtype=np.float64)        # [B, Hkv, cap, D]
        self.V = np.array(V, dtype=np.float64)
        self.b = int(block_size)
        self.L = [int(x) for x in seq_lens]
        B, H, cap, D = self.K.shape
        mcap = num_blocks(cap, self.b)
        self.kmin = np.full((B, H, mcap, D), np.nan)
        self.kmax = np.full((B, H, mcap, D), np.nan)
        for bi in range(B):
            for hi in range(H):
                mn, mx = block_summaries(self.K[bi, hi], self.L[bi], self.b)
                M = mn.shape[0]
                self.kmin[bi, hi, :M] = mn
                self.kmax[bi, hi, :M] = mx

    def append(self, k_new, v_new):
        """Alg. 1: write the new token's key/value and fold it into the block keys."""
        B, H = self.K.shape[:2]
        for bi in range(B):
            pos = self.L[bi]
            for hi in range(H):
                self.K[bi, hi, pos] = k_new[bi, hi]
                self.V[bi, hi, pos] = v_new[bi, hi]
                update_summary(self.kmin[bi, hi], self.kmax[bi, hi], pos, self.b,
                               self.K[bi, hi, pos])
            self.L[bi] = pos + 1

    def select(self, q, sparsity, min_blocks, n_local):
        """Pool, score and select for every group; returns (scores, idx lists, n)."""
        B, H = self.K.shape[:2]
        qg = split_heads(np.asarray(q, dtype=np.float64), H)
        scores, idx, ns = {}, {}, {}
        for bi in range(B):
            M = num_blocks(self.L[bi], self.b)
            for hi in range(H):
                s = block_scores(pooled_query(qg[bi, hi]), self.kmin[bi, hi, :M],
                                 self.kmax[bi, hi, :M])
                n = num_selected(M, sparsity, min_blocks, n_local)
                scores[bi, hi] = s
                ns[bi, hi] = n
                idx[bi, hi] = select_blocks(s, n, n_local)
        return scores, idx, ns

    def attend(self, q, idx, sm_scale):
        """Eq. 2 for every group with the given block sets: ``(O [B,Hq,D], lse [B,Hq])``."""
        B, H = self.K.shape[:2]
        qg = split_heads(np.asarray(q, dtype=np.float64), H)
        g = qg.shape[2]
        out = np.zeros((B, H * g, self.K.shape[3]))
        lse = np.zeros((B, H * g))
        for bi in range(B):
            for hi in range(H):
                o, s = sparse_attend(qg[bi, hi], self.K[bi, hi], self.V[bi, hi], self.L[bi],
                                     idx[bi, hi], self.b, sm_scale)
                out[bi, hi * g:(hi + 1) * g] = o
                lse[bi, hi * g:(hi + 1) * g] = s
        return out, lse

    def rectify(self, q_f, k_f, v_f, f, sm_scale):
        """Sec. 2.2 for every group: ``q_f [B,Hq,f,D]``, ``k_f, v_f [B,Hkv,f,D]``."""
        B, H = self.K.shape[:2]
        qg = split_heads(np.asarray(q_f, dtype=np.float64), H)
        g = qg.shape[2]
        out = np.zeros((B, H * g, f, self.K.shape[3]))
        lse = np.zeros((B, H * g, f))
        for bi in range(B):
            for hi in range(H):
                o, s = rectify_group(qg[bi, hi], self.K[bi, hi], self.V[bi, hi],
                                     self.kmin[bi, hi], self.kmax[bi, hi], self.L[bi], f,
                                     self.b, sm_scale, k_f[bi, hi], v_f[bi, hi])
                out[bi, hi * g:(hi + 1) * g] = o
                lse[bi, hi * g:(hi + 1) * g] = s
        return out, lse
