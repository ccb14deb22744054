"""Planted mistakes in copies of the oracle's functions must fail a pin.

Each mutant is a plausible slip (a dropped term, a wrong sign, an off-by-one
index, a swapped operand, a missing rule of the paper). The pins live in
``test_oracle_pins.py``; here they must return False on the mutant.
"""
import math

import numpy as np
import pytest

import oracle as O
import test_oracle_pins as P


# ------------------------------------------------------------------ mutants

def summaries_off_by_one(K, seq_len, block_size, blocks=None):
    L, b = int(seq_len), int(block_size)
    M = -(-L // b)
    kmin = np.empty((M, K.shape[1]))
    kmax = np.empty((M, K.shape[1]))
    for m in range(M):
        rows = K[m * b:min((m + 1) * b + 1, L)]
        kmin[m], kmax[m] = rows.min(axis=0), rows.max(axis=0)
    return kmin, kmax


def summaries_ignore_length(K, seq_len, block_size, blocks=None):
    L, b = int(seq_len), int(block_size)
    M = -(-L // b)
    kmin = np.empty((M, K.shape[1]))
    kmax = np.empty((M, K.shape[1]))
    for m in range(M):
        rows = K[m * b:(m + 1) * b]
        kmin[m], kmax[m] = rows.min(axis=0), rows.max(axis=0)
    return kmin, kmax


def scores_min(qbar, kmin, kmax):
    return np.minimum(qbar[None] * kmax, qbar[None] * kmin).sum(axis=1)


def scores_kmax_only(qbar, kmin, kmax):
    return (qbar[None] * kmax).sum(axis=1)


def scores_swapped(qbar, kmin, kmax):
    return np.maximum(qbar[None] * kmin, qbar[None] * kmin[::-1]).sum(axis=1)


def pooled_sum(q):
    return np.asarray(q, dtype=np.float64).sum(axis=0)


def pooled_first(q):
    return np.asarray(q, dtype=np.float64)[0]


def count_s_as_keep(M, s, nmin, nloc):
    if M <= 0:
        return 0
    return min(M, max(nmin, nloc, math.ceil(M * s)))


def count_float_ceil(M, s, nmin, nloc):
    if M <= 0:
        return 0
    return min(M, max(nmin, nloc, math.ceil(M * (1 - s))))


def count_no_local(M, s, nmin, nloc):
    if M <= 0:
        return 0
    from fractions import Fraction
    return min(M, max(nmin, math.ceil(M * (1 - Fraction(str(s))))))


def count_no_clamp(M, s, nmin, nloc):
    if M <= 0:
        return 0
    from fractions import Fraction
    return max(nmin, nloc, math.ceil(M * (1 - Fraction(str(s)))))


def select_no_forcing(scores, n, n_local):
    order = sorted(range(len(scores)), key=lambda m: (-scores[m], m))
    return np.array(sorted(order[:n]), dtype=np.int64)


def select_high_index_ties(scores, n, n_local):
    s = np.array(scores, dtype=np.float64)
    if n_local > 0:
        s[len(s) - n_local:] = np.inf
    order = sorted(range(len(s)), key=lambda m: (-s[m], -m))
    return np.array(sorted(order[:n]), dtype=np.int64)


def select_unsorted(scores, n, n_local):
    s = np.array(scores, dtype=np.float64)
    if n_local > 0:
        s[len(s) - n_local:] = np.inf
    order = sorted(range(len(s)), key=lambda m: (-s[m], m))
    return np.array(order[:n], dtype=np.int64)


def attend_no_scale(q, K, V, tokens, sm_scale):
    return O.attend(q, K, V, tokens, 1.0)


def attend_kv_swapped(q, K, V, tokens, sm_scale):
    return O.attend(q, V, K, tokens, sm_scale)


def attend_lse_drops_max(q, K, V, tokens, sm_scale):
    o, l = O.attend(q, K, V, tokens, sm_scale)
    z = (np.atleast_2d(q) @ K[list(tokens)].T) * sm_scale
    return o, l - z.max(axis=1)


def attend_no_normalise(q, K, V, tokens, sm_scale):
    q = np.atleast_2d(q)
    t = list(tokens)
    z = (q @ K[t].T) * sm_scale
    w = np.exp(z - z.max(axis=1, keepdims=True))
    return w @ V[t], z.max(axis=1) + np.log(w.sum(axis=1))


def dense_no_scale(q, K, V, L, sm_scale):
    return O.attend(q, K, V, range(L), 1.0)


def sparse_last_token_dropped(q, K, V, L, ids, b, sm_scale):
    toks = [t for m in ids for t in range(m * b, min((m + 1) * b, L) - 1)]
    return O.attend(q, K, V, toks, sm_scale)


def sparse_mask_to_zero(q, K, V, L, ids, b, sm_scale):
    """Eq. 2 read literally: masked logits set to 0 instead of excluded."""
    q = np.atleast_2d(q)
    sel = set(O.block_tokens(ids, L, b).tolist())
    z = (q @ K[:L].T) * sm_scale
    for t in range(L):
        if t not in sel:
            z[:, t] = 0.0
    w = np.exp(z - z.max(axis=1, keepdims=True))
    den = w.sum(axis=1)
    return (w @ V[:L]) / den[:, None], z.max(axis=1) + np.log(den)


def merge_wrong_sign(outs, lses):
    return O.merge_partials(outs, -np.asarray(lses))


def rectify_non_causal(q_f, K, V, kmin, kmax, L, f, b, sm_scale, k_f, v_f):
    K[L - f:L], V[L - f:L] = k_f, v_f
    g = q_f.shape[0]
    out = np.zeros((g, f, V.shape[1]))
    lse = np.zeros((g, f))
    for r in range(f):
        out[:, r], lse[:, r] = O.attend(q_f[:, r], K, V, range(L), sm_scale)
    lo, M = (L - f) // b, -(-L // b)
    nmin, nmax = O.block_summaries(K, L, b)
    kmin[lo:M], kmax[lo:M] = nmin[lo:M], nmax[lo:M]
    return out, lse


def rectify_causal_off_by_one(q_f, K, V, kmin, kmax, L, f, b, sm_scale, k_f, v_f):
    K[L - f:L], V[L - f:L] = k_f, v_f
    g = q_f.shape[0]
    out = np.zeros((g, f, V.shape[1]))
    lse = np.zeros((g, f))
    for r in range(f):
        out[:, r], lse[:, r] = O.attend(q_f[:, r], K, V, range(max(L - f + r, 1)), sm_scale)
    lo, M = (L - f) // b, -(-L // b)
    nmin, nmax = O.block_summaries(K, L, b)
    kmin[lo:M], kmax[lo:M] = nmin[lo:M], nmax[lo:M]
    return out, lse


def rectify_no_refresh(q_f, K, V, kmin, kmax, L, f, b, sm_scale, k_f, v_f):
    K[L - f:L], V[L - f:L] = k_f, v_f
    g = q_f.shape[0]
    out = np.zeros((g, f, V.shape[1]))
    lse = np.zeros((g, f))
    for r in range(f):
        out[:, r], lse[:, r] = O.attend(q_f[:, r], K, V, range(L - f + r + 1), sm_scale)
    return out, lse


def rectify_refresh_short(q_f, K, V, kmin, kmax, L, f, b, sm_scale, k_f, v_f):
    """Refreshes from block (L - f) / b + 1: misses the block holding row L - f."""
    K[L - f:L], V[L - f:L] = k_f, v_f
    g = q_f.shape[0]
    out = np.zeros((g, f, V.shape[1]))
    lse = np.zeros((g, f))
    for r in range(f):
        out[:, r], lse[:, r] = O.attend(q_f[:, r], K, V, range(L - f + r + 1), sm_scale)
    lo, M = (L - f) // b + 1, -(-L // b)
    nmin, nmax = O.block_summaries(K, L, b)
    kmin[lo:M], kmax[lo:M] = nmin[lo:M], nmax[lo:M]
    return out, lse


def update_no_reinit(kmin, kmax, pos, b, k_new):
    m = pos // b
    kmin[m] = np.fmin(kmin[m], k_new)
    kmax[m] = np.fmax(kmax[m], k_new)


def update_wrong_block(kmin, kmax, pos, b, k_new):
    m = (pos + 1) // b
    if pos % b == 0:
        kmin[m] = k_new
        kmax[m] = k_new
    else:
        kmin[m] = np.minimum(kmin[m], k_new)
        kmax[m] = np.maximum(kmax[m], k_new)


def split_heads_interleaved(q, num_kv_heads):
    """Query head h taken as a member of kv head h % Hkv (not h // g)."""
    B, Hq = q.shape[:2]
    g = Hq // num_kv_heads
    return np.swapaxes(q.reshape(B, g, num_kv_heads, *q.shape[2:]), 1, 2)


class StateAttendScattered(O.DecodeState):
    """Groups attended correctly but written back at heads i, i + Hkv, ..."""

    def attend(self, q, idx, sm_scale):
        out, lse = super().attend(q, idx, sm_scale)
        B, H = self.K.shape[:2]
        g = out.shape[1] // H
        return (np.swapaxes(out.reshape(B, H, g, -1), 1, 2).reshape(out.shape),
                np.swapaxes(lse.reshape(B, H, g), 1, 2).reshape(lse.shape))


class StateSelectFirstHead(O.DecodeState):
    """Each group scored with its first query head instead of the pooled mean."""

    def select(self, q, sparsity, min_blocks, n_local):
        q = np.asarray(q, dtype=np.float64)
        B, Hq = q.shape[:2]
        g = Hq // self.K.shape[1]
        q1 = np.repeat(q[:, ::g], g, axis=1)
        return super().select(q1, sparsity, min_blocks, n_local)


def with_split_heads(fn, pin):
    """Runs ``pin`` with the oracle module's split_heads replaced by ``fn``."""
    def run():
        saved = O.resa_oracle.split_heads
        O.resa_oracle.split_heads = fn
        try:
            return pin()
        finally:
            O.resa_oracle.split_heads = saved
    return run


# ------------------------------------------------------------------- table

S, Q, C, SEL = O.block_summaries, O.pooled_query, O.num_selected, O.select_blocks
CASES = {
    "summaries_off_by_one": lambda: P.pin_summaries_bruteforce(summaries_off_by_one),
    "summaries_ignore_length": lambda: P.pin_summaries_bruteforce(summaries_ignore_length),
    "scores_min": lambda: P.pin_quest_upper_bound(S, Q, scores_min),
    "scores_kmax_only": lambda: P.pin_score_sign_split(scores_kmax_only),
    "scores_swapped": lambda: P.pin_worked_example(S, Q, scores_swapped, C, SEL),
    "pooled_sum": lambda: P.pin_worked_example(S, pooled_sum, O.block_scores, C, SEL),
    "pooled_first": lambda: P.pin_score_b1_is_dot(S, pooled_first, O.block_scores),
    "count_s_as_keep": lambda: P.pin_eq5_table(count_s_as_keep),
    "count_float_ceil": lambda: P.pin_eq5_table(count_float_ceil),
    "count_no_local": lambda: P.pin_eq5_table(count_no_local),
    "count_no_clamp": lambda: P.pin_eq5_closed_form(count_no_clamp),
    "select_no_forcing": lambda: P.pin_select_bruteforce(select_no_forcing),
    "select_high_index_ties": lambda: P.pin_select_bruteforce(select_high_index_ties),
    "select_unsorted": lambda: P.pin_select_bruteforce(select_unsorted),
    "attend_no_scale": lambda: P.pin_attend_naive(attend_no_scale),
    "attend_kv_swapped": lambda: P.pin_attend_naive(attend_kv_swapped),
    "attend_lse_drops_max": lambda: P.pin_attend_naive(attend_lse_drops_max),
    "attend_no_normalise": lambda: P.pin_attend_naive(attend_no_normalise),
    "dense_no_scale": lambda: P.pin_attend_sdpa(dense_no_scale),
    "sparse_last_token_dropped": lambda: P.pin_worked_attention(sparse_last_token_dropped),
    "sparse_mask_to_zero": lambda: P.pin_worked_attention(sparse_mask_to_zero),
    "merge_wrong_sign": lambda: P.pin_partition_merge(O.sparse_attend, merge_wrong_sign),
    "rectify_non_causal": lambda: P.pin_rectify_textbook(rectify_non_causal, S),
    "rectify_causal_off_by_one": lambda: P.pin_rectify_textbook(rectify_causal_off_by_one, S),
    "rectify_no_refresh": lambda: P.pin_rectify_textbook(rectify_no_refresh, S),
    "rectify_refresh_short": lambda: P.pin_worked_rectify(rectify_refresh_short),
    "update_no_reinit": lambda: P.pin_incremental_summary(update_no_reinit, S),
    "update_wrong_block": lambda: P.pin_incremental_summary(update_wrong_block, S),
    "split_heads_interleaved_attend": with_split_heads(
        split_heads_interleaved, lambda: P.pin_gqa_attend(O.DecodeState)),
    "split_heads_interleaved_select": with_split_heads(
        split_heads_interleaved, lambda: P.pin_gqa_select(O.DecodeState)),
    "split_heads_interleaved_rectify": with_split_heads(
        split_heads_interleaved, lambda: P.pin_gqa_rectify(O.DecodeState)),
    "state_attend_scattered": lambda: P.pin_gqa_attend(StateAttendScattered),
    "state_select_first_head": lambda: P.pin_gqa_select(StateSelectFirstHead),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_pin_catches_mutant(name):
    try:
        ok = CASES[name]()
    except (IndexError, ValueError, AssertionError):
        ok = False  # the mutant broke outright: also caught
    assert ok is False, f"mutant {name} passed its pin"
