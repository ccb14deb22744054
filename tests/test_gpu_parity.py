"""GPU parity of every step of the ReSA decode path against the CPU oracle.

All calls go through the C ABI (via the ctypes binding). Bars: summaries and
indices bit-exact (selection up to documented near-ties, |score - threshold|
<= 1e-3), attention outputs and lse within 2e-3 absolute (bf16 in, fp32
accumulate).
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
import paper_2506_04108_amd as R
import workloads as W
from gpu_util import (SENTINEL, dev, down, i32, make_cache, make_paged_cache, oracle_summaries,
                      select_stats,
                      padded_idx, unpage, up)
from oracle.compare import check_selection, max_abs_err

pytestmark = pytest.mark.gpu
TOL = 2e-3


def small(g=4, b=16, L=1000, cap=1024, B=2, H=2, tag="t", **kw):
    return W.TINY_4K.with_(batch=B, num_kv_heads=H, num_q_heads=g * H, seq_len=L, block_size=b,
                           seed_tag=f"{tag}-{g}-{b}-{L}", **kw), cap


# ------------------------------------------------------------------ summaries

@pytest.mark.parametrize("b", [16, 32, 64])
def test_summarize_bitexact(b):
    w, cap = small(b=b, tag="sum")
    lens = [1000, 777]
    K, V = W.kv_cache(w, capacity=cap)
    cache = make_cache(K, V, b)
    R.block_summarize(cache, i32(lens))
    torch.cuda.synchronize()
    gmin, gmax = down(cache.kmin), down(cache.kmax)
    ref = oracle_summaries(O.bf16_to_f64(K), lens, b)
    for (bi, hi), (mn, mx) in ref.items():
        M = mn.shape[0]
        assert np.array_equal(O.bf16_to_f64(gmin[bi, hi, :M]), mn)
        assert np.array_equal(O.bf16_to_f64(gmax[bi, hi, :M]), mx)
        assert np.all(gmin[bi, hi, M:] == SENTINEL) and np.all(gmax[bi, hi, M:] == SENTINEL)


def test_summarize_range_only():
    w, cap = small(tag="sumr")
    lens = [1000, 100]
    K, V = W.kv_cache(w, capacity=cap)
    cache = make_cache(K, V, 16)
    R.block_summarize(cache, i32(lens), 3, 10)
    torch.cuda.synchronize()
    gmin = down(cache.kmin)
    ref = oracle_summaries(O.bf16_to_f64(K), lens, 16)
    for bi, M in ((0, 63), (1, 7)):
        mn = ref[bi, 0][0]
        assert np.array_equal(O.bf16_to_f64(gmin[bi, 0, 3:min(10, M)]), mn[3:min(10, M)])
        assert np.all(gmin[bi, 0, :3] == SENTINEL)
        assert np.all(gmin[bi, 0, min(10, M):] == SENTINEL)


# --------------------------------------------------------------------- append

def test_append_incremental_summaries():
    w, cap = small(L=100, cap=256, tag="app")
    lens = [100, 93]
    K, V = W.kv_cache(w, capacity=cap)
    cache = make_cache(K, V, 16, sentinel=False)
    lt = i32(lens)
    R.block_summarize(cache, lt)
    st = O.DecodeState(O.bf16_to_f64(K), O.bf16_to_f64(V), lens, 16)
    for step in range(40):
        kn, vn = W.decode_kv(w, step)
        R.append_kv(cache, up(kn), up(vn), lt, max(st.L))
        st.append(O.bf16_to_f64(kn), O.bf16_to_f64(vn))
    torch.cuda.synchronize()
    assert lt.cpu().tolist() == st.L == [140, 133]
    assert np.array_equal(O.bf16_to_f64(down(cache.k)), st.K)
    assert np.array_equal(O.bf16_to_f64(down(cache.v)), st.V)
    gmin, gmax = O.bf16_to_f64(down(cache.kmin)), O.bf16_to_f64(down(cache.kmax))
    for bi in range(2):
        M = O.num_blocks(st.L[bi], 16)
        assert np.array_equal(gmin[bi, :, :M], st.kmin[bi, :, :M])
        assert np.array_equal(gmax[bi, :, :M], st.kmax[bi, :, :M])


def test_append_full_cache_is_left_alone():
    w, cap = small(L=64, cap=64, B=1, tag="full")
    K, V = W.kv_cache(w, capacity=cap)
    cache = make_cache(K, V, 16, sentinel=False)
    lt = i32([64])
    kn, vn = W.decode_kv(w, 0)
    with pytest.raises(R.ResaError):
        R.append_kv(cache, up(kn[:1]), up(vn[:1]), lt, 64)
    # A host bound below the device length: the kernel itself refuses to write.
    R.append_kv(cache, up(kn[:1]), up(vn[:1]), lt, 10)
    torch.cuda.synchronize()
    assert lt.cpu().tolist() == [64]
    assert np.array_equal(down(cache.k), K)


# ------------------------------------------------------------------ selection

def run_select(w, cap, lens, q, scores=True, sparsity=None, min_blocks=None, K=None, V=None):
    if K is None:
        K, V = W.kv_cache(w, capacity=cap)
    cache = make_cache(K, V, w.block_size)
    lt = i32(lens)
    R.block_summarize(cache, lt)
    s = w.sparsity if sparsity is None else sparsity
    nm = w.min_blocks if min_blocks is None else min_blocks
    mseq = -(-max(lens) // w.block_size)
    sc = torch.full((w.batch, w.num_kv_heads, mseq), float("nan"), device=dev()) if scores else None
    idx, ns = R.select_blocks(cache, up(q), lt, max(lens), s, nm, w.n_local, scores_out=sc)
    torch.cuda.synchronize()
    st = O.DecodeState(O.bf16_to_f64(K), O.bf16_to_f64(V), lens, w.block_size)
    ref_s, ref_i, ref_n = st.select(O.bf16_to_f64(q), s, nm, w.n_local)
    return cache, idx.cpu().numpy(), ns.cpu().numpy(), (sc.cpu().numpy() if scores else None), \
        ref_s, ref_i, ref_n, st


@pytest.mark.parametrize("b", [16, 32, 64])
def test_select_vs_oracle_tiny4k(b):
    w = W.TINY_4K.with_(block_size=b, min_tokens=64 * b)
    q = W.decode_query(w)
    _, gi, gn, gs, rs, ri, rn, _ = run_select(w, 4096, [4096], q)
    swaps = 0
    for hi in range(w.num_kv_heads):
        M = O.num_blocks(4096, b)
        assert gn[0, hi] == rn[0, hi] == O.num_selected(M, w.sparsity, w.min_blocks, 1)
        assert max_abs_err(gs[0, hi, :M], rs[0, hi]) <= 1e-3
        swaps += check_selection(gi[0, hi, :gn[0, hi]], ri[0, hi], rs[0, hi], rn[0, hi], 1)
        assert np.all(gi[0, hi, gn[0, hi]:] == -1)
    assert swaps <= 2


@pytest.mark.parametrize("g", [1, 3, 5, 6, 7])
def test_select_ragged_batch_and_sparsities(g):
    """Ragged lengths (one sequence of 17 tokens) at several sparsities and
    minimum budgets, for group sizes whose pooled query averages 1 to 7
    heads."""
    w, cap = small(g=g, L=3000, cap=3072, B=3, H=2, tag="selr")
    lens = [3000, 17, 2049]
    q = W.decode_query(w)
    for s, nm in ((0.8, 4), (0.95, 0), (0.0, 0), (1.0, 2)):
        _, gi, gn, gs, rs, ri, rn, _ = run_select(w, cap, lens, q, sparsity=s, min_blocks=nm)
        for bi in range(3):
            for hi in range(2):
                M = O.num_blocks(lens[bi], 16)
                assert gn[bi, hi] == rn[bi, hi]
                assert max_abs_err(gs[bi, hi, :M], rs[bi, hi]) <= 1e-3
                check_selection(gi[bi, hi, :gn[bi, hi]], ri[bi, hi], rs[bi, hi], rn[bi, hi], 1)


def test_select_exact_ties():
    """Small-integer keys and dyadic queries make every score exact in fp32 and
    float64, with many exact ties: the sets must then match bit for bit,
    including the lowest-id tie-break."""
    w, cap = small(g=4, L=2000, cap=2048, B=2, H=2, tag="ties")
    rng = np.random.default_rng(7)
    Kf = rng.integers(-2, 3, size=(2, 2, cap, 128)).astype(np.float32)
    Vf = rng.standard_normal((2, 2, cap, 128)).astype(np.float32)
    qf = rng.integers(-1, 2, size=(2, 8, 128)).astype(np.float32)
    K, V, q = W.f32_to_bf16_bits(Kf), W.f32_to_bf16_bits(Vf), W.f32_to_bf16_bits(qf)
    lens = [2000, 1500]
    _, gi, gn, gs, rs, ri, rn, _ = run_select(w, cap, lens, q, sparsity=0.9, min_blocks=3, K=K, V=V)
    for bi in range(2):
        for hi in range(2):
            M = O.num_blocks(lens[bi], 16)
            assert np.array_equal(gs[bi, hi, :M].astype(np.float64), rs[bi, hi])
            assert len(set(rs[bi, hi].tolist())) < M // 2  # plenty of exact ties
            assert list(gi[bi, hi, :gn[bi, hi]]) == list(ri[bi, hi])


@pytest.mark.parametrize("M", [300, 5000, 20000])
def test_select_exact_ties_large(M):
    """Exact ties at several group sizes: the bucket of the n-th largest score
    holds many equal keys, resolved by ranking when it is small and by a third
    digit pass when it is not; the lowest ids must win either way."""
    L = M * 16 - 7
    w = W.TINY_4K.with_(batch=1, num_q_heads=4, num_kv_heads=1, seq_len=L, min_tokens=0,
                        seed_tag=f"ties{M}")
    rng = np.random.default_rng(M)
    Kf = rng.integers(-2, 3, size=(1, 1, M * 16, 128)).astype(np.float32)
    Vf = np.zeros((1, 1, M * 16, 128), dtype=np.float32)
    qf = rng.integers(-1, 2, size=(1, 4, 128)).astype(np.float32)
    K, V, q = W.f32_to_bf16_bits(Kf), W.f32_to_bf16_bits(Vf), W.f32_to_bf16_bits(qf)
    _, gi, gn, gs, rs, ri, rn, _ = run_select(w, M * 16, [L], q, sparsity=0.93, min_blocks=0,
                                              K=K, V=V)
    assert O.num_blocks(L, 16) == M
    assert np.array_equal(gs[0, 0, :M].astype(np.float64), rs[0, 0])
    assert len(set(rs[0, 0].tolist())) < M // 4
    assert list(gi[0, 0, :gn[0, 0]]) == list(ri[0, 0])


@pytest.mark.parametrize("M", [2049, 2600, 3500, 4096, 4097, 8193, 12000, 16400, 20000, 28000, 32768,
                               32800])
def test_select_large_groups(M):
    """Group sizes that take each per-thread key count of the fused selection:
    up to 4096 blocks in 128-block ranges the 512-thread workgroups (2049,
    2600, 3500 and 4096 take 5, 6, 8 and 8 keys per thread), from 4097 the
    1024-thread ones (just past 4 keys per thread, up to the 32768-key
    budget); 32800 blocks exceed it, so scoring and the standalone top-n
    kernel run instead."""
    w = W.TINY_4K.with_(batch=1, num_q_heads=4, num_kv_heads=1, seq_len=M * 16 - 5,
                        min_tokens=0, seed_tag=f"large{M}")
    cap = M * 16
    q = W.decode_query(w)
    _, gi, gn, gs, rs, ri, rn, _ = run_select(w, cap, [w.seq_len], q, sparsity=0.97)
    assert O.num_blocks(w.seq_len, 16) == M
    assert gn[0, 0] == rn[0, 0] == O.num_selected(M, 0.97, 0, 1)
    assert max_abs_err(gs[0, 0, :M], rs[0, 0]) <= 1e-3
    check_selection(gi[0, 0, :gn[0, 0]], ri[0, 0], rs[0, 0], rn[0, 0], 1)


def test_select_reused_workspace():
    """Consecutive selections on one workspace (tickets and key histograms must
    return to zero after each call)."""
    w, cap = small(g=4, L=3000, cap=3072, B=2, H=2, tag="selws")
    lens = [3000, 2500]
    K, V = W.kv_cache(w, capacity=cap)
    cache = make_cache(K, V, 16)
    lt = i32(lens)
    R.block_summarize(cache, lt)
    ws = R.Workspace(dev())
    st = O.DecodeState(O.bf16_to_f64(K), O.bf16_to_f64(V), lens, 16)
    for step, s_ in enumerate([0.9, 0.5, 0.95, 0.8]):
        q = W.decode_query(w, step)
        idx, ns = R.select_blocks(cache, up(q), lt, 3000, s_, 4, 1, workspace=ws)
        rs, ri, rn = st.select(O.bf16_to_f64(q), s_, 4, 1)
        gi, gn = idx.cpu().numpy(), ns.cpu().numpy()
        for bi in range(2):
            for hi in range(2):
                assert gn[bi, hi] == rn[bi, hi]
                check_selection(gi[bi, hi, :gn[bi, hi]], ri[bi, hi], rs[bi, hi], rn[bi, hi], 1)
    tickets = ws.buf[:16].view(torch.int32).cpu().numpy()
    assert np.all(tickets == 0)


@pytest.mark.parametrize("L", [4800, 80000])
def test_select_window_hint(L):
    """The digit-window hint a call leaves in the workspace must never change
    the result: queries scaled by powers of two (and negated) move the score
    distribution so the hint hits, misses above and misses below; every call
    must equal a call on a fresh workspace and the oracle."""
    w, cap = small(g=4, L=L, cap=L + 64, B=1, H=2, tag=f"win{L}")
    K, V = W.kv_cache(w, capacity=cap)
    cache = make_cache(K, V, 16)
    lt = i32([L])
    R.block_summarize(cache, lt)
    ws = R.Workspace(dev())
    st = O.DecodeState(O.bf16_to_f64(K), O.bf16_to_f64(V), [L], 16)
    q0 = W.bf16_bits_to_f32(W.decode_query(w, 0))
    for scale in [1.0, 1.0, 4.0, 0.25, -1.0, 1.0, 64.0]:
        q = W.f32_to_bf16_bits(q0 * scale)
        idx, ns = R.select_blocks(cache, up(q), lt, L, 0.9, 4, 1, workspace=ws)
        idx2, ns2 = R.select_blocks(cache, up(q), lt, L, 0.9, 4, 1)
        torch.cuda.synchronize()
        assert torch.equal(idx, idx2) and torch.equal(ns, ns2)
        rs, ri, rn = st.select(O.bf16_to_f64(q), 0.9, 4, 1)
        gi, gn = idx.cpu().numpy(), ns.cpu().numpy()
        for hi in range(2):
            assert gn[0, hi] == rn[0, hi]
            check_selection(gi[0, hi, :gn[0, hi]], ri[0, hi], rs[0, hi], rn[0, hi], 1)


@pytest.mark.parametrize("b", [16, 64])
def test_select_window_hint_ragged(b):
    """Repeated calls on one workspace use the digit window the previous
    call left behind: every call must equal a call on a fresh workspace and
    the oracle, over ragged lengths, several workgroups per group, the forced
    local block and a moving score distribution."""
    w, cap = small(g=4, b=b, L=20000, cap=20480, B=3, H=2, tag=f"wl{b}")
    lens = [20000, 13001, 700]
    K, V = W.kv_cache(w, capacity=cap)
    cache = make_cache(K, V, b)
    lt = i32(lens)
    R.block_summarize(cache, lt)
    ws = R.Workspace(dev())
    st = O.DecodeState(O.bf16_to_f64(K), O.bf16_to_f64(V), lens, b)
    q0 = W.bf16_bits_to_f32(W.decode_query(w, 1))
    for scale in [1.0, 1.0, 1.0, 1.25, 1.25, 0.8, 1.0]:
        q = W.f32_to_bf16_bits(q0 * scale)
        idx, ns = R.select_blocks(cache, up(q), lt, max(lens), 0.9, 4, 1, workspace=ws)
        idx2, ns2 = R.select_blocks(cache, up(q), lt, max(lens), 0.9, 4, 1)
        torch.cuda.synchronize()
        assert torch.equal(idx, idx2) and torch.equal(ns, ns2), scale
        rs, ri, rn = st.select(O.bf16_to_f64(q), 0.9, 4, 1)
        gi, gn = idx.cpu().numpy(), ns.cpu().numpy()
        for bi in range(3):
            for hi in range(2):
                assert gn[bi, hi] == rn[bi, hi]
                check_selection(gi[bi, hi, :gn[bi, hi]], ri[bi, hi], rs[bi, hi], rn[bi, hi], 1)


def _window_lists_calls(w, cap, lens, scales, qstep, sparsity=0.9):
    """Calls on one workspace against calls on a fresh one and the oracle;
    returns the workspace's in-window top-n counters."""
    B, H = w.batch, w.num_kv_heads
    K, _ = W.kv_cache(w, capacity=cap)
    cache = make_cache(K, K, 16)
    lt = i32(lens)
    R.block_summarize(cache, lt)
    ws = R.Workspace(dev())
    # The oracle's summaries (Eq. 3) of every group, once: the calls append
    # nothing.
    summ = {(bi, hi): O.block_summaries(O.bf16_to_f64(K[bi, hi]), lens[bi], 16)
            for bi in range(B) for hi in range(H)}
    q0 = W.bf16_bits_to_f32(W.decode_query(w, qstep))
    for scale in scales:
        q = W.f32_to_bf16_bits(q0 * scale)
        idx, ns = R.select_blocks(cache, up(q), lt, max(lens), sparsity, 4, 1, workspace=ws)
        idx2, ns2 = R.select_blocks(cache, up(q), lt, max(lens), sparsity, 4, 1)
        torch.cuda.synchronize()
        assert torch.equal(idx, idx2) and torch.equal(ns, ns2), scale
        qg = O.split_heads(O.bf16_to_f64(q), H)
        gi, gn = idx.cpu().numpy(), ns.cpu().numpy()
        for bi in range(B):
            for hi in range(H):
                kmin, kmax = summ[bi, hi]
                rs = O.block_scores(O.pooled_query(qg[bi, hi]), kmin, kmax)
                rn = O.num_selected(kmin.shape[0], sparsity, 4, 1)
                assert gn[bi, hi] == rn
                check_selection(gi[bi, hi, :gn[bi, hi]], O.select_blocks(rs, rn, 1), rs, rn, 1)
    return select_stats(ws, B, H)


def test_select_window_lists_hint():
    """Groups of 12500 blocks (16 keys per top-n thread, 8 groups of 31 score
    ranges) at sparsity 0.95 (n = 625, so the list entries fit the tail's
    1024 threads): a call whose threshold falls in the window hint takes the
    in-window path, which reads the scoring's above-window bits and in-window
    lists instead of every key (the workspace counter of such calls must
    grow). Queries scaled by powers of two (and negated) make the hint hit,
    miss above and miss below; every call must equal a call on a fresh
    workspace and the oracle."""
    w, cap = small(g=4, b=16, L=200000, cap=200064, B=1, H=8, tag="wlist")
    stats = _window_lists_calls(w, cap, [200000], [1.0, 1.0, 4.0, 0.25, -1.0, 1.0, 64.0, 1.0], 0,
                                sparsity=0.95)
    print(f"in-window top-n calls per group: {stats.ravel().tolist()}", flush=True)
    assert stats.sum() > 0


def test_select_window_lists_ragged():
    """The in-window path over ragged lengths: groups of 12500, 8126 and 44
    blocks (28, 19 and 1 score ranges) with a moving score distribution; at
    sparsity 0.9 the 8126-block groups (n = 813) take the path."""
    w, cap = small(g=4, b=16, L=200000, cap=200064, B=3, H=3, tag="wlong")
    stats = _window_lists_calls(w, cap, [200000, 130001, 700], [1.0, 1.0, 1.0, 1.25, 1.25, 0.8, 2.0, 1.0], 2)
    print(f"in-window top-n calls per group: {stats.ravel().tolist()}", flush=True)
    assert stats[1].sum() > 0


def test_select_planted_blocks_win():
    w = W.TINY_4K.with_(plant_norm=math.sqrt(128), seed_tag="strong")
    q = W.decode_query(w)
    _, gi, gn, *_ = run_select(w, 4096, [4096], q, scores=False)
    for hi in range(w.num_kv_heads):
        planted = set(W.planted_blocks(w, 0, hi).tolist())
        assert planted <= set(gi[0, hi, :gn[0, hi]].tolist())


# --------------------------------------------------------------------- decode

def oracle_select_idx(w, K64, lens, q, sparsity, min_blocks):
    st = O.DecodeState(K64, K64, lens, w.block_size)  # values unused for selection
    _, ri, rn = st.select(O.bf16_to_f64(q), sparsity, min_blocks, w.n_local)
    return ri


@pytest.mark.parametrize("g", [1, 2, 3, 4, 5, 6, 7, 8])
@pytest.mark.parametrize("b", [16, 32, 64])
@pytest.mark.parametrize("splits", [0, 1, 5, 24])
def test_decode_on_oracle_blocks(g, b, splits):
    """Decode on the oracle's selection against the oracle's attention, for
    every group size the library instantiates (g = 1 .. 8); 24 splits take
    the combine spread over g merging splits (one head each)."""
    w, cap = small(g=g, b=b, tag="dec")
    lens = [1000, 777]
    K, V = W.kv_cache(w, capacity=cap)
    q = W.decode_query(w)
    K64, V64 = O.bf16_to_f64(K), O.bf16_to_f64(V)
    ri = oracle_select_idx(w, K64, lens, q, 0.8, 4)
    n_cap = max(len(v) for v in ri.values()) + 3
    idx, ns = padded_idx(ri, 2, 2, n_cap)
    cache = make_cache(K, V, b)
    out, lse = R.sparse_decode(cache, up(q), i32(lens), i32(idx), i32(ns), num_splits=splits)
    torch.cuda.synchronize()
    st = O.DecodeState(K64, V64, lens, b)
    ref_o, ref_l = st.attend(O.bf16_to_f64(q), ri, w.sm_scale)
    assert max_abs_err(out.cpu().numpy(), ref_o) <= TOL
    assert max_abs_err(lse.cpu().numpy(), ref_l) <= TOL


def test_decode_all_blocks_is_dense():
    w, cap = small(g=4, tag="dense")
    lens = [1000, 777]
    K, V = W.kv_cache(w, capacity=cap)
    q = W.decode_query(w)
    all_idx = {(bi, hi): list(range(O.num_blocks(lens[bi], 16))) for bi in range(2) for hi in range(2)}
    idx, ns = padded_idx(all_idx, 2, 2, 63)
    cache = make_cache(K, V, 16)
    out, lse = R.sparse_decode(cache, up(q), i32(lens), i32(idx), i32(ns))
    torch.cuda.synchronize()
    K64, V64, q64 = O.bf16_to_f64(K), O.bf16_to_f64(V), O.bf16_to_f64(q)
    for bi in range(2):
        for hi in range(2):
            ro, rl = O.dense_attend(q64[bi, 4 * hi:4 * hi + 4], K64[bi, hi], V64[bi, hi], lens[bi],
                                    w.sm_scale)
            assert max_abs_err(out[bi, 4 * hi:4 * hi + 4].cpu().numpy(), ro) <= TOL
            assert max_abs_err(lse[bi, 4 * hi:4 * hi + 4].cpu().numpy(), rl) <= TOL


@pytest.mark.parametrize("splits", [9, 20])
def test_decode_edge_cases(splits):
    """Empty selection, a single valid token, unsorted ids, ids out of range,
    and more splits than chunks (empty splits; 20 splits take the combine
    spread over the g merging splits, whose all-empty heads must give 0 and
    -inf)."""
    w, cap = small(g=4, L=40, cap=64, B=4, H=1, tag="edge")
    lens = [40, 1, 33, 40]
    K, V = W.kv_cache(w, capacity=cap, garbage=1e4)
    q = W.decode_query(w)
    ids = {(0, 0): [], (1, 0): [0], (2, 0): [2, 0], (3, 0): [1, 7, -1, 2]}
    idx, ns = padded_idx(ids, 4, 1, 4)
    cache = make_cache(K, V, 16)
    out, lse = R.sparse_decode(cache, up(q), i32(lens), i32(idx), i32(ns), num_splits=splits)
    torch.cuda.synchronize()
    o, l = out.cpu().numpy(), lse.cpu().numpy()
    K64, V64, q64 = O.bf16_to_f64(K), O.bf16_to_f64(V), O.bf16_to_f64(q)
    assert np.all(o[0] == 0) and np.all(np.isneginf(l[0]))
    assert max_abs_err(o[1], np.repeat(V64[1, 0, :1], 4, axis=0)) <= 1e-6
    ro, rl = O.sparse_attend(q64[2], K64[2, 0], V64[2, 0], 33, [0, 2], 16, w.sm_scale)
    assert max_abs_err(o[2], ro) <= TOL and max_abs_err(l[2], rl) <= TOL
    ro, rl = O.sparse_attend(q64[3], K64[3, 0], V64[3, 0], 40, [1, 2], 16, w.sm_scale)
    assert max_abs_err(o[3], ro) <= TOL and max_abs_err(l[3], rl) <= TOL


def test_decode_reused_workspace_many_splits():
    """Consecutive calls on one workspace with different queries, block sets
    and split counts (one merging split, and from 16 splits one per query
    head): each call's merging splits must merge only that call's partials
    (ready flags tagged with the call count and the split count, which
    moves the flags' layout), leave the merge counters at zero and count the
    merged calls of every group."""
    w, cap = small(g=4, L=2000, cap=2048, tag="reuse")
    lens = [2000, 1985]
    K, V = W.kv_cache(w, capacity=cap)
    K64, V64 = O.bf16_to_f64(K), O.bf16_to_f64(V)
    cache = make_cache(K, V, 16)
    ws = R.Workspace(dev())
    # Sized once for the largest call (a growing workspace is reallocated and
    # cleared, which would restart the call counts).
    ws.get(R.lib().resa_decode_workspace_size(2, 2, 8, 125, 16, 128))
    st = O.DecodeState(K64, V64, lens, 16)
    calls = []
    for step, (s, S) in enumerate([(0.5, 7), (0.9, 32), (0.8, 64), (0.95, 3), (0.5, 128), (0.9, 1),
                                   (0.8, 33)]):
        q = W.decode_query(w, step)
        ri = oracle_select_idx(w, K64, lens, q, s, 4)
        idx, ns = padded_idx(ri, 2, 2, 125)
        out, lse = R.sparse_decode(cache, up(q), i32(lens), i32(idx), i32(ns), num_splits=S,
                                   workspace=ws)
        calls.append((out.clone(), lse.clone(), q, ri))
    torch.cuda.synchronize()
    for out, lse, q, ri in calls:
        ro, rl = st.attend(O.bf16_to_f64(q), ri, w.sm_scale)
        assert max_abs_err(out.cpu().numpy(), ro) <= TOL
        assert max_abs_err(lse.cpu().numpy(), rl) <= TOL
    words = ws.buf[:32].view(torch.int32).cpu().numpy()
    assert np.all(words[:4] == 0)  # tickets
    assert np.all(words[4:8] == 6)  # merged calls: every call but the single-split one


def test_decode_deterministic():
    w, cap = small(g=4, tag="det")
    lens = [1000, 999]
    K, V = W.kv_cache(w, capacity=cap)
    q = W.decode_query(w)
    cache = make_cache(K, V, 16)
    lt = i32(lens)
    R.block_summarize(cache, lt)
    idx, ns = R.select_blocks(cache, up(q), lt, 1000, 0.9, 4, 1)
    a, la = R.sparse_decode(cache, up(q), lt, idx, ns)
    idx2, ns2 = R.select_blocks(cache, up(q), lt, 1000, 0.9, 4, 1)
    b, lb = R.sparse_decode(cache, up(q), lt, idx2, ns2)
    torch.cuda.synchronize()
    assert torch.equal(idx, idx2) and torch.equal(a, b) and torch.equal(la, lb)


def test_decode_tagged_flags_many_calls():
    """Forty calls on one workspace, cycling through split counts that move
    the ready flags' layout (and through the single merger and the spread
    combine): every call is bit-identical to the same call on a freshly
    zeroed workspace, so no flag of an earlier call is ever taken for one of
    the current call, and the per-group call counts advance once per call."""
    w, cap = small(g=4, L=2000, cap=2048, B=3, H=2, tag="tags")
    lens = [2000, 1500, 1999]
    K, V = W.kv_cache(w, capacity=cap)
    cache = make_cache(K, V, 16)
    lt = i32(lens)
    R.block_summarize(cache, lt)
    ws = R.Workspace(dev())
    ws.get(R.lib().resa_decode_workspace_size(3, 2, 8, 125, 16, 64))
    splits = [16, 24, 3, 32, 33, 64, 17, 4]
    for call in range(40):
        q = W.decode_query(w, call)
        idx, ns = R.select_blocks(cache, up(q), lt, 2000, 0.5, 4, 1)
        S = splits[call % len(splits)]
        a, la = R.sparse_decode(cache, up(q), lt, idx, ns, num_splits=S, workspace=ws)
        b, lb = R.sparse_decode(cache, up(q), lt, idx, ns, num_splits=S, workspace=R.Workspace(dev()))
        torch.cuda.synchronize()
        assert torch.equal(a, b) and torch.equal(la, lb), (call, S)
    words = ws.buf[:48].view(torch.int32).cpu().numpy()
    assert np.all(words[:6] == 0)  # tickets
    assert np.all(words[6:12] == 40)  # merged calls


@pytest.mark.parametrize("b,n_local,M", [(16, 1, 40), (16, 0, 40), (32, 1, 40), (64, 0, 40),
                                         (16, 1, 12500), (16, 1, 33000)])
def test_append_select_matches_separate(b, n_local, M):
    """resa_append_select == resa_append_kv then resa_select_blocks, bit for
    bit: ids, counts, scores, cache rows, summaries and lengths, over three
    steps with appends that open a block and appends inside one, and the ids
    equal to a selection on a fresh workspace (no window hint) of the same
    cache (M = 12500 with 8 kv heads takes the in-window top-n path from the
    second step on: at sparsity 0.95 its n = 625 list entries fit the tail's
    1024 threads, and the workspace counters of such calls must grow; M = 33000
    the standalone top-n kernel)."""
    B = 3 if M < 1000 else 1
    H, g = (8 if M == 12500 else 2), 4
    sp = 0.95 if M == 12500 else 0.9
    cap = M * b
    rng = np.random.default_rng(b * 100 + n_local + M)
    lens0 = [cap - 3 * b, cap // 2 - 1, cap // 3 + 5][:B]
    Kf = rng.standard_normal((B, H, cap, 128)).astype(np.float32)
    Vf = rng.standard_normal((B, H, cap, 128)).astype(np.float32)
    K, V = W.f32_to_bf16_bits(Kf), W.f32_to_bf16_bits(Vf)
    del Kf, Vf
    c1 = make_cache(K, V, b, sentinel=False)
    c2 = make_cache(K, V, b, sentinel=False)
    l1, l2 = i32(lens0), i32(lens0)
    R.block_summarize(c1, l1)
    R.block_summarize(c2, l2)
    ws1, ws2 = R.Workspace(dev()), R.Workspace(dev())
    bound = max(lens0)
    for step in range(3):
        kn = W.f32_to_bf16_bits(rng.standard_normal((B, H, 128)).astype(np.float32))
        vn = W.f32_to_bf16_bits(rng.standard_normal((B, H, 128)).astype(np.float32))
        q = W.f32_to_bf16_bits(rng.standard_normal((B, H * g, 128)).astype(np.float32))
        mseq = -(-(bound + 1) // b)
        n_cap = R.num_selected(mseq, sp, 2, n_local)
        s1 = torch.full((B, H, mseq), float("nan"), device=dev())
        s2 = torch.full((B, H, mseq), float("nan"), device=dev())
        R.append_kv(c1, up(kn), up(vn), l1, bound)
        i1, n1 = R.select_blocks(c1, up(q), l1, bound + 1, sp, 2, n_local, n_cap=n_cap,
                                 scores_out=s1, workspace=ws1)
        i2, n2 = R.append_select(c2, up(kn), up(vn), up(q), l2, bound, sp, 2, n_local,
                                 n_cap=n_cap, scores_out=s2, workspace=ws2)
        i3, n3 = R.select_blocks(c2, up(q), l2, bound + 1, sp, 2, n_local, n_cap=n_cap)
        torch.cuda.synchronize()
        assert torch.equal(l1, l2)
        assert torch.equal(n1, n2) and torch.equal(i1, i2)
        assert torch.equal(n3, n2) and torch.equal(i3, i2)
        assert torch.equal(s1.isnan(), s2.isnan())
        assert torch.equal(torch.nan_to_num(s1), torch.nan_to_num(s2))
        bound += 1
    assert l2.cpu().tolist() == [x + 3 for x in lens0]
    if M == 12500:
        for ws in (ws1, ws2):
            assert select_stats(ws, B, H).sum() > 0, "the in-window top-n path was not taken"
    for name in ("k", "v", "kmin", "kmax"):
        assert torch.equal(getattr(c1, name), getattr(c2, name)), name


# -------------------------------------------------------------------- rectify

@pytest.mark.parametrize("g,f", [(4, 16), (4, 1), (7, 32), (8, 32), (2, 64), (1, 16), (3, 32), (5, 16),
                                 (6, 8)])
def test_rectify_vs_oracle(g, f):
    w, cap = small(g=g, L=300, cap=320, tag="rect")
    lens = [300, 257]
    K, V = W.kv_cache(w, capacity=cap)
    K0 = K.copy()
    cache = make_cache(K, V, 16, sentinel=False)
    lt = i32(lens)
    R.block_summarize(cache, lt)
    base_k = np.stack([np.stack([K[bi, hi, lens[bi] - f:lens[bi]] for hi in range(2)]) for bi in range(2)])
    base_v = np.stack([np.stack([V[bi, hi, lens[bi] - f:lens[bi]] for hi in range(2)]) for bi in range(2)])
    qf, kf, vf = W.rectify_inputs(w, 3, base_k, base_v, f)
    out, lse = R.dense_rectify(cache, up(qf), up(kf), up(vf), lt, 300)
    torch.cuda.synchronize()
    st = O.DecodeState(O.bf16_to_f64(K), O.bf16_to_f64(V), lens, 16)
    ro, rl = st.rectify(O.bf16_to_f64(qf), O.bf16_to_f64(kf), O.bf16_to_f64(vf), f, w.sm_scale)
    eo, el = max_abs_err(out.cpu().numpy(), ro), max_abs_err(lse.cpu().numpy(), rl)
    print(f"rectify g={g} f={f}: max |dO| {eo:.2e}, max |dlse| {el:.2e}")
    assert eo <= TOL and el <= TOL
    gk = down(cache.k)
    for bi in range(2):
        L = lens[bi]
        assert np.array_equal(gk[bi, :, L - f:L], kf[bi])
        assert np.array_equal(gk[bi, :, :L - f], K0[bi, :, :L - f])
        assert np.array_equal(gk[bi, :, L:], K0[bi, :, L:])
        M = O.num_blocks(L, 16)
        assert np.array_equal(O.bf16_to_f64(down(cache.kmin)[bi, :, :M]), st.kmin[bi, :, :M])
        assert np.array_equal(O.bf16_to_f64(down(cache.kmax)[bi, :, :M]), st.kmax[bi, :, :M])


@pytest.mark.parametrize("g,f,lens,cap", [
    (4, 32, [2000, 1500], 2048),    # decode-time window: 4-wave workgroups, several key splits
    (4, 300, [1000, 777], 1024),    # long window: 8-wave workgroups
])
def test_rectify_large_and_tiny_v(g, f, lens, cap):
    """Rectification is finite and within 2e-3 of the oracle, scaled per head
    dimension d by max(1, max |V[:, d]|), for every finite bf16 value:
    planted V entries of +-3e38, 1e5 and 7e4 (above the fp16 range, at the
    first key of a split, inside a tile and inside the rewritten window) and
    of 1e-7 (below fp16's normal range), next to N(0, 1) dimensions, which
    stay within 2e-3 absolutely."""
    w, cap = small(g=g, L=max(lens), cap=cap, tag=f"bigv{f}")
    K, V = W.kv_cache(w, capacity=cap)
    cache_k = K
    bits = lambda x: int(W.f32_to_bf16_bits(np.array([x], dtype=np.float32))[0])
    V = V.copy()
    # (sequence, kv head, row, dim, value): rows below L - f sit in the cache,
    # rows at or past it in the rewritten window (planted into v_f below).
    plants = [(0, 0, 3, 5, 3e38), (0, 0, 512 + 5, 5, -2.5e38), (0, 0, 700, 17, 1e5),
              (0, 1, 0, 100, -1e5), (0, 1, 1200, 101, 7e4), (1, 0, 64, 9, 3.3e38),
              (1, 1, 400, 33, 1e5), (0, 0, 900, 40, 1e-7), (1, 1, 20, 41, -1e-7)]
    win = [(0, 0, 2, 6, 3e38), (1, 1, f - 1, 17, -1e5), (0, 1, 0, 70, 6e4), (1, 0, 5, 42, 1e-7)]
    for bi, hi, row, d, x in plants:
        if row < lens[bi] - f:
            V[bi, hi, row, d] = bits(x)
    cache = make_cache(cache_k, V, 16, sentinel=False)
    lt = i32(lens)
    R.block_summarize(cache, lt)
    base_k = np.stack([np.stack([K[bi, hi, lens[bi] - f:lens[bi]] for hi in range(2)]) for bi in range(2)])
    base_v = np.stack([np.stack([V[bi, hi, lens[bi] - f:lens[bi]] for hi in range(2)]) for bi in range(2)])
    qf, kf, vf = W.rectify_inputs(w, 9, base_k, base_v, f)
    vf = vf.copy()
    for bi, hi, r, d, x in win:
        vf[bi, hi, r, d] = bits(x)
    out, lse = R.dense_rectify(cache, up(qf), up(kf), up(vf), lt, max(lens))
    torch.cuda.synchronize()
    go, gl = out.cpu().numpy(), lse.cpu().numpy()
    assert np.all(np.isfinite(go)), "non-finite rectify output"
    st = O.DecodeState(O.bf16_to_f64(K), O.bf16_to_f64(V), lens, 16)
    ro, rl = st.rectify(O.bf16_to_f64(qf), O.bf16_to_f64(kf), O.bf16_to_f64(vf), f, w.sm_scale)
    assert max_abs_err(gl, rl) <= TOL
    for bi in range(2):
        for hi in range(2):
            L = lens[bi]
            vmax = np.abs(st.V[bi, hi, :L]).max(axis=0)          # [D], after the rewrite
            scale = np.maximum(1.0, vmax)
            heads = slice(hi * g, (hi + 1) * g)
            err = np.abs(go[bi, heads] - ro[bi, heads]) / scale  # [g, f, D]
            worst = float(err.max())
            print(f"large V g={g} f={f} seq {bi} head {hi}: max |dO| / max(1, |V_d|) {worst:.2e}",
                  flush=True)
            assert worst <= TOL


def test_rectify_workspace_sized_for_longer_context():
    """A workspace sized once (C ABI) for the longest context serves a shorter
    call that splits its keys more finely: one group and one query row take
    512 key splits of 128 keys at L = 65536, where a 65600-token call takes
    342 splits of 192 keys; the call must succeed and match the oracle."""
    import ctypes as C
    g, f, L, Lmax = 1, 1, 65536, 65600
    w, cap = small(g=g, L=L, cap=Lmax + 64, B=1, H=1, tag="rws")
    K, V = W.kv_cache(w, capacity=cap)
    cache = make_cache(K, V, 16, sentinel=False)
    lt = i32([L])
    R.block_summarize(cache, lt)
    qf, kf, vf = W.rectify_inputs(w, 4, K[:, :, L - f:L], V[:, :, L - f:L], f)
    lib = R.lib()
    nbytes = lib.resa_rectify_workspace_size(1, 1, g, f, Lmax)
    assert nbytes >= lib.resa_rectify_workspace_size(1, 1, g, f, L) > 0
    ws = torch.zeros(nbytes, dtype=torch.uint8, device=dev())
    q_d, k_d, v_d = up(qf), up(kf), up(vf)
    out = torch.empty((1, g, f, 128), dtype=torch.float32, device=dev())
    lse = torch.empty((1, g, f), dtype=torch.float32, device=dev())
    d = cache.desc()
    rc = lib.resa_dense_rectify(C.byref(d), q_d.data_ptr(), k_d.data_ptr(), v_d.data_ptr(), g, f,
                                lt.data_ptr(), None, L, C.c_float(w.sm_scale), out.data_ptr(),
                                lse.data_ptr(), 1, ws.data_ptr(), C.c_size_t(nbytes),
                                C.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == 0, lib.resa_last_error()
    torch.cuda.synchronize()
    st = O.DecodeState(O.bf16_to_f64(K), O.bf16_to_f64(V), [L], 16)
    ro, rl = st.rectify(O.bf16_to_f64(qf), O.bf16_to_f64(kf), O.bf16_to_f64(vf), f, w.sm_scale)
    eo, el = max_abs_err(out.cpu().numpy(), ro), max_abs_err(lse.cpu().numpy(), rl)
    print(f"rectify on a workspace sized for {Lmax}: max |dO| {eo:.2e}, max |dlse| {el:.2e}")
    assert eo <= TOL and el <= TOL


def test_rectify_tiny4k_full():
    """The tiny 4K layer: f = 16 rows, causal over the whole 4096 cache."""
    w = W.TINY_4K
    K, V = W.kv_cache(w)
    cache = make_cache(K, V, 16, sentinel=False)
    lt = i32([4096])
    R.block_summarize(cache, lt)
    qf, kf, vf = W.rectify_inputs(w, 0, K[:, :, 4080:], V[:, :, 4080:], 16)
    out, lse = R.dense_rectify(cache, up(qf), up(kf), up(vf), lt, 4096)
    torch.cuda.synchronize()
    st = O.DecodeState(O.bf16_to_f64(K), O.bf16_to_f64(V), [4096], 16)
    ro, rl = st.rectify(O.bf16_to_f64(qf), O.bf16_to_f64(kf), O.bf16_to_f64(vf), 16, w.sm_scale)
    eo, el = max_abs_err(out.cpu().numpy(), ro), max_abs_err(lse.cpu().numpy(), rl)
    print(f"rectify tiny4k: max |dO| {eo:.2e}, max |dlse| {el:.2e}")
    assert eo <= TOL and el <= TOL


@pytest.mark.parametrize("g,f,lens,cap", [
    (4, 300, [1000, 777], 1024),     # a prompt chunk after a cached prefix
    (4, 512, [512, 512], 512),       # whole-prompt prefill, f = L
    (8, 640, [640, 400], 704),       # prefill; the short sequence is left as it is
    (2, 2080, [2100, 2080], 2112),   # long chunk: many query blocks, causal key clamp
])
def test_rectify_prefill(g, f, lens, cap):
    """Chunked and whole-prompt prefill through the rectification call: the
    chunk's rows are written, its queries attend causally over the cache and
    themselves, and every touched block summary is rebuilt. Sequences shorter
    than f are untouched (zero rows, lse -inf)."""
    w, cap = small(g=g, L=max(lens), cap=cap, tag=f"prefill{f}")
    K, V = W.kv_cache(w, capacity=cap)
    K0 = K.copy()
    cache = make_cache(K, V, 16, sentinel=False)
    lt = i32(lens)
    if f < min(lens):
        R.block_summarize(cache, lt)
    kmin0, kmax0 = down(cache.kmin), down(cache.kmax)
    base_k = np.stack([np.stack([K[bi, hi, max(lens[bi] - f, 0):max(lens[bi] - f, 0) + f]
                                 for hi in range(2)]) for bi in range(2)])
    base_v = np.stack([np.stack([V[bi, hi, max(lens[bi] - f, 0):max(lens[bi] - f, 0) + f]
                                 for hi in range(2)]) for bi in range(2)])
    qf, kf, vf = W.rectify_inputs(w, 5, base_k, base_v, f)
    out, lse = R.dense_rectify(cache, up(qf), up(kf), up(vf), lt, max(lens))
    torch.cuda.synchronize()
    go, gl = out.cpu().numpy(), lse.cpu().numpy()
    gk = down(cache.k)
    qg = O.split_heads(O.bf16_to_f64(qf), 2)
    Kd, Vd = O.bf16_to_f64(K), O.bf16_to_f64(V)
    for bi in range(2):
        L = lens[bi]
        if L < f:
            assert np.all(go[bi] == 0) and np.all(np.isneginf(gl[bi]))
            assert np.array_equal(gk[bi], K0[bi])
            assert np.array_equal(down(cache.kmin)[bi], kmin0[bi])
            continue
        for hi in range(2):
            M = O.num_blocks(L, 16)
            kmin, kmax = O.block_summaries(Kd[bi, hi], L, 16)
            ro, rl = O.rectify_group(qg[bi, hi], Kd[bi, hi].copy(), Vd[bi, hi].copy(), kmin, kmax,
                                     L, f, 16, w.sm_scale, O.bf16_to_f64(kf[bi, hi]),
                                     O.bf16_to_f64(vf[bi, hi]))
            eo = max_abs_err(go[bi, hi * g:(hi + 1) * g], ro)
            el = max_abs_err(gl[bi, hi * g:(hi + 1) * g], rl)
            print(f"prefill g={g} f={f} seq {bi} head {hi}: |dO| {eo:.2e} |dlse| {el:.2e}",
                  flush=True)
            assert eo <= TOL and el <= TOL
            assert np.array_equal(gk[bi, hi, L - f:L], kf[bi, hi])
            assert np.array_equal(gk[bi, hi, :L - f], K0[bi, hi, :L - f])
            assert np.array_equal(gk[bi, hi, L:], K0[bi, hi, L:])
            lo = (L - f) // 16
            assert np.array_equal(O.bf16_to_f64(down(cache.kmin)[bi, hi, lo:M]), kmin[lo:M])
            assert np.array_equal(O.bf16_to_f64(down(cache.kmax)[bi, hi, lo:M]), kmax[lo:M])


# ---------------------------------------------------------------- decode loop

@pytest.mark.parametrize("fused,paged", [(False, False), (True, False), (True, True)])
def test_decode_loop_small(fused, paged):
    """Kernel-level Alg. 1 loop (append, select, decode; rectify every f steps)
    on a reduced copy of the 64K batch-8 workload (outlier key channels);
    `fused` runs the append and the selection as one resa_append_select;
    `paged` keeps K and V in a shuffled page pool behind a block table."""
    w = W.LONG_64K.with_(batch=2, num_q_heads=8, num_kv_heads=2, seq_len=600, min_tokens=64,
                         seed_tag="loop")
    f, steps, cap = 16, 40, 704
    K, V = W.kv_cache(w, capacity=cap)
    lens = [600, 555]
    if paged:
        cache = make_paged_cache(K, V, 16, [x + steps for x in lens], seed=11, sentinel=False)
    else:
        cache = make_cache(K, V, 16, sentinel=False)
    lt = i32(lens)
    R.block_summarize(cache, lt)
    st = O.DecodeState(O.bf16_to_f64(K), O.bf16_to_f64(V), lens, 16)
    swaps = 0
    for step in range(steps):
        kn, vn = W.decode_kv(w, step)
        q = W.decode_query(w, step)
        if fused:
            idx, ns = R.append_select(cache, up(kn), up(vn), up(q), lt, max(st.L), w.sparsity,
                                      w.min_blocks, 1)
            st.append(O.bf16_to_f64(kn), O.bf16_to_f64(vn))
        else:
            R.append_kv(cache, up(kn), up(vn), lt, max(st.L))
            st.append(O.bf16_to_f64(kn), O.bf16_to_f64(vn))
            idx, ns = R.select_blocks(cache, up(q), lt, max(st.L), w.sparsity, w.min_blocks, 1)
        out, _ = R.sparse_decode(cache, up(q), lt, idx, ns)
        rs, ri, rn = st.select(O.bf16_to_f64(q), w.sparsity, w.min_blocks, 1)
        ro, _ = st.attend(O.bf16_to_f64(q), ri, w.sm_scale)
        gi, gn, go = idx.cpu().numpy(), ns.cpu().numpy(), out.cpu().numpy()
        for bi in range(2):
            for hi in range(2):
                s = check_selection(gi[bi, hi, :gn[bi, hi]], ri[bi, hi], rs[bi, hi], rn[bi, hi], 1)
                swaps += s
                if s == 0:
                    assert max_abs_err(go[bi, 4 * hi:4 * hi + 4], ro[bi, 4 * hi:4 * hi + 4]) <= TOL
                else:
                    # Near-tie swap: the attention on the GPU's own set.
                    q64 = O.bf16_to_f64(q)[bi, 4 * hi:4 * hi + 4]
                    own, _ = O.sparse_attend(q64, st.K[bi, hi], st.V[bi, hi], st.L[bi],
                                             gi[bi, hi, :gn[bi, hi]], 16, w.sm_scale)
                    assert max_abs_err(go[bi, 4 * hi:4 * hi + 4], own) <= TOL
        if (step + 1) % f == 0:
            # The window is the f rows appended since the last rectification.
            rows = [W.decode_kv(w, s) for s in range(step - f + 1, step + 1)]
            lastk = np.stack([r[0] for r in rows], axis=2)
            lastv = np.stack([r[1] for r in rows], axis=2)
            qf, kf, vf = W.rectify_inputs(w, step, lastk, lastv, f)
            rout, _ = R.dense_rectify(cache, up(qf), up(kf), up(vf), lt, max(st.L))
            rr, _ = st.rectify(O.bf16_to_f64(qf), O.bf16_to_f64(kf), O.bf16_to_f64(vf), f, w.sm_scale)
            assert max_abs_err(rout.cpu().numpy(), rr) <= TOL
    torch.cuda.synchronize()
    assert lt.cpu().tolist() == st.L
    assert swaps <= 4
    if paged:
        gk, gv = unpage(cache, st.L)
        for bi in range(2):
            L = st.L[bi]
            assert np.array_equal(O.bf16_to_f64(gk[bi, :, :L]), st.K[bi, :, :L])
            assert np.array_equal(O.bf16_to_f64(gv[bi, :, :L]), st.V[bi, :, :L])


# ------------------------------------------------------------------ HIP graph

def test_graph_replay_matches_eager():
    """One decode step (fused append + selection, then sparse decode) recorded
    once in a HIP graph and replayed for several steps, with eager work and
    synchronisations between the replays, gives bit-identical selections,
    outputs, lengths and caches to the same calls made eagerly."""
    w = W.LONG_64K.with_(batch=2, num_q_heads=8, num_kv_heads=2, seq_len=600, min_tokens=64,
                         seed_tag="graph")
    b, cap, steps = 16, 704, 4
    B, H, Hq = 2, 2, 8
    K, V = W.kv_cache(w, capacity=cap)
    c1 = make_cache(K, V, b, sentinel=False)
    c2 = make_cache(K, V, b, sentinel=False)
    lens0 = [600, 555]
    l1, l2 = i32(lens0), i32(lens0)
    R.block_summarize(c1, l1)
    R.block_summarize(c2, l2)
    bound = max(lens0) + steps  # one host bound that holds for every step
    mseq = -(-(bound + 1) // b)
    n_cap = R.num_selected(mseq, w.sparsity, w.min_blocks, w.n_local)
    splits = R.decode_num_splits(B, H, n_cap, b)
    d = dev()
    bf = torch.bfloat16
    kn_s = torch.zeros((B, H, 128), dtype=bf, device=d)
    vn_s = torch.zeros((B, H, 128), dtype=bf, device=d)
    q_s = torch.zeros((B, Hq, 128), dtype=bf, device=d)
    idx2 = torch.empty((B, H, n_cap), dtype=torch.int32, device=d)
    ns2 = torch.empty((B, H), dtype=torch.int32, device=d)
    out2 = torch.empty((B, Hq, 128), dtype=torch.float32, device=d)
    lse2 = torch.empty((B, Hq), dtype=torch.float32, device=d)
    wss = [R.Workspace(d) for _ in range(4)]
    lib = R.lib()
    for ws_sel, ws_dec in (wss[:2], wss[2:]):
        ws_sel.get(lib.resa_select_workspace_size(B, H, bound + 1, b))
        ws_dec.get(lib.resa_decode_workspace_size(B, H, Hq, n_cap, b, splits))
    torch.cuda.synchronize()

    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(graph, stream=side):
        R.append_select(c2, kn_s, vn_s, q_s, l2, bound, w.sparsity, w.min_blocks, w.n_local,
                        n_cap=n_cap, block_idx=idx2, num_sel=ns2, workspace=wss[0])
        R.sparse_decode(c2, q_s, l2, idx2, ns2, num_splits=splits, out=out2, lse=lse2,
                        workspace=wss[1])
    torch.cuda.synchronize()
    for step in range(steps):
        kn, vn = W.decode_kv(w, step)
        q = W.decode_query(w, step)
        kn_s.copy_(up(kn))
        vn_s.copy_(up(vn))
        q_s.copy_(up(q))
        graph.replay()
        torch.cuda.synchronize()
        i1, n1 = R.append_select(c1, up(kn), up(vn), up(q), l1, bound, w.sparsity, w.min_blocks,
                                 w.n_local, n_cap=n_cap, workspace=wss[2])
        o1, s1 = R.sparse_decode(c1, up(q), l1, i1, n1, num_splits=splits, workspace=wss[3])
        torch.cuda.synchronize()
        print(f"graph replay {step}: n_sel {ns2.cpu().tolist()}", flush=True)
        assert torch.equal(l1, l2)
        assert torch.equal(n1, ns2) and torch.equal(i1, idx2)
        assert torch.equal(o1, out2) and torch.equal(s1, lse2)
    assert l2.cpu().tolist() == [x + steps for x in lens0]
    for name in ("k", "v", "kmin", "kmax"):
        assert torch.equal(getattr(c1, name), getattr(c2, name)), name


def test_rectify_graph_replay_matches_eager():
    """Rectification (row rewrite, summary refresh, key-split attention and
    the split merge) recorded once in a HIP graph and replayed with new
    re-encoded rows each time, with eager work and synchronisations between
    the replays, gives bit-identical outputs, lse, caches and summaries to the
    same calls made eagerly."""
    g, f, B, H = 4, 32, 2, 2
    w, cap = small(g=g, L=2000, cap=2048, B=B, H=H, tag="rgraph")
    lens = [2000, 1500]
    K, V = W.kv_cache(w, capacity=cap)
    c1 = make_cache(K, V, 16, sentinel=False)
    c2 = make_cache(K, V, 16, sentinel=False)
    l1, l2 = i32(lens), i32(lens)
    R.block_summarize(c1, l1)
    R.block_summarize(c2, l2)
    lib = R.lib()
    nbytes = lib.resa_rectify_workspace_size(B, H, g * H, f, max(lens))
    assert nbytes > 0  # several key splits: the merge kernel runs too
    d = dev()
    bf = torch.bfloat16
    q_s = torch.zeros((B, g * H, f, 128), dtype=bf, device=d)
    k_s = torch.zeros((B, H, f, 128), dtype=bf, device=d)
    v_s = torch.zeros((B, H, f, 128), dtype=bf, device=d)
    out2 = torch.empty((B, g * H, f, 128), dtype=torch.float32, device=d)
    lse2 = torch.empty((B, g * H, f), dtype=torch.float32, device=d)
    ws1, ws2 = R.Workspace(d), R.Workspace(d)
    ws1.get(nbytes)
    ws2.get(nbytes)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(graph, stream=side):
        R.dense_rectify(c2, q_s, k_s, v_s, l2, max(lens), out=out2, lse=lse2, workspace=ws2)
    torch.cuda.synchronize()
    for rep in range(3):
        base_k = np.stack([np.stack([K[bi, hi, lens[bi] - f:lens[bi]] for hi in range(H)]) for bi in range(B)])
        base_v = np.stack([np.stack([V[bi, hi, lens[bi] - f:lens[bi]] for hi in range(H)]) for bi in range(B)])
        qf, kf, vf = W.rectify_inputs(w, 20 + rep, base_k, base_v, f)
        q_s.copy_(up(qf))
        k_s.copy_(up(kf))
        v_s.copy_(up(vf))
        graph.replay()
        torch.cuda.synchronize()
        o1, s1 = R.dense_rectify(c1, up(qf), up(kf), up(vf), l1, max(lens), workspace=ws1)
        torch.cuda.synchronize()
        print(f"rectify graph replay {rep}: max |out| {float(out2.abs().max()):.3f}", flush=True)
        assert torch.equal(o1, out2) and torch.equal(s1, lse2)
        for name in ("k", "v", "kmin", "kmax"):
            assert torch.equal(getattr(c1, name), getattr(c2, name)), name
