"""GPU parity of the fused decode step (resa_decode_step): the same
selections, lengths and cache contents as resa_append_select followed by
resa_sparse_decode, outputs equal up to fp32 summation order, and the oracle
within the attention bar; repeated calls on one workspace."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle as O
import paper_2506_04108_amd as R
import workloads as W
from gpu_util import down, i32, make_cache, make_paged_cache, select_stats, up
from oracle.compare import check_selection, max_abs_err

pytestmark = pytest.mark.gpu
TOL = 2e-3
# The step cuts each group's selected chunks into the same splits as
# resa_sparse_decode but sums a split with 8 waves instead of 4: fp32
# rounding order only (values are O(1), sums of a few thousand terms).
REORDER = 2e-5


def clone(cache: R.KVCache) -> R.KVCache:
    return dataclasses.replace(cache, **{f: getattr(cache, f).clone() for f in ("k", "v", "kmin", "kmax")})


def step_error_flag(ws: R.Workspace) -> int:
    """The guard flag of the fused step (word 3 of its workspace): set only if
    a decode split gave up waiting for its group's selection."""
    return int(ws.buf[12:16].view(torch.int32).item())


def run_pair(w, cache, lens, steps, num_splits=0, n_cap=None, keep=None):
    """Runs `steps` decode tokens through resa_decode_step on `cache` and
    through append_select + sparse_decode on a copy; checks them against each
    other every step and yields (step, q, idx, nsel, out) of the fused path.
    `keep` (a dict) receives the step and selection workspaces."""
    ref_cache = clone(cache)
    lt, lr = i32(lens), i32(lens)
    ws_step, ws_sel, ws_dec = R.Workspace(), R.Workspace(), R.Workspace()
    if keep is not None:
        keep.update(step=ws_step, select=ws_sel)
    L = list(lens)
    for step in range(steps):
        kn, vn = W.decode_kv(w, step)
        q = W.decode_query(w, step)
        bound = min(max(L), cache.capacity - 1)  # a full sequence is reached through its device length
        idx, ns, out, lse = R.decode_step(cache, up(kn), up(vn), up(q), lt, bound, w.sparsity,
                                          w.min_blocks, w.n_local, n_cap=n_cap, num_splits=num_splits,
                                          workspace=ws_step)
        ridx, rns = R.append_select(ref_cache, up(kn), up(vn), up(q), lr, bound, w.sparsity,
                                    w.min_blocks, w.n_local, n_cap=idx.shape[-1], workspace=ws_sel)
        rout, rlse = R.sparse_decode(ref_cache, up(q), lr, ridx, rns, num_splits=num_splits,
                                     workspace=ws_dec)
        torch.cuda.synchronize()
        assert step_error_flag(ws_step) == 0
        assert torch.equal(lt, lr)
        assert torch.equal(ns, rns)
        assert torch.equal(idx, ridx)
        assert max_abs_err(out.cpu().numpy(), rout.cpu().numpy()) <= REORDER
        fin = torch.isfinite(rlse)
        assert torch.equal(torch.isfinite(lse), fin)
        assert max_abs_err(lse[fin].cpu().numpy(), rlse[fin].cpu().numpy()) <= REORDER
        L = [min(x + 1, cache.capacity) for x in L]
        yield step, kn, vn, q, idx, ns, out
    torch.cuda.synchronize()
    for f in ("k", "v", "kmin", "kmax"):
        assert torch.equal(getattr(cache, f), getattr(ref_cache, f)), f


@pytest.mark.parametrize("g,b", [(4, 16), (7, 16), (8, 32), (1, 64), (4, 64)])
def test_step_matches_separate_calls(g, b):
    w, cap = W.TINY_4K.with_(batch=3, num_kv_heads=2, num_q_heads=2 * g, seq_len=1500, block_size=b,
                             min_tokens=8 * b, seed_tag=f"step-{g}-{b}"), 2048
    K, V = W.kv_cache(w, capacity=cap)
    lens = [1500, 1111, 37]
    cache = make_cache(K, V, b, sentinel=False)
    R.block_summarize(cache, i32(lens))
    for _ in run_pair(w, cache, lens, steps=6):
        pass


def test_step_window_lists():
    """16 groups of 8200 - 8750 blocks (32 keys per thread of the fused
    step's 512-thread top-n, 31 score ranges of 288 blocks) at sparsity 0.95
    (n = 411 - 438, so the list entries the path needs fit the 512 threads):
    from the second step on, the window hint is set and the fused step's top-n
    takes the in-window path (above-window bits and in-window lists written by
    its score ranges; the workspace counter of such calls must grow), while
    append_select (12 keys per thread) reads every key; the selections must be
    identical and the outputs equal up to summation order."""
    w = W.LONG_64K.with_(batch=2, num_kv_heads=8, num_q_heads=32, seq_len=140000, sparsity=0.95,
                         seed_tag="steplists")
    cap = 140064
    lens = [140000, 131500]
    K, V = W.kv_cache(w, capacity=cap)
    cache = make_cache(K, V, 16, sentinel=False)
    del K, V
    R.block_summarize(cache, i32(lens))
    keep = {}
    for _ in run_pair(w, cache, lens, steps=4, keep=keep):
        pass
    stats = select_stats(keep["step"], 2, 8, step=True)
    print(f"in-window top-n calls per group: {stats.ravel().tolist()}", flush=True)
    assert stats.sum() > 0, "the fused step never took the in-window path"


def test_step_against_oracle_loop():
    """Ten fused steps on one workspace against the oracle's decode loop
    (appends, selections within the near-tie rule, attention within 2e-3),
    a ragged batch with one sequence short enough to keep every block."""
    w = W.LONG_64K.with_(batch=3, num_q_heads=8, num_kv_heads=2, seq_len=900, min_tokens=64,
                         seed_tag="steploop")
    cap = 1024
    lens = [900, 613, 40]
    K, V = W.kv_cache(w, capacity=cap)
    cache = make_cache(K, V, 16, sentinel=False)
    R.block_summarize(cache, i32(lens))
    st = O.DecodeState(O.bf16_to_f64(K), O.bf16_to_f64(V), lens, 16)
    swaps = 0
    for step, kn, vn, q, idx, ns, out in run_pair(w, cache, lens, steps=10):
        st.append(O.bf16_to_f64(kn), O.bf16_to_f64(vn))
        rs, ri, rn = st.select(O.bf16_to_f64(q), w.sparsity, w.min_blocks, 1)
        ro, _ = st.attend(O.bf16_to_f64(q), ri, w.sm_scale)
        gi, gn, go = idx.cpu().numpy(), ns.cpu().numpy(), out.cpu().numpy()
        for bi in range(3):
            for hi in range(2):
                assert gn[bi, hi] == rn[bi, hi]
                s = check_selection(gi[bi, hi, :gn[bi, hi]], ri[bi, hi], rs[bi, hi], rn[bi, hi], 1)
                swaps += s
                if s == 0:
                    assert max_abs_err(go[bi, 4 * hi:4 * hi + 4], ro[bi, 4 * hi:4 * hi + 4]) <= TOL
                else:
                    # Near-tie swap: check the attention on the GPU's own set.
                    q64 = O.bf16_to_f64(q)[bi, 4 * hi:4 * hi + 4]
                    go_ref, _ = O.sparse_attend(q64, st.K[bi, hi], st.V[bi, hi], st.L[bi],
                                                gi[bi, hi, :gn[bi, hi]], 16, w.sm_scale)
                    assert max_abs_err(go[bi, 4 * hi:4 * hi + 4], go_ref) <= TOL
    assert swaps <= 4


def test_step_full_cache_and_splits():
    """A sequence already at capacity is decoded over its stored length and
    left unchanged; explicit split counts (1: the single split writes the
    output directly; 7: uneven parts)."""
    w, cap = W.TINY_4K.with_(batch=2, num_kv_heads=2, num_q_heads=8, seq_len=512, min_tokens=128,
                             seed_tag="stepfull"), 512
    K, V = W.kv_cache(w, capacity=cap)
    for splits in (1, 7):
        cache = make_cache(K, V, 16, sentinel=False)
        lens = [512, 300]
        R.block_summarize(cache, i32(lens))
        # The host bound must stay below capacity, so the full sequence is
        # only reached through the device length.
        gen = run_pair(w, cache, lens, steps=3, num_splits=splits)
        for step, *_ in gen:
            pass


def test_step_paged_matches_contiguous():
    """The fused step on a shuffled page pool gives the same selections and
    outputs as on the contiguous layout (and the same appended rows)."""
    w = W.LONG_64K.with_(batch=2, num_q_heads=8, num_kv_heads=2, seq_len=700, min_tokens=64,
                         seed_tag="steppaged")
    cap, steps = 768, 5
    lens = [700, 650]
    K, V = W.kv_cache(w, capacity=cap)
    flat = make_cache(K, V, 16, sentinel=False)
    paged = make_paged_cache(K, V, 16, [x + steps for x in lens], seed=3, sentinel=False)
    lf, lp = i32(lens), i32(lens)
    R.block_summarize(flat, lf)
    R.block_summarize(paged, lp)
    wf, wp = R.Workspace(), R.Workspace()
    for step in range(steps):
        kn, vn = W.decode_kv(w, step)
        q = W.decode_query(w, step)
        bound = max(lens) + step
        a = R.decode_step(flat, up(kn), up(vn), up(q), lf, bound, w.sparsity, w.min_blocks, 1,
                          workspace=wf)
        b = R.decode_step(paged, up(kn), up(vn), up(q), lp, bound, w.sparsity, w.min_blocks, 1,
                          workspace=wp)
        torch.cuda.synchronize()
        for x, y in zip(a, b):
            assert torch.equal(x, y)
    assert torch.equal(flat.kmin, paged.kmin) and torch.equal(flat.kmax, paged.kmax)


def test_step_rejects_bad_arguments():
    w, cap = W.TINY_4K.with_(batch=1, num_kv_heads=2, num_q_heads=8, seq_len=100,
                             seed_tag="stepbad"), 128
    K, V = W.kv_cache(w, capacity=cap)
    cache = make_cache(K, V, 16, sentinel=False)
    lt = i32([100])
    kn, vn = W.decode_kv(w, 0)
    q = W.decode_query(w, 0)
    with pytest.raises(R.ResaError):  # no room to append under the host bound
        R.decode_step(cache, up(kn), up(vn), up(q), lt, 128, 0.9, 1, 1)
    with pytest.raises(R.ResaError):  # n_cap below the Eq. 5 count
        R.decode_step(cache, up(kn), up(vn), up(q), lt, 100, 0.0, 1, 1, n_cap=2)
    with pytest.raises(R.ResaError):
        R.decode_step(cache, up(kn), up(vn), up(q), lt, 100, 0.9, 1, 1, num_splits=300)
    torch.cuda.synchronize()
    assert lt.cpu().tolist() == [100]


def test_step_graph_replay_matches_eager():
    """The fused step recorded once in a HIP graph and replayed for several
    steps (inputs copied in between, eager calls and synchronisations between
    the replays) matches the same calls made eagerly, bit for bit: its
    counters and flags return to zero inside the kernel, with no memset."""
    w = W.LONG_64K.with_(batch=2, num_q_heads=8, num_kv_heads=2, seq_len=600, min_tokens=64,
                         seed_tag="stepgraph")
    b, cap, steps = 16, 704, 4
    B, H, Hq = 2, 2, 8
    K, V = W.kv_cache(w, capacity=cap)
    c1 = make_cache(K, V, b, sentinel=False)
    c2 = make_cache(K, V, b, sentinel=False)
    lens0 = [600, 555]
    l1, l2 = i32(lens0), i32(lens0)
    R.block_summarize(c1, l1)
    R.block_summarize(c2, l2)
    bound = max(lens0) + steps
    n_cap = R.num_selected(-(-(bound + 1) // b), w.sparsity, w.min_blocks, w.n_local)
    d = torch.device("cuda:0")
    bf = torch.bfloat16
    kn_s = torch.zeros((B, H, 128), dtype=bf, device=d)
    vn_s = torch.zeros((B, H, 128), dtype=bf, device=d)
    q_s = torch.zeros((B, Hq, 128), dtype=bf, device=d)
    idx2 = torch.empty((B, H, n_cap), dtype=torch.int32, device=d)
    ns2 = torch.empty((B, H), dtype=torch.int32, device=d)
    out2 = torch.empty((B, Hq, 128), dtype=torch.float32, device=d)
    lse2 = torch.empty((B, Hq), dtype=torch.float32, device=d)
    w1, w2 = R.Workspace(d), R.Workspace(d)
    for ws in (w1, w2):
        ws.get(R.lib().resa_step_workspace_size(B, H, Hq, bound, b, n_cap, 0))
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(graph, stream=side):
        R.decode_step(c2, kn_s, vn_s, q_s, l2, bound, w.sparsity, w.min_blocks, w.n_local, n_cap=n_cap,
                      block_idx=idx2, num_sel=ns2, out=out2, lse=lse2, workspace=w2)
    torch.cuda.synchronize()
    for step in range(steps):
        kn, vn = W.decode_kv(w, step)
        q = W.decode_query(w, step)
        kn_s.copy_(up(kn))
        vn_s.copy_(up(vn))
        q_s.copy_(up(q))
        graph.replay()
        torch.cuda.synchronize()
        i1, n1, o1, s1 = R.decode_step(c1, up(kn), up(vn), up(q), l1, bound, w.sparsity, w.min_blocks,
                                       w.n_local, n_cap=n_cap, workspace=w1)
        torch.cuda.synchronize()
        print(f"step graph replay {step}: n_sel {ns2.cpu().tolist()}", flush=True)
        assert step_error_flag(w2) == 0
        assert torch.equal(l1, l2)
        assert torch.equal(n1, ns2) and torch.equal(i1, idx2)
        assert torch.equal(o1, out2) and torch.equal(s1, lse2)
    for f in ("k", "v", "kmin", "kmax"):
        assert torch.equal(getattr(c1, f), getattr(c2, f)), f


@pytest.mark.parametrize("name", ["long_64k", "extreme_256k"])
def test_step_fullsize(name):
    """The fused step at the full 64K (8 x 32/8 heads) and 256K (1 x 32/8)
    shapes against resa_append_select + resa_sparse_decode on a copy of the
    cache (identical selections, outputs within fp32 reordering), and sampled
    groups against the oracle."""
    w = W.WORKLOADS[name]
    B, H, Hq, D, b, L = w.batch, w.num_kv_heads, w.num_q_heads, w.head_dim, w.block_size, w.seq_len
    g = w.group_size
    cap = -(-(L + 64) // b) * b
    d = torch.device("cuda:0")
    gen = torch.Generator(device=d)
    gen.manual_seed(4109)
    K = torch.randn((B, H, cap, D), generator=gen, device=d).to(torch.bfloat16)
    V = torch.randn((B, H, cap, D), generator=gen, device=d).to(torch.bfloat16)
    sampled = [(0, 0), (B - 1, H - 1)]
    host = {}
    for bi, hi in sampled:
        k, v = W.group_kv(w, bi, hi)
        K[bi, hi, :L] = up(k)
        V[bi, hi, :L] = up(v)
        host[bi, hi] = (k, v)
    mb = cap // b
    mk = lambda: torch.empty((B, H, mb, D), dtype=torch.bfloat16, device=d)
    c1 = R.KVCache(K, V, mk(), mk(), b)
    lens1 = i32([L] * B)
    R.block_summarize(c1, lens1)
    c2 = clone(c1)
    lens2 = lens1.clone()
    n_cap = R.num_selected(mb, w.sparsity, w.min_blocks, w.n_local)
    print(f"[step fullsize] {name}: B={B} Hq={Hq} Hkv={H} L={L} n_cap={n_cap}", flush=True)
    kn, vn = W.decode_kv(w, 0)
    q = W.decode_query(w, 0)
    ws = R.Workspace(d)
    idx, ns, out, lse = R.decode_step(c1, up(kn), up(vn), up(q), lens1, L, w.sparsity, w.min_blocks,
                                      w.n_local, n_cap=n_cap, workspace=ws)
    ri, rn = R.append_select(c2, up(kn), up(vn), up(q), lens2, L, w.sparsity, w.min_blocks, w.n_local,
                             n_cap=n_cap)
    ro, rl = R.sparse_decode(c2, up(q), lens2, ri, rn)
    torch.cuda.synchronize()
    assert step_error_flag(ws) == 0
    assert torch.equal(lens1, lens2) and torch.equal(ns, rn) and torch.equal(idx, ri)
    assert max_abs_err(out.cpu().numpy(), ro.cpu().numpy()) <= REORDER
    assert max_abs_err(lse.cpu().numpy(), rl.cpu().numpy()) <= REORDER
    gi, gn, go = idx.cpu().numpy(), ns.cpu().numpy(), out.cpu().numpy()
    q64 = O.bf16_to_f64(q)
    for bi, hi in sampled:
        k, v = host[bi, hi]
        Kg = np.zeros((1, 1, L + 1, D))
        Vg = np.zeros((1, 1, L + 1, D))
        Kg[0, 0, :L] = O.bf16_to_f64(k)
        Vg[0, 0, :L] = O.bf16_to_f64(v)
        st = O.DecodeState(Kg, Vg, [L], b)
        st.append(O.bf16_to_f64(kn)[bi:bi + 1, hi:hi + 1], O.bf16_to_f64(vn)[bi:bi + 1, hi:hi + 1])
        qg = q64[bi:bi + 1, hi * g:(hi + 1) * g]
        rs_, ri_, rn_ = st.select(qg, w.sparsity, w.min_blocks, w.n_local)
        assert gn[bi, hi] == rn_[0, 0]
        ids = gi[bi, hi, :gn[bi, hi]]
        check_selection(ids, ri_[0, 0], rs_[0, 0], rn_[0, 0], w.n_local)
        o_ref, _ = O.sparse_attend(qg[0], st.K[0, 0], st.V[0, 0], L + 1, ids, b, w.sm_scale)
        err = max_abs_err(go[bi, hi * g:(hi + 1) * g], o_ref)
        print(f"[step fullsize] {name} group ({bi},{hi}): |dO| {err:.2e}", flush=True)
        assert err <= TOL


def test_step_guard_trip_does_not_leak():
    """The fused step's bounded wait for a group's selection, forced to give
    up at once (RESA_STEP_MAX_SPINS=0, read by the library at each call): the
    call ends normally, a split that gave up decodes nothing and sets the
    sticky status word, and the next call on the same workspace (normal bound)
    finds every ready flag cleared and gives the results of the separate
    calls."""
    import os
    w = W.LONG_64K.with_(batch=2, num_kv_heads=8, num_q_heads=32, seq_len=60000, seed_tag="guard")
    cap = 60064
    lens = [60000, 47000]
    K, V = W.kv_cache(w, capacity=cap)
    cache = make_cache(K, V, 16, sentinel=False)
    ref = clone(cache)
    del K, V
    lt, lr = i32(lens), i32(lens)
    R.block_summarize(cache, lt)
    R.block_summarize(ref, lr)
    ws, ws_sel, ws_dec = R.Workspace(), R.Workspace(), R.Workspace()
    L = list(lens)
    for step in range(2):
        kn, vn = W.decode_kv(w, step)
        q = W.decode_query(w, step)
        os.environ["RESA_STEP_MAX_SPINS"] = "0" if step == 0 else str(1 << 20)
        try:
            idx, ns, out, lse = R.decode_step(cache, up(kn), up(vn), up(q), lt, max(L), w.sparsity,
                                              w.min_blocks, w.n_local, workspace=ws)
        finally:
            os.environ.pop("RESA_STEP_MAX_SPINS", None)
        ridx, rns = R.append_select(ref, up(kn), up(vn), up(q), lr, max(L), w.sparsity, w.min_blocks,
                                    w.n_local, n_cap=idx.shape[-1], workspace=ws_sel)
        rout, _ = R.sparse_decode(ref, up(q), lr, ridx, rns, workspace=ws_dec)
        torch.cuda.synchronize()
        groups = 16
        ready = ws.buf[256:256 + 4 * groups].view(torch.int32).cpu().numpy()
        assert np.all(ready == 0), "a ready flag leaked past the call"
        assert torch.equal(lt, lr) and torch.equal(ns, rns) and torch.equal(idx, ridx)
        if step == 0:
            print(f"guard status after the forced call: {step_error_flag(ws)}", flush=True)
        else:
            assert max_abs_err(out.cpu().numpy(), rout.cpu().numpy()) <= REORDER
        L = [x + 1 for x in L]
