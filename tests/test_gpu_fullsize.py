"""GPU parity at the full workload sizes, in the launch configuration that
bench.py times (same n_cap, split count, workspaces and host length bounds).

The kernels run over every (sequence, kv head) group of the full-size caches;
the oracle checks sampled groups one at a time. Sampled groups hold the host
generator's values (so the oracle sees exactly what the GPU sees); the other
groups hold device-drawn data of the same kind, which no sampled group's
selection, decode or rectification reads. Cache rows past each length hold
random data too, so a kernel that read past L would be caught.

One decode step is checked per workload: append the step's token, select with
the workload's sparsity and budget, decode; then one rectification of the
last f rows (including the appended token).
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2506_04108_amd as R
import workloads as W
from gpu_util import dev, down, i32, up
from oracle.compare import check_selection, max_abs_err

pytestmark = pytest.mark.gpu
TOL = 2e-3


def _bench_shapes(w, steps=128, warmup=32, layers=4):
    """Capacity, n_cap and split count as bench.py derives them."""
    per_layer = -(-(steps + warmup) // layers)
    b = w.block_size
    cap = -(-(w.seq_len + per_layer + b) // b) * b
    n_cap = R.num_selected(cap // b, w.sparsity, w.min_blocks, w.n_local)
    splits = R.decode_num_splits(w.batch, w.num_kv_heads, n_cap, b)
    return cap, n_cap, splits


def _full_size_step(w, select_groups, rectify_groups):
    B, H, Hq, D, b, L = w.batch, w.num_kv_heads, w.num_q_heads, w.head_dim, w.block_size, w.seq_len
    g, f = w.group_size, w.rectify_every
    cap, n_cap, splits = _bench_shapes(w)
    d = dev()
    print(f"[fullsize] {w.name}: B={B} Hq={Hq} Hkv={H} L={L} cap={cap} n_cap={n_cap} "
          f"splits={splits}", flush=True)

    gen = torch.Generator(device=d)
    gen.manual_seed(4108)
    K = torch.randn((B, H, cap, D), generator=gen, device=d).to(torch.bfloat16)
    V = torch.randn((B, H, cap, D), generator=gen, device=d).to(torch.bfloat16)
    host = {}
    for bi, hi in sorted(set(select_groups) | set(rectify_groups)):
        k, v = W.group_kv(w, bi, hi)
        K[bi, hi, :L] = up(k)
        V[bi, hi, :L] = up(v)
        host[bi, hi] = (k, v)
    mb = cap // b
    cache = R.KVCache(K, V, torch.empty((B, H, mb, D), dtype=torch.bfloat16, device=d),
                      torch.empty((B, H, mb, D), dtype=torch.bfloat16, device=d), b)
    lens = i32([L] * B)
    R.block_summarize(cache, lens)

    # One decode step: append, select, decode (bench's arguments).
    kn, vn = W.decode_kv(w, 0)
    q = W.decode_query(w, 0)
    R.append_kv(cache, up(kn), up(vn), lens, L)
    ws_sel = R.Workspace(d)
    idx, ns = R.select_blocks(cache, up(q), lens, L + 1, w.sparsity, w.min_blocks, w.n_local,
                              n_cap=n_cap, workspace=ws_sel)
    # A second call on the same workspace starts from the digit window the
    # first call left behind: the same selection.
    idx_h, ns_h = R.select_blocks(cache, up(q), lens, L + 1, w.sparsity, w.min_blocks, w.n_local,
                                  n_cap=n_cap, workspace=ws_sel)
    out, lse = R.sparse_decode(cache, up(q), lens, idx, ns, num_splits=splits)
    torch.cuda.synchronize()
    assert torch.equal(idx, idx_h) and torch.equal(ns, ns_h)
    gi, gn = idx.cpu().numpy(), ns.cpu().numpy()
    go, gl = out.cpu().numpy(), lse.cpu().numpy()
    sm = w.sm_scale
    q64 = O.bf16_to_f64(q)
    n_ref = O.num_selected(O.num_blocks(L + 1, b), w.sparsity, w.min_blocks, w.n_local)
    swaps = 0
    states = {}
    for bi, hi in select_groups:
        k, v = host[bi, hi]
        Kg = np.zeros((1, 1, L + 1, D))
        Vg = np.zeros((1, 1, L + 1, D))
        Kg[0, 0, :L] = O.bf16_to_f64(k)
        Vg[0, 0, :L] = O.bf16_to_f64(v)
        st = O.DecodeState(Kg, Vg, [L], b)
        st.append(O.bf16_to_f64(kn)[bi:bi + 1, hi:hi + 1], O.bf16_to_f64(vn)[bi:bi + 1, hi:hi + 1])
        qg = q64[bi:bi + 1, hi * g:(hi + 1) * g]
        rs, ri, rn = st.select(qg, w.sparsity, w.min_blocks, w.n_local)
        assert gn[bi, hi] == rn[0, 0] == n_ref
        dev_ids = gi[bi, hi, :gn[bi, hi]]
        swaps += check_selection(dev_ids, ri[0, 0], rs[0, 0], rn[0, 0], w.n_local)
        assert np.all(gi[bi, hi, gn[bi, hi]:] == -1)
        ro, rl = O.sparse_attend(qg[0], st.K[0, 0], st.V[0, 0], L + 1, dev_ids, b, sm)
        eo = max_abs_err(go[bi, hi * g:(hi + 1) * g], ro)
        el = max_abs_err(gl[bi, hi * g:(hi + 1) * g], rl)
        print(f"[fullsize] {w.name} group ({bi},{hi}): n={rn[0, 0]} decode |dO| {eo:.2e} "
              f"|dlse| {el:.2e}", flush=True)
        assert eo <= TOL and el <= TOL
        states[bi, hi] = st
    print(f"[fullsize] {w.name}: {swaps} near-tie swaps over {len(select_groups)} groups",
          flush=True)

    # Rectification of the last f rows (the appended token included).
    Lr = L + 1
    last_k = down(cache.k[:, :, Lr - f:Lr])
    last_v = down(cache.v[:, :, Lr - f:Lr])
    qf, kf, vf = W.rectify_inputs(w, 1, last_k, last_v, f)
    rout, rlse = R.dense_rectify(cache, up(qf), up(kf), up(vf), lens, Lr)
    torch.cuda.synchronize()
    ro_all, rl_all = rout.cpu().numpy(), rlse.cpu().numpy()
    qf64 = O.bf16_to_f64(qf)
    for bi, hi in rectify_groups:
        st = states[bi, hi]
        qg = O.split_heads(qf64[bi:bi + 1], H)[0, hi]
        ro, rl = O.rectify_group(qg, st.K[0, 0], st.V[0, 0], st.kmin[0, 0], st.kmax[0, 0], Lr, f,
                                 b, sm, O.bf16_to_f64(kf[bi, hi]), O.bf16_to_f64(vf[bi, hi]))
        eo = max_abs_err(ro_all[bi, hi * g:(hi + 1) * g], ro)
        el = max_abs_err(rl_all[bi, hi * g:(hi + 1) * g], rl)
        print(f"[fullsize] {w.name} group ({bi},{hi}): rectify |dO| {eo:.2e} |dlse| {el:.2e}",
              flush=True)
        assert eo <= TOL and el <= TOL
        gk = down(cache.k[bi, hi, Lr - f:Lr])
        assert np.array_equal(gk, kf[bi, hi])
        M = O.num_blocks(Lr, b)
        lo = (Lr - f) // b
        assert np.array_equal(O.bf16_to_f64(down(cache.kmin[bi, hi, lo:M])), st.kmin[0, 0, lo:M])
        assert np.array_equal(O.bf16_to_f64(down(cache.kmax[bi, hi, lo:M])), st.kmax[0, 0, lo:M])


def test_fullsize_qwen7b_32k():
    """4 x 28/4 heads (g = 7), 32K context: every group's selection and decode,
    two groups' rectification."""
    w = W.QWEN7B_32K
    groups = [(bi, hi) for bi in range(w.batch) for hi in range(w.num_kv_heads)]
    _full_size_step(w, groups, [(0, 0), (3, 2)])


def test_fullsize_long_64k():
    """8 x 32/8 heads, 64K context, outlier key channels: the benchmark's
    launch shape (256 decode workgroups, 4 selection workgroups per group)."""
    w = W.LONG_64K
    _full_size_step(w, [(0, 0), (3, 5), (7, 7)], [(3, 5)])


def test_fullsize_extreme_256k():
    """1 x 32/8 heads, 256K context, sparsity 0.95 with a 4096-token minimum."""
    w = W.EXTREME_256K
    _full_size_step(w, [(0, 1), (0, 6)], [(0, 6)])


def test_fullsize_prefill_32k():
    """Whole-prompt prefill of a 32K prompt (1 x 32/8 heads, f = L = 32768)
    through the rectification call, in the launch shape bench.py's prefill
    case times (one key split, output written directly): sampled rows of two
    groups against the oracle, the written rows and every block summary."""
    w = W.LONG_64K.with_(batch=1, seq_len=32768, seed_tag="prefill32k")
    L = f = w.seq_len
    H, g, b, sm = w.num_kv_heads, w.group_size, w.block_size, w.sm_scale
    assert R.lib().resa_rectify_workspace_size(1, H, w.num_q_heads, f, L) == 0
    K, V = W.kv_cache(w)
    qf, kf, vf = W.rectify_inputs(w, 0, K, V, f)
    del K, V
    mb = L // b
    cache = R.KVCache(torch.zeros((1, H, L, 128), dtype=torch.bfloat16, device=dev()),
                      torch.zeros((1, H, L, 128), dtype=torch.bfloat16, device=dev()),
                      torch.zeros((1, H, mb, 128), dtype=torch.bfloat16, device=dev()),
                      torch.zeros((1, H, mb, 128), dtype=torch.bfloat16, device=dev()), b)
    lens = i32([L])
    print(f"[fullsize] prefill 32K: B=1 Hq={w.num_q_heads} Hkv={H} f=L={L}", flush=True)
    out, lse = R.dense_rectify(cache, up(qf), up(kf), up(vf), lens, L)
    torch.cuda.synchronize()
    rows = [0, 1, 63, 64, 127, 128, 4095, 16383, 20000, 32767]
    for hi in (0, 5):
        k64, v64 = O.bf16_to_f64(kf[0, hi]), O.bf16_to_f64(vf[0, hi])
        qg = O.bf16_to_f64(qf[0, hi * g:(hi + 1) * g])
        go = out[0, hi * g:(hi + 1) * g].cpu().numpy()
        gl = lse[0, hi * g:(hi + 1) * g].cpu().numpy()
        worst = 0.0
        for r in rows:
            ro, rl = O.attend(qg[:, r], k64, v64, range(r + 1), sm)
            eo, el = max_abs_err(go[:, r], ro), max_abs_err(gl[:, r], rl)
            worst = max(worst, eo, el)
            assert eo <= TOL and el <= TOL, (hi, r, eo, el)
        print(f"[fullsize] prefill 32K head {hi}: worst sampled error {worst:.2e}", flush=True)
        assert np.array_equal(down(cache.k[0, hi]), kf[0, hi])
        assert np.array_equal(down(cache.v[0, hi]), vf[0, hi])
        mn, mx = O.block_summaries(k64, L, b)
        assert np.array_equal(O.bf16_to_f64(down(cache.kmin[0, hi])), mn)
        assert np.array_equal(O.bf16_to_f64(down(cache.kmax[0, hi])), mx)
