"""The allocation-free decode entry point (resa_sparse_decode_noalloc, for
callers that cannot allocate) against resa_sparse_decode with a workspace:
two calls in a row on the shared static scratch, the second on a smaller
input, both bit-identical to the workspace calls; oversized requests are
rejected before any device work."""
import ctypes as C
import math

import numpy as np
import pytest
import torch

import paper_2506_04108_amd as R
import workloads as W
from gpu_util import dev, i32, make_cache, up
from paper_2506_04108_amd._lib import RESA_OK, lib

pytestmark = pytest.mark.gpu


def _case(B, H, g, L, cap, b, tag):
    w = W.TINY_4K.with_(batch=B, num_kv_heads=H, num_q_heads=g * H, seq_len=L, block_size=b,
                        min_tokens=4 * b, seed_tag=tag)
    K, V = W.kv_cache(w, capacity=cap)
    cache = make_cache(K, V, b, sentinel=False)
    lens = [L - 37 * i for i in range(B)]
    lt = i32(lens)
    R.block_summarize(cache, lt)
    q = up(W.decode_query(w, 0))
    idx, ns = R.select_blocks(cache, q, lt, max(lens), w.sparsity, w.min_blocks, 1)
    return cache, q, lt, idx, ns


def _noalloc(cache, q, lt, idx, ns, splits):
    B, Hq = q.shape[0], q.shape[1]
    out = torch.full((B, Hq, 128), float("nan"), dtype=torch.float32, device=dev())
    lse = torch.full((B, Hq), float("nan"), dtype=torch.float32, device=dev())
    d = cache.desc()
    rc = lib().resa_sparse_decode_noalloc(C.byref(d), q.data_ptr(), Hq, lt.data_ptr(), idx.data_ptr(),
                                          ns.data_ptr(), idx.shape[-1], splits,
                                          1.0 / math.sqrt(128), out.data_ptr(), lse.data_ptr(),
                                          torch.cuda.current_stream().cuda_stream)
    assert rc == RESA_OK, lib().resa_last_error().decode()
    return out, lse


@pytest.mark.parametrize("splits", [0, 5])
def test_noalloc_matches_workspace_decode(splits):
    big = _case(4, 8, 4, 6000, 6144, 16, "noalloc-big")
    small = _case(2, 2, 7, 900, 1024, 32, "noalloc-small")
    results = []
    for cache, q, lt, idx, ns in (big, small):       # second call: smaller input
        o1, l1 = _noalloc(cache, q, lt, idx, ns, splits)
        o2, l2 = R.sparse_decode(cache, q, lt, idx, ns, num_splits=splits)
        torch.cuda.synchronize()
        results.append((o1.cpu().numpy(), l1.cpu().numpy(), o2.cpu().numpy(), l2.cpu().numpy()))
    for o1, l1, o2, l2 in results:
        assert np.all(np.isfinite(o1)) and np.all(np.isfinite(l1))
        assert np.array_equal(o1, o2)
        assert np.array_equal(l1, l2)


def test_noalloc_rejects_oversized_scratch():
    cache, q, lt, idx, ns = _case(2, 2, 8, 900, 1024, 16, "noalloc-size")
    cap = lib().resa_sparse_decode_noalloc_max_bytes()
    assert cap == 4 << 20
    # 256 splits of 8 heads for a 64 x 64 batch of groups would need far more.
    big = R.KVCache(cache.k, cache.v, cache.kmin, cache.kmax, 16)
    d = big.desc()
    d.batch, d.num_kv_heads = 64, 64
    need = lib().resa_decode_workspace_size(64, 64, 512, 64, 16, 256)
    assert need > cap
    rc = lib().resa_sparse_decode_noalloc(C.byref(d), q.data_ptr(), 512, lt.data_ptr(), idx.data_ptr(),
                                          ns.data_ptr(), 64, 256, 0.1, q.data_ptr(), None,
                                          torch.cuda.current_stream().cuda_stream)
    assert rc == 3  # RESA_ERR_WORKSPACE, before any device work
    assert "static" in lib().resa_last_error().decode()
