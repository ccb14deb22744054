"""Helpers for the GPU parity tests: upload generator output, build caches,
and run the oracle on the same inputs."""
from __future__ import annotations

import numpy as np
import torch

import oracle as O
import paper_2506_04108_amd as R

SENTINEL = 0x7F7F  # bf16 ~3.4e38: marks summary rows a kernel must not touch


def dev():
    assert torch.cuda.is_available(), "GPU test without a GPU"
    return torch.device("cuda:0")


def up(a: np.ndarray) -> torch.Tensor:
    """uint16 bf16 bits -> device bf16 tensor."""
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev())


def down(t: torch.Tensor) -> np.ndarray:
    """device bf16 tensor -> uint16 bits."""
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def i32(values) -> torch.Tensor:
    return torch.tensor(values, dtype=torch.int32, device=dev())


def make_cache(K: np.ndarray, V: np.ndarray, block_size: int, sentinel=True) -> R.KVCache:
    B, H, cap, D = K.shape
    mb = cap // block_size
    fill = np.full((B, H, mb, D), SENTINEL if sentinel else 0, dtype=np.uint16)
    return R.KVCache(up(K), up(V), up(fill), up(fill.copy()), block_size)


def oracle_summaries(K64: np.ndarray, lens, b):
    out = {}
    for bi in range(K64.shape[0]):
        for hi in range(K64.shape[1]):
            out[bi, hi] = O.block_summaries(K64[bi, hi], lens[bi], b)
    return out


def padded_idx(idx_lists, B, H, n_cap):
    a = np.full((B, H, n_cap), -1, dtype=np.int32)
    n = np.zeros((B, H), dtype=np.int32)
    for (bi, hi), ids in idx_lists.items():
        a[bi, hi, :len(ids)] = ids
        n[bi, hi] = len(ids)
    return a, n


def make_paged_cache(K: np.ndarray, V: np.ndarray, block_size: int, lens_final, seed=0,
                     spare=5, sentinel=True) -> R.KVCache:
    """The same contents as make_cache in the paged layout: every logical
    block that holds a token of sequence b (up to lens_final[b]) gets its own
    page of a shuffled pool with `spare` extra pages; the other table entries
    stay -1 (unassigned), so a kernel that touched them would be caught."""
    B, H, cap, D = K.shape
    mb = cap // block_size
    used = [min(-(-int(L) // block_size), mb) for L in lens_final]
    P = sum(used) + spare
    rng = np.random.default_rng(seed)
    perm = rng.permutation(P).astype(np.int32)
    table = np.full((B, mb), -1, dtype=np.int32)
    Kp = rng.integers(0, 2 ** 16, size=(P, H, block_size, D), dtype=np.uint16) & 0xBFFF  # finite junk
    Vp = rng.integers(0, 2 ** 16, size=(P, H, block_size, D), dtype=np.uint16) & 0xBFFF
    i = 0
    for bi in range(B):
        for m in range(used[bi]):
            p = perm[i]
            i += 1
            table[bi, m] = p
            Kp[p] = K[bi, :, m * block_size:(m + 1) * block_size]
            Vp[p] = V[bi, :, m * block_size:(m + 1) * block_size]
    fill = np.full((B, H, mb, D), SENTINEL if sentinel else 0, dtype=np.uint16)
    return R.KVCache(up(Kp), up(Vp), up(fill), up(fill.copy()), block_size,
                     torch.from_numpy(table).to(dev()))


def unpage(cache: R.KVCache, lens):
    """Rows [0, L_b) of a paged cache, gathered back to ``[B, Hkv, cap, D]``
    uint16 (rows past L_b are zero)."""
    table = cache.block_table.cpu().numpy()
    Kp, Vp = down(cache.k), down(cache.v)
    B, mb = table.shape
    b = cache.block_size
    H = Kp.shape[1]
    K = np.zeros((B, H, mb * b, Kp.shape[3]), dtype=np.uint16)
    V = np.zeros_like(K)
    for bi in range(B):
        for m in range(-(-int(lens[bi]) // b)):
            K[bi, :, m * b:(m + 1) * b] = Kp[table[bi, m]]
            V[bi, :, m * b:(m + 1) * b] = Vp[table[bi, m]]
        K[bi, :, lens[bi]:] = 0
        V[bi, :, lens[bi]:] = 0
    return K, V


def select_stats(ws, batch, kv_heads, step=False) -> np.ndarray:
    """The per-group diagnostic counters of a selection (or fused step)
    workspace: calls whose top-n finished on its in-window path."""
    from paper_2506_04108_amd._lib import lib
    off = (lib().resa_step_stats_offset if step else lib().resa_select_stats_offset)(batch, kv_heads)
    n = batch * kv_heads
    return ws.buf[off:off + 4 * n].view(torch.int32).cpu().numpy().reshape(batch, kv_heads)
