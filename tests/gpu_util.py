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
