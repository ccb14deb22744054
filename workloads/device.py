"""Bulk synthetic caches generated directly on the GPU (benchmark inputs).

Same recipe as ``workloads`` (N(0, 1) keys/values rounded to bf16, per
(kv head, channel) LogNormal key scale, planted heavy-hitter blocks, decode
rows and rectification rows) but drawn with torch's seeded device generator,
because drawing gigabytes on the host takes minutes. Parity tests use the host
generator instead; the benchmark only needs the distribution.
"""
from __future__ import annotations

import torch

from . import Workload


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def caches(w: Workload, capacity: int, layer: int, device="cuda"):
    """K, V bf16 ``[B, Hkv, capacity, 128]`` for one layer (rows >= L are zero),
    the key channel scale ``[Hkv, 128]`` (or None) and the planted directions
    ``[B, Hkv, 128]`` (or None), which the decode queries of the layer carry too."""
    B, H, D, L = w.batch, w.num_kv_heads, w.head_dim, w.seq_len
    g = _gen(4108 * 1000 + 17 * layer + w.tag() % 997, device)
    K = torch.zeros((B, H, capacity, D), dtype=torch.bfloat16, device=device)
    V = torch.zeros_like(K)
    scale = None
    plant = torch.zeros((B, H, D), device=device) if w.planted_per_head > 0 else None
    if w.key_scale_sigma > 0:
        scale = torch.empty((H, D), device=device).log_normal_(0.0, w.key_scale_sigma, generator=g)
    for bi in range(B):
        k = torch.randn((H, L, D), generator=g, device=device)
        if scale is not None:
            k *= scale[:, None, :]
        if w.planted_per_head > 0:
            M = w.num_blocks
            for hi in range(H):
                u = torch.randn(D, generator=g, device=device)
                u *= w.plant_norm / u.norm()
                plant[bi, hi] = u
                blocks = torch.randperm(max(M - 1, 1), generator=g, device=device)[:w.planted_per_head]
                rows = (blocks[:, None] * w.block_size + torch.arange(w.block_size, device=device)).reshape(-1)
                rows = rows[rows < L]
                k[hi, rows] += w.plant_gain * u
        K[bi, :, :L] = k.to(torch.bfloat16)
        V[bi, :, :L] = torch.randn((H, L, D), generator=g, device=device).to(torch.bfloat16)
    return K, V, scale, plant


def step_inputs(w: Workload, steps: int, layer: int, scale=None, plant=None, device="cuda"):
    """Per-step decode rows: q ``[steps, B, Hq, 128]``, k, v ``[steps, B, Hkv, 128]`` (bf16).
    Each query head of kv group i gets that group's planted direction added."""
    B, H, D = w.batch, w.num_kv_heads, w.head_dim
    g = _gen(4108 * 2000 + 17 * layer + w.tag() % 997, device)
    q = torch.randn((steps, B, w.num_q_heads, D), generator=g, device=device)
    k = torch.randn((steps, B, H, D), generator=g, device=device)
    v = torch.randn((steps, B, H, D), generator=g, device=device)
    if scale is not None:
        k *= scale[None, None]
    if plant is not None:
        q += plant.repeat_interleave(w.group_size, dim=1)[None]
    return q.to(torch.bfloat16), k.to(torch.bfloat16), v.to(torch.bfloat16)


def rectify_rows(w: Workload, k_last: torch.Tensor, v_last: torch.Tensor, f: int, seed: int,
                 device="cuda"):
    """Re-encoded rows: q_f ``[B, Hq, f, 128]`` ~ N(0, 1); k_f, v_f = the last f rows + 0.05 N(0, 1)."""
    g = _gen(4108 * 3000 + seed, device)
    B, D = w.batch, w.head_dim
    q = torch.randn((B, w.num_q_heads, f, D), generator=g, device=device).to(torch.bfloat16)
    k = (k_last.float() + 0.05 * torch.randn(k_last.shape, generator=g, device=device)).to(torch.bfloat16)
    v = (v_last.float() + 0.05 * torch.randn(v_last.shape, generator=g, device=device)).to(torch.bfloat16)
    return q.contiguous(), k.contiguous(), v.contiguous()


def to_pages(X: torch.Tensor, table: torch.Tensor, block_size: int) -> torch.Tensor:
    """Contiguous ``[B, Hkv, cap, 128]`` -> page pool ``[B * cap / b, Hkv, b, 128]``
    with logical block m of sequence s on page ``table[s, m]``."""
    B, H, cap, D = X.shape
    mb = cap // block_size
    pool = torch.empty((B * mb, H, block_size, D), dtype=X.dtype, device=X.device)
    pool[table.reshape(-1).long()] = X.view(B, H, mb, block_size, D).permute(0, 2, 1, 3, 4).reshape(
        B * mb, H, block_size, D)
    return pool
