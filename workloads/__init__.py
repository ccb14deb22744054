"""Seeded synthetic inputs for ReSA decode workloads.

This module feeds both the CPU oracle and the HIP path. It holds no attention
arithmetic: only random draws, float32 -> bf16 rounding (round to nearest
even), the heavy-hitter planting and the per-channel key scaling that define
the synthetic workloads.

Every tensor of every (batch, kv-head) group is drawn from its own seed
(``SeedSequence([4108, workload, tensor, batch, kv_head, ...])``), so a single
group can be regenerated on its own at full size, which is how full-size parity
checks sample groups without rebuilding a whole cache on the host.

All tensors are returned as ``numpy.uint16`` arrays holding bf16 bit patterns.
Layouts follow the library's: K/V caches ``[B, Hkv, capacity, D]``, decode
queries ``[B, Hq, D]`` with query head ``h = i * g + j`` belonging to kv head
``i`` (grouped-query attention, Eq. 1), rectify queries ``[B, Hq, f, D]``.
"""
from __future__ import annotations

import dataclasses
import math
import zlib

import numpy as np

SEED = 4108

# Tensor tags: each kind of tensor gets its own stream of random numbers.
_TAGS = {
    "k": 1, "v": 2, "q": 3, "plant_u": 4, "plant_blocks": 5, "chan_scale": 6,
    "step_q": 7, "step_k": 8, "step_v": 9, "rect_q": 10, "rect_dk": 11,
    "rect_dv": 12, "garbage": 13,
}

_CHUNK = 1 << 22  # elements converted per chunk (bounds temporaries)


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic decode workload (shape plus input recipe)."""

    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    seq_len: int            # cache length L after prefill
    block_size: int         # b
    sparsity: float         # fraction of blocks skipped; keep = 1 - sparsity
    min_tokens: int         # minimum budget in tokens (n_min = ceil(min_tokens / b))
    n_local: int = 1        # most recent blocks always kept
    rectify_every: int = 32  # f
    planted_per_head: int = 0   # heavy-hitter blocks per (batch, kv head)
    plant_norm: float = 1.0     # |u| of the planted direction
    plant_gain: float = 2.0     # K += gain * u inside planted blocks
    key_scale_sigma: float = 0.0  # >0: keys scaled per (kv head, channel) by LogNormal(0, sigma)
    decode_steps: int = 0       # length of the decode loop (0: single step)
    seed_tag: str = ""          # defaults to ``name``

    @property
    def group_size(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def num_blocks(self) -> int:
        return -(-self.seq_len // self.block_size)

    @property
    def min_blocks(self) -> int:
        return -(-self.min_tokens // self.block_size)

    @property
    def sm_scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    def tag(self) -> int:
        return zlib.crc32((self.seed_tag or self.name).encode())


# The five workloads: a tiny 4K layer, a Qwen-7B-like 32K layer (28 query / 4 kv
# heads, head_dim 128), a 64K batch-8 decode loop with outlier key channels, a
# 256K single-sequence decode, and the 64K sweep base.
TINY_4K = Workload("tiny_4k", 1, 32, 8, 128, 4096, 16, 0.9, 64 * 16, 1, 16,
                   planted_per_head=8)
QWEN7B_32K = Workload("qwen7b_32k", 4, 28, 4, 128, 32768, 16, 0.9, 2048, 1, 32,
                      planted_per_head=20)
LONG_64K = Workload("long_64k", 8, 32, 8, 128, 65536, 16, 0.9, 2048, 1, 32,
                    key_scale_sigma=0.5, decode_steps=128)
EXTREME_256K = Workload("extreme_256k", 1, 32, 8, 128, 262144, 16, 0.95, 4096, 1, 32,
                        planted_per_head=164)
SWEEP_64K = Workload("sweep_64k", 8, 32, 8, 128, 65536, 16, 0.9, 2048, 1, 32,
                     planted_per_head=41)

WORKLOADS = {w.name: w for w in (TINY_4K, QWEN7B_32K, LONG_64K, EXTREME_256K, SWEEP_64K)}


def sweep_points():
    """The 64K sweep grid: block size x sparsity x rectify interval."""
    pts = []
    for b in (16, 32, 64):
        for s in (0.8, 0.9, 0.95):
            for f in (16, 32, 64):
                m = SWEEP_64K.seq_len // b
                pts.append(SWEEP_64K.with_(block_size=b, sparsity=s, rectify_every=f,
                                           planted_per_head=round(0.01 * m)))
    return pts


# --------------------------------------------------------------------------- rng

def rng(w: Workload, tensor: str, *idx: int) -> np.random.Generator:
    ss = np.random.SeedSequence([SEED, w.tag(), _TAGS[tensor], *[int(i) for i in idx]])
    return np.random.Generator(np.random.PCG64(ss))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); returns uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    flat = x.reshape(-1)
    out = np.empty(flat.shape, dtype=np.uint16)
    tmp = np.empty(min(flat.size, _CHUNK), dtype=np.uint32)
    lsb = np.empty_like(tmp)
    for s in range(0, flat.size, _CHUNK):
        u = flat[s:s + _CHUNK].view(np.uint32)
        n = u.size
        np.right_shift(u, 16, out=lsb[:n])
        np.bitwise_and(lsb[:n], 1, out=lsb[:n])
        np.add(u, 0x7FFF, out=tmp[:n])
        np.add(tmp[:n], lsb[:n], out=tmp[:n])
        np.right_shift(tmp[:n], 16, out=tmp[:n])
        out[s:s + n] = tmp[:n]
    return out.reshape(x.shape)


def bf16_bits_to_f32(u: np.ndarray) -> np.ndarray:
    """Widen bf16 bits to float32 (exact)."""
    return (np.asarray(u, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _normal(g: np.random.Generator, shape) -> np.ndarray:
    return g.standard_normal(shape, dtype=np.float32)


# ------------------------------------------------------------------ per-group data

def plant_vector(w: Workload, bi: int, hi: int) -> np.ndarray | None:
    """Planted direction u for group (bi, hi): a seeded vector of norm ``plant_norm``."""
    if w.planted_per_head <= 0:
        return None
    u = rng(w, "plant_u", bi, hi).standard_normal(w.head_dim).astype(np.float64)
    u *= w.plant_norm / np.linalg.norm(u)
    return u.astype(np.float32)


def planted_blocks(w: Workload, bi: int, hi: int) -> np.ndarray:
    """Block ids (drawn from 0..M-2, so never the forced last block) that carry u."""
    if w.planted_per_head <= 0:
        return np.zeros(0, dtype=np.int64)
    m = w.num_blocks
    p = min(w.planted_per_head, max(m - 1, 0))
    return np.sort(rng(w, "plant_blocks", bi, hi).choice(max(m - 1, 1), size=p, replace=False))


def channel_scale(w: Workload) -> np.ndarray | None:
    """Per (kv head, channel) key scale ~ LogNormal(0, sigma), shared over the batch."""
    if w.key_scale_sigma <= 0:
        return None
    g = rng(w, "chan_scale")
    return g.lognormal(0.0, w.key_scale_sigma, size=(w.num_kv_heads, w.head_dim)).astype(np.float32)


def group_kv(w: Workload, bi: int, hi: int, rows: int | None = None):
    """Prefill keys and values of group (bi, hi): two uint16 arrays ``[L, D]``."""
    L = w.seq_len if rows is None else rows
    D = w.head_dim
    k = _normal(rng(w, "k", bi, hi), (L, D))
    v = _normal(rng(w, "v", bi, hi), (L, D))
    sc = channel_scale(w)
    if sc is not None:
        k *= sc[hi][None, :]
    u = plant_vector(w, bi, hi)
    if u is not None:
        b = w.block_size
        for m in planted_blocks(w, bi, hi):
            lo, hi_ = m * b, min((m + 1) * b, L)
            if lo < hi_:
                k[lo:hi_] += w.plant_gain * u[None, :]
    return f32_to_bf16_bits(k), f32_to_bf16_bits(v)


def kv_cache(w: Workload, capacity: int | None = None, garbage: float | None = None):
    """Whole caches ``[B, Hkv, capacity, D]`` (uint16). Rows >= L are zero, or a
    seeded garbage pattern of magnitude ``garbage`` when given."""
    cap = w.seq_len if capacity is None else capacity
    assert cap >= w.seq_len
    shape = (w.batch, w.num_kv_heads, cap, w.head_dim)
    K = np.zeros(shape, dtype=np.uint16)
    V = np.zeros(shape, dtype=np.uint16)
    for bi in range(w.batch):
        for hi in range(w.num_kv_heads):
            k, v = group_kv(w, bi, hi)
            K[bi, hi, :w.seq_len] = k
            V[bi, hi, :w.seq_len] = v
            if garbage is not None and cap > w.seq_len:
                gz = _normal(rng(w, "garbage", bi, hi), (2, cap - w.seq_len, w.head_dim))
                gz *= garbage
                K[bi, hi, w.seq_len:] = f32_to_bf16_bits(gz[0])
                V[bi, hi, w.seq_len:] = f32_to_bf16_bits(gz[1])
    return K, V


def _plant_queries(w: Workload, q: np.ndarray) -> np.ndarray:
    """Add each group's planted direction to its g query heads (float32 in place)."""
    g = w.group_size
    for bi in range(w.batch):
        for hi in range(w.num_kv_heads):
            u = plant_vector(w, bi, hi)
            if u is not None:
                q[bi, hi * g:(hi + 1) * g] += u
    return q


def decode_query(w: Workload, step: int = 0) -> np.ndarray:
    """Decode queries ``[B, Hq, D]`` for decode step ``step``."""
    q = _normal(rng(w, "step_q", step), (w.batch, w.num_q_heads, w.head_dim))
    return f32_to_bf16_bits(_plant_queries(w, q))


def decode_kv(w: Workload, step: int):
    """New key/value rows ``[B, Hkv, D]`` appended at decode step ``step``."""
    k = _normal(rng(w, "step_k", step), (w.batch, w.num_kv_heads, w.head_dim))
    v = _normal(rng(w, "step_v", step), (w.batch, w.num_kv_heads, w.head_dim))
    sc = channel_scale(w)
    if sc is not None:
        k *= sc[None, :, :]
    return f32_to_bf16_bits(k), f32_to_bf16_bits(v)


def rectify_inputs(w: Workload, step: int, last_k: np.ndarray, last_v: np.ndarray, f: int):
    """Refreshed rows for a rectification after ``step``.

    ``last_k``/``last_v`` are the f most recent cache rows ``[B, Hkv, f, D]`` (uint16);
    the refreshed rows are those plus 0.05 * N(0, 1). Queries are fresh N(0, 1)
    draws (plus the planted direction). Returns ``(q_f [B,Hq,f,D], k_f, v_f [B,Hkv,f,D])``.
    """
    B, Hkv, D = w.batch, w.num_kv_heads, w.head_dim
    assert last_k.shape == (B, Hkv, f, D)
    q = _normal(rng(w, "rect_q", step), (B, w.num_q_heads, f, D))
    g = w.group_size
    for bi in range(B):
        for hi in range(Hkv):
            u = plant_vector(w, bi, hi)
            if u is not None:
                q[bi, hi * g:(hi + 1) * g] += u
    dk = _normal(rng(w, "rect_dk", step), (B, Hkv, f, D))
    dv = _normal(rng(w, "rect_dv", step), (B, Hkv, f, D))
    k = bf16_bits_to_f32(last_k) + 0.05 * dk
    v = bf16_bits_to_f32(last_v) + 0.05 * dv
    return f32_to_bf16_bits(q), f32_to_bf16_bits(k), f32_to_bf16_bits(v)


def small(w: Workload, **kw) -> Workload:
    """A reduced copy of a workload (for quick tests), keeping its recipe."""
    return w.with_(**kw)
