"""ReSA (Rectified Sparse Attention) decode path for AMD MI355X.

A thin binding over libresa.so: it marshals torch tensors into the C ABI of
include/resa.h (device pointers, sizes, the current HIP stream) and allocates
outputs and workspaces with torch when the caller does not pass them. Every
step of the path runs in the library's HIP kernels.

    cache = KVCache.empty(batch, kv_heads, capacity, block_size, device="cuda")
    block_summarize(cache, seq_lens)
    idx, nsel = select_blocks(cache, q, seq_lens, max_seq_len, sparsity=0.9,
                              min_blocks=128, n_local=1)
    out, lse = sparse_decode(cache, q, seq_lens, idx, nsel)
    dense_rectify(cache, q_f, k_f, v_f, seq_lens, max_seq_len)
"""
from __future__ import annotations

import ctypes as C
import dataclasses
import math

import torch

from ._lib import KVCacheDesc, ResaError, SelectParams, check, lib

__all__ = ["KVCache", "Workspace", "ResaError", "num_selected", "block_summarize", "append_kv",
           "select_blocks", "append_select", "sparse_decode", "decode_step", "dense_rectify",
           "decode_num_splits", "version"]

HEAD_DIM = 128


def _ptr(t: torch.Tensor | None) -> int | None:
    return None if t is None else t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _need(t: torch.Tensor, name: str, dtype, shape=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on the GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return t


def version() -> str:
    return lib().resa_version().decode()


@dataclasses.dataclass
class KVCache:
    """A layer's KV cache and block-key cache (caller-owned device tensors).

    Contiguous layout: k, v are ``[B, Hkv, capacity, 128]``. Paged layout
    (``block_table`` given): k, v are page pools ``[num_pages, Hkv,
    block_size, 128]`` and ``block_table`` (int32 ``[B, capacity /
    block_size]``) names the page of each logical block of each sequence.
    Summaries are per sequence in both layouts."""

    k: torch.Tensor      # bf16 [B, Hkv, capacity, 128] or [num_pages, Hkv, b, 128]
    v: torch.Tensor
    kmin: torch.Tensor   # bf16 [B, Hkv, capacity / block_size, 128]
    kmax: torch.Tensor
    block_size: int
    block_table: torch.Tensor | None = None  # int32 [B, capacity / block_size]

    @classmethod
    def empty(cls, batch, kv_heads, capacity, block_size, device="cuda"):
        shape = (batch, kv_heads, capacity, HEAD_DIM)
        mb = capacity // block_size
        mk = dict(dtype=torch.bfloat16, device=device)
        return cls(torch.zeros(shape, **mk), torch.zeros(shape, **mk),
                   torch.zeros((batch, kv_heads, mb, HEAD_DIM), **mk),
                   torch.zeros((batch, kv_heads, mb, HEAD_DIM), **mk), block_size)

    @classmethod
    def empty_paged(cls, batch, kv_heads, capacity, block_size, num_pages, device="cuda"):
        """Zeroed page pools of ``num_pages`` pages and an identity-free table
        (all entries -1: the caller assigns pages)."""
        mk = dict(dtype=torch.bfloat16, device=device)
        pool = (num_pages, kv_heads, block_size, HEAD_DIM)
        mb = capacity // block_size
        return cls(torch.zeros(pool, **mk), torch.zeros(pool, **mk),
                   torch.zeros((batch, kv_heads, mb, HEAD_DIM), **mk),
                   torch.zeros((batch, kv_heads, mb, HEAD_DIM), **mk), block_size,
                   torch.full((batch, mb), -1, dtype=torch.int32, device=device))

    @property
    def paged(self) -> bool:
        return self.block_table is not None

    @property
    def batch(self):
        return self.kmin.shape[0]

    @property
    def kv_heads(self):
        return self.k.shape[1]

    @property
    def capacity(self):
        return self.kmin.shape[2] * self.block_size

    def desc(self) -> KVCacheDesc:
        for name in ("k", "v", "kmin", "kmax"):
            _need(getattr(self, name), name, torch.bfloat16)
        B, H, mb = self.kmin.shape[0], self.kmin.shape[1], self.kmin.shape[2]
        if self.block_table is None:
            _need(self.k, "k", torch.bfloat16, (B, H, mb * self.block_size, HEAD_DIM))
            _need(self.v, "v", torch.bfloat16, (B, H, mb * self.block_size, HEAD_DIM))
            return KVCacheDesc(self.k.data_ptr(), self.v.data_ptr(), self.kmin.data_ptr(),
                               self.kmax.data_ptr(), B, H, HEAD_DIM, mb * self.block_size,
                               self.block_size, None, 0)
        P = self.k.shape[0]
        _need(self.k, "k", torch.bfloat16, (P, H, self.block_size, HEAD_DIM))
        _need(self.v, "v", torch.bfloat16, (P, H, self.block_size, HEAD_DIM))
        _need(self.block_table, "block_table", torch.int32, (B, mb))
        return KVCacheDesc(self.k.data_ptr(), self.v.data_ptr(), self.kmin.data_ptr(),
                           self.kmax.data_ptr(), B, H, HEAD_DIM, mb * self.block_size,
                           self.block_size, self.block_table.data_ptr(), P)


class Workspace:
    """A zero-initialised device scratch buffer that grows on demand.

    Use one per operation kind. The decode kernel keeps one merge counter per
    group at the start of its workspace and leaves it at zero after every
    call (and a count of merged calls that tags its ready flags), so the
    buffer is cleared only when it is (re)allocated. Calls that
    share a workspace must be ordered on one stream.
    """

    def __init__(self, device="cuda"):
        self.device = device
        self.buf = None

    def get(self, nbytes: int) -> torch.Tensor:
        if self.buf is None or self.buf.numel() < nbytes:
            self.buf = torch.zeros(max(nbytes, 256), dtype=torch.uint8, device=self.device)
        return self.buf


def num_selected(num_blocks: int, sparsity: float, min_blocks: int, n_local: int) -> int:
    """Eq. 5 block count (host arithmetic of the library)."""
    n = lib().resa_num_selected(num_blocks, sparsity, min_blocks, n_local)
    if n < 0:
        raise ResaError(1, lib().resa_last_error().decode())
    return n


def decode_num_splits(batch, kv_heads, n_cap, block_size) -> int:
    return lib().resa_decode_num_splits(batch, kv_heads, n_cap, block_size)


def block_summarize(cache: KVCache, seq_lens: torch.Tensor, blk_begin: int = 0, blk_end: int = -1,
                    stream=None) -> None:
    """Eq. 3 summaries of blocks [blk_begin, blk_end) of every sequence."""
    _need(seq_lens, "seq_lens", torch.int32, (cache.batch,))
    d = cache.desc()
    check(lib().resa_block_summarize(C.byref(d), seq_lens.data_ptr(), blk_begin, blk_end,
                                     _stream(stream)))


def append_kv(cache: KVCache, k_new: torch.Tensor, v_new: torch.Tensor, seq_lens: torch.Tensor,
              max_seq_len: int, stream=None) -> None:
    """Alg. 1 append of one token per sequence; seq_lens is incremented in place."""
    shape = (cache.batch, cache.kv_heads, HEAD_DIM)
    _need(k_new, "k_new", torch.bfloat16, shape)
    _need(v_new, "v_new", torch.bfloat16, shape)
    _need(seq_lens, "seq_lens", torch.int32, (cache.batch,))
    d = cache.desc()
    check(lib().resa_append_kv(C.byref(d), k_new.data_ptr(), v_new.data_ptr(), seq_lens.data_ptr(),
                               max_seq_len, _stream(stream)))


def select_blocks(cache: KVCache, q: torch.Tensor, seq_lens: torch.Tensor, max_seq_len: int,
                  sparsity: float, min_blocks: int, n_local: int = 1, n_cap: int | None = None,
                  block_idx: torch.Tensor | None = None, num_sel: torch.Tensor | None = None,
                  scores_out: torch.Tensor | None = None, workspace: Workspace | None = None,
                  stream=None):
    """Pooled-query Quest scores (Eq. 4) and the Eq. 5 top-n per group.

    Returns ``(block_idx [B, Hkv, n_cap] int32 ascending, -1 padded,
    num_sel [B, Hkv] int32)``.
    """
    B, Hkv = cache.batch, cache.kv_heads
    hq = q.shape[1]
    _need(q, "q", torch.bfloat16, (B, hq, HEAD_DIM))
    _need(seq_lens, "seq_lens", torch.int32, (B,))
    mseq = -(-max_seq_len // cache.block_size)
    if n_cap is None:
        n_cap = max(num_selected(mseq, sparsity, min_blocks, n_local), 1)
    if block_idx is None:
        block_idx = torch.empty((B, Hkv, n_cap), dtype=torch.int32, device=q.device)
    if num_sel is None:
        num_sel = torch.empty((B, Hkv), dtype=torch.int32, device=q.device)
    _need(block_idx, "block_idx", torch.int32, (B, Hkv, n_cap))
    _need(num_sel, "num_sel", torch.int32, (B, Hkv))
    if scores_out is not None:
        _need(scores_out, "scores_out", torch.float32, (B, Hkv, mseq))
    ws_bytes = lib().resa_select_workspace_size(B, Hkv, max_seq_len, cache.block_size)
    ws = (workspace or Workspace(q.device)).get(ws_bytes)
    ws_ptr, ws_bytes = ws.data_ptr(), ws.numel()
    params = SelectParams(float(sparsity), int(min_blocks), int(n_local))
    d = cache.desc()
    check(lib().resa_select_blocks(C.byref(d), q.data_ptr(), hq, seq_lens.data_ptr(), max_seq_len,
                                   C.byref(params), block_idx.data_ptr(), num_sel.data_ptr(), n_cap,
                                   _ptr(scores_out), ws_ptr, ws_bytes, _stream(stream)))
    return block_idx, num_sel


def append_select(cache: KVCache, k_new: torch.Tensor, v_new: torch.Tensor, q: torch.Tensor,
                  seq_lens: torch.Tensor, max_seq_len: int, sparsity: float, min_blocks: int,
                  n_local: int = 1, n_cap: int | None = None, block_idx: torch.Tensor | None = None,
                  num_sel: torch.Tensor | None = None, scores_out: torch.Tensor | None = None,
                  workspace: Workspace | None = None, stream=None):
    """Alg. 1 append of one token per sequence fused with the Eq. 4-5
    selection over the grown sequences (one launch); seq_lens is incremented
    in place. ``max_seq_len`` bounds seq_lens before the call. Returns
    ``(block_idx, num_sel)`` as :func:`select_blocks`."""
    B, Hkv = cache.batch, cache.kv_heads
    hq = q.shape[1]
    shape = (B, Hkv, HEAD_DIM)
    _need(k_new, "k_new", torch.bfloat16, shape)
    _need(v_new, "v_new", torch.bfloat16, shape)
    _need(q, "q", torch.bfloat16, (B, hq, HEAD_DIM))
    _need(seq_lens, "seq_lens", torch.int32, (B,))
    sel_len = max_seq_len + 1
    mseq = -(-sel_len // cache.block_size)
    if n_cap is None:
        n_cap = max(num_selected(mseq, sparsity, min_blocks, n_local), 1)
    if block_idx is None:
        block_idx = torch.empty((B, Hkv, n_cap), dtype=torch.int32, device=q.device)
    if num_sel is None:
        num_sel = torch.empty((B, Hkv), dtype=torch.int32, device=q.device)
    _need(block_idx, "block_idx", torch.int32, (B, Hkv, n_cap))
    _need(num_sel, "num_sel", torch.int32, (B, Hkv))
    if scores_out is not None:
        _need(scores_out, "scores_out", torch.float32, (B, Hkv, mseq))
    ws_bytes = lib().resa_select_workspace_size(B, Hkv, sel_len, cache.block_size)
    ws = (workspace or Workspace(q.device)).get(ws_bytes)
    params = SelectParams(float(sparsity), int(min_blocks), int(n_local))
    d = cache.desc()
    check(lib().resa_append_select(C.byref(d), k_new.data_ptr(), v_new.data_ptr(), q.data_ptr(), hq,
                                   seq_lens.data_ptr(), max_seq_len, C.byref(params),
                                   block_idx.data_ptr(), num_sel.data_ptr(), n_cap, _ptr(scores_out),
                                   ws.data_ptr(), ws.numel(), _stream(stream)))
    return block_idx, num_sel


def sparse_decode(cache: KVCache, q: torch.Tensor, seq_lens: torch.Tensor, block_idx: torch.Tensor,
                  num_sel: torch.Tensor, num_splits: int = 0, sm_scale: float | None = None,
                  out: torch.Tensor | None = None, lse: torch.Tensor | None = None,
                  with_lse: bool = True, workspace: Workspace | None = None, stream=None):
    """Eq. 2 / Alg. 2 block-sparse flash decoding. Returns ``(out fp32 [B, Hq, 128],
    lse fp32 [B, Hq] or None)``."""
    B, Hkv = cache.batch, cache.kv_heads
    hq = q.shape[1]
    _need(q, "q", torch.bfloat16, (B, hq, HEAD_DIM))
    _need(seq_lens, "seq_lens", torch.int32, (B,))
    n_cap = block_idx.shape[-1]
    _need(block_idx, "block_idx", torch.int32, (B, Hkv, n_cap))
    _need(num_sel, "num_sel", torch.int32, (B, Hkv))
    if sm_scale is None:
        sm_scale = 1.0 / math.sqrt(HEAD_DIM)
    if out is None:
        out = torch.empty((B, hq, HEAD_DIM), dtype=torch.float32, device=q.device)
    _need(out, "out", torch.float32, (B, hq, HEAD_DIM))
    if lse is None and with_lse:
        lse = torch.empty((B, hq), dtype=torch.float32, device=q.device)
    if lse is not None:
        _need(lse, "lse", torch.float32, (B, hq))
    ws_bytes = lib().resa_decode_workspace_size(B, Hkv, hq, n_cap, cache.block_size, num_splits)
    ws = (workspace or Workspace(q.device)).get(ws_bytes)
    d = cache.desc()
    check(lib().resa_sparse_decode(C.byref(d), q.data_ptr(), hq, seq_lens.data_ptr(),
                                   block_idx.data_ptr(), num_sel.data_ptr(), n_cap, num_splits,
                                   float(sm_scale), out.data_ptr(), _ptr(lse), ws.data_ptr(),
                                   ws.numel(), _stream(stream)))
    return out, lse


def decode_step(cache: KVCache, k_new: torch.Tensor, v_new: torch.Tensor, q: torch.Tensor,
                seq_lens: torch.Tensor, max_seq_len: int, sparsity: float, min_blocks: int,
                n_local: int = 1, n_cap: int | None = None, num_splits: int = 0,
                sm_scale: float | None = None, block_idx: torch.Tensor | None = None,
                num_sel: torch.Tensor | None = None, out: torch.Tensor | None = None,
                lse: torch.Tensor | None = None, with_lse: bool = True,
                workspace: Workspace | None = None, stream=None):
    """One decode token (Alg. 1) in one launch: append (seq_lens incremented
    in place), Eq. 4-5 selection and Eq. 2 / Alg. 2 sparse decoding.
    ``max_seq_len`` bounds seq_lens before the call. Returns
    ``(block_idx, num_sel, out, lse)`` as :func:`append_select` and
    :func:`sparse_decode`."""
    B, Hkv = cache.batch, cache.kv_heads
    hq = q.shape[1]
    shape = (B, Hkv, HEAD_DIM)
    _need(k_new, "k_new", torch.bfloat16, shape)
    _need(v_new, "v_new", torch.bfloat16, shape)
    _need(q, "q", torch.bfloat16, (B, hq, HEAD_DIM))
    _need(seq_lens, "seq_lens", torch.int32, (B,))
    mseq = -(-(max_seq_len + 1) // cache.block_size)
    if n_cap is None:
        n_cap = max(num_selected(mseq, sparsity, min_blocks, n_local), 1)
    if block_idx is None:
        block_idx = torch.empty((B, Hkv, n_cap), dtype=torch.int32, device=q.device)
    if num_sel is None:
        num_sel = torch.empty((B, Hkv), dtype=torch.int32, device=q.device)
    _need(block_idx, "block_idx", torch.int32, (B, Hkv, n_cap))
    _need(num_sel, "num_sel", torch.int32, (B, Hkv))
    if sm_scale is None:
        sm_scale = 1.0 / math.sqrt(HEAD_DIM)
    if out is None:
        out = torch.empty((B, hq, HEAD_DIM), dtype=torch.float32, device=q.device)
    _need(out, "out", torch.float32, (B, hq, HEAD_DIM))
    if lse is None and with_lse:
        lse = torch.empty((B, hq), dtype=torch.float32, device=q.device)
    if lse is not None:
        _need(lse, "lse", torch.float32, (B, hq))
    ws_bytes = lib().resa_step_workspace_size(B, Hkv, hq, max_seq_len, cache.block_size, n_cap,
                                              num_splits)
    ws = (workspace or Workspace(q.device)).get(ws_bytes)
    params = SelectParams(float(sparsity), int(min_blocks), int(n_local))
    d = cache.desc()
    check(lib().resa_decode_step(C.byref(d), k_new.data_ptr(), v_new.data_ptr(), q.data_ptr(), hq,
                                 seq_lens.data_ptr(), max_seq_len, C.byref(params),
                                 block_idx.data_ptr(), num_sel.data_ptr(), n_cap, num_splits,
                                 float(sm_scale), out.data_ptr(), _ptr(lse), ws.data_ptr(), ws.numel(),
                                 _stream(stream)))
    return block_idx, num_sel, out, lse


def dense_rectify(cache: KVCache, q_f: torch.Tensor, k_f: torch.Tensor, v_f: torch.Tensor,
                  seq_lens: torch.Tensor, max_seq_len: int, sm_scale: float | None = None,
                  out: torch.Tensor | None = None, lse: torch.Tensor | None = None,
                  with_lse: bool = True, refresh: bool = True, workspace: Workspace | None = None,
                  seq_mask: torch.Tensor | None = None, stream=None):
    """Sec. 2.2 rectification of the last f rows. Returns ``(out fp32 [B, Hq, f, 128], lse)``.
    ``seq_mask`` (int32 [B] on the device, or None for every sequence) selects the
    sequences rectified by this call; the others are left untouched."""
    B, Hkv = cache.batch, cache.kv_heads
    hq, f = q_f.shape[1], q_f.shape[2]
    _need(q_f, "q_f", torch.bfloat16, (B, hq, f, HEAD_DIM))
    _need(k_f, "k_f", torch.bfloat16, (B, Hkv, f, HEAD_DIM))
    _need(v_f, "v_f", torch.bfloat16, (B, Hkv, f, HEAD_DIM))
    _need(seq_lens, "seq_lens", torch.int32, (B,))
    if seq_mask is not None:
        _need(seq_mask, "seq_mask", torch.int32, (B,))
    if sm_scale is None:
        sm_scale = 1.0 / math.sqrt(HEAD_DIM)
    if out is None:
        out = torch.empty((B, hq, f, HEAD_DIM), dtype=torch.float32, device=q_f.device)
    _need(out, "out", torch.float32, (B, hq, f, HEAD_DIM))
    if lse is None and with_lse:
        lse = torch.empty((B, hq, f), dtype=torch.float32, device=q_f.device)
    if lse is not None:
        _need(lse, "lse", torch.float32, (B, hq, f))
    ws_bytes = lib().resa_rectify_workspace_size(B, Hkv, hq, f, max_seq_len)
    ws = (workspace or Workspace(q_f.device)).get(ws_bytes)
    d = cache.desc()
    check(lib().resa_dense_rectify(C.byref(d), q_f.data_ptr(), k_f.data_ptr(), v_f.data_ptr(), hq, f,
                                   seq_lens.data_ptr(), _ptr(seq_mask), max_seq_len, float(sm_scale),
                                   out.data_ptr(), _ptr(lse), int(bool(refresh)), ws.data_ptr(),
                                   ws.numel(), _stream(stream)))
    return out, lse
