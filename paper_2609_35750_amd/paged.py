"""Python binding of the streamed paged KV cache of libkvs (ctypes).

The inference side of KV-streams (Section 2, "KV-streams"; Section 4,
"Inference engine implementation"): one (K, V) entry per generated token in
a paged cache, evicted entries dropped in place, and decode attention over
the entries live when a query is generated.  ``PagedKVCache`` owns the device
pools (torch tensors: memory only) and a native block manager; every step
runs in libkvs (host bookkeeping in C++, updates and attention in HIP
kernels).  Argument marshalling only.
"""
from __future__ import annotations

import ctypes
import math
from typing import Optional, Sequence, Tuple

import numpy as np
import torch

from .kvs import KvsError, _check, _ptr, _stream, _workspace, lib


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _np_ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


class BlockManager:
    """Host-side block bookkeeping (``kvs_bm_*``)."""

    def __init__(self, num_blocks: int, block_size: int, num_seqs: int, max_blocks: int):
        h = ctypes.c_void_p()
        _check("kvs_bm_create", lib.kvs_bm_create(num_blocks, block_size, num_seqs, max_blocks, ctypes.byref(h)))
        self._h = h
        self.num_blocks, self.block_size, self.num_seqs, self.max_blocks = num_blocks, block_size, num_seqs, max_blocks

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            lib.kvs_bm_destroy(h)
            self._h = None

    def append(self, seq: int, positions: Sequence[int]) -> np.ndarray:
        pos = _i32(positions)
        slots = np.empty_like(pos)
        _check("kvs_bm_append", lib.kvs_bm_append(self._h, seq, _np_ptr(pos), pos.size, _np_ptr(slots)))
        return slots

    def evict(self, seq: int, positions: Sequence[int]) -> np.ndarray:
        pos = _i32(positions)
        slots = np.empty_like(pos)
        _check("kvs_bm_evict", lib.kvs_bm_evict(self._h, seq, _np_ptr(pos), pos.size, _np_ptr(slots)))
        return slots

    def release(self, seq: int) -> np.ndarray:
        slots = np.empty(max(self.live(seq), 1), dtype=np.int32)
        n = ctypes.c_int()
        _check("kvs_bm_release", lib.kvs_bm_release(self._h, seq, _np_ptr(slots), ctypes.byref(n)))
        return slots[: n.value]

    def tables(self) -> Tuple[np.ndarray, np.ndarray]:
        table = np.empty((self.num_seqs, self.max_blocks), dtype=np.int32)
        nblk = np.empty(self.num_seqs, dtype=np.int32)
        _check("kvs_bm_tables", lib.kvs_bm_tables(self._h, _np_ptr(table), _np_ptr(nblk)))
        return table, nblk

    def free_blocks(self) -> int:
        return lib.kvs_bm_free_blocks(self._h)

    def live(self, seq: int) -> int:
        return lib.kvs_bm_live(self._h, seq)


def kvs_paged_append(k_new, v_new, positions, slots, k_cache, v_cache, slot_pos, block_size: int) -> None:
    """``kvs_paged_append``: k_new/v_new [n, Hkv, D] bf16, positions/slots int32 [n] (device)."""
    n, Hkv, D = k_new.shape
    nb = k_cache.shape[0]
    _check("kvs_paged_append", lib.kvs_paged_append(
        _ptr(k_new), _ptr(v_new), _ptr(positions), _ptr(slots), n, _ptr(k_cache), _ptr(v_cache), _ptr(slot_pos),
        nb, block_size, Hkv, D, _stream(k_cache)))


def kvs_paged_evict(slots, slot_pos, num_blocks: int, block_size: int) -> None:
    _check("kvs_paged_evict", lib.kvs_paged_evict(_ptr(slots), slots.numel(), _ptr(slot_pos), num_blocks,
                                                   block_size, _stream(slot_pos)))


def kvs_paged_decode(q, k_cache, v_cache, slot_pos, block_table, seq_blocks, softmax_scale=None,
                     out=None, lse=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """``kvs_paged_decode``: q [S, Hq, D] bf16; caches [num_blocks, Hkv, block_size, D]; returns (O, LSE)."""
    S, Hq, D = q.shape
    nb, Hkv, bs, Dk = k_cache.shape
    if Dk != D or v_cache.shape != k_cache.shape:
        raise ValueError("cache shapes do not match q")
    if q.dtype != torch.bfloat16 or k_cache.dtype != torch.bfloat16 or v_cache.dtype != torch.bfloat16:
        raise ValueError("q and the caches must be bfloat16")
    for t in (slot_pos, block_table, seq_blocks):
        if t.dtype != torch.int32:
            raise ValueError("slot_pos, block_table and seq_blocks must be int32")
    if block_table.dim() != 2 or block_table.shape[0] != S or seq_blocks.shape != (S,):
        raise ValueError("block_table must be [S, max_blocks] and seq_blocks [S]")
    if slot_pos.numel() != nb * bs:
        raise ValueError("slot_pos must hold num_blocks * block_size entries")
    max_blocks = block_table.shape[1]
    scale = 1.0 / math.sqrt(D) if softmax_scale is None else float(softmax_scale)
    o = torch.empty_like(q) if out is None else out
    lse = torch.empty((S, Hq), dtype=torch.float32, device=q.device) if lse is None else lse
    need = lib.kvs_paged_decode_workspace(S, Hq, Hkv, D, max_blocks, bs)
    ws = _workspace(need, q.device)
    _check("kvs_paged_decode", lib.kvs_paged_decode(
        _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(slot_pos), _ptr(block_table), _ptr(seq_blocks), _ptr(o),
        _ptr(lse), S, Hq, Hkv, D, nb, bs, max_blocks, scale, _ptr(ws), need, _stream(q)))
    return o, lse


class PagedKVCache:
    """Device pools of a streamed paged KV cache plus its native block manager.

    ``append(seq, positions, k, v)`` stores new entries, ``evict(seq,
    positions)`` drops entries in place, ``decode(q)`` attends one query per
    sequence over the live entries of every sequence.
    """

    def __init__(self, num_blocks: int, block_size: int, num_seqs: int, max_blocks: int, Hkv: int, D: int,
                 device="cuda"):
        self.bm = BlockManager(num_blocks, block_size, num_seqs, max_blocks)
        self.num_blocks, self.block_size, self.num_seqs, self.max_blocks = num_blocks, block_size, num_seqs, max_blocks
        self.Hkv, self.D = Hkv, D
        self.device = torch.device(device)
        self.k = torch.zeros((num_blocks, Hkv, block_size, D), dtype=torch.bfloat16, device=self.device)
        self.v = torch.zeros_like(self.k)
        self.slot_pos = torch.full((num_blocks * block_size,), -1, dtype=torch.int32, device=self.device)
        self._tables = None

    def append(self, seq: int, positions, k_new: torch.Tensor, v_new: torch.Tensor) -> np.ndarray:
        pos = _i32(positions)
        if k_new.shape != (pos.size, self.Hkv, self.D) or v_new.shape != k_new.shape:
            raise ValueError("k_new/v_new must be [n, Hkv, D]")
        slots = self.bm.append(seq, pos)
        if pos.size:
            kvs_paged_append(k_new.contiguous(), v_new.contiguous(), torch.from_numpy(pos).to(self.device),
                             torch.from_numpy(slots).to(self.device), self.k, self.v, self.slot_pos, self.block_size)
        self._tables = None
        return slots

    def evict(self, seq: int, positions) -> np.ndarray:
        slots = self.bm.evict(seq, _i32(positions))
        if slots.size:
            kvs_paged_evict(torch.from_numpy(slots).to(self.device), self.slot_pos, self.num_blocks, self.block_size)
        self._tables = None
        return slots

    def release(self, seq: int) -> np.ndarray:
        slots = self.bm.release(seq)
        if slots.size:
            kvs_paged_evict(torch.from_numpy(slots).to(self.device), self.slot_pos, self.num_blocks, self.block_size)
        self._tables = None
        return slots

    def device_tables(self) -> Tuple[torch.Tensor, torch.Tensor]:
        if self._tables is None:
            table, nblk = self.bm.tables()
            self._tables = (torch.from_numpy(table).to(self.device), torch.from_numpy(nblk).to(self.device))
        return self._tables

    def decode(self, q: torch.Tensor, softmax_scale=None, out=None, lse=None):
        table, nblk = self.device_tables()
        return kvs_paged_decode(q, self.k, self.v, self.slot_pos, table, nblk, softmax_scale, out, lse)
