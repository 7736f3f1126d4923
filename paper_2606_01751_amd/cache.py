"""Python binding of the segment-level cache manager declared in include/sx_cache.h (ctypes,
argument marshalling only; the bookkeeping runs in libsx).

    c = BlockCache(n_blocks, block_size, limit=0.9)
    tokens, spans = c.pad([(tokens, reuse, extra_key), ...], pad_token)
    s = c.schedule(tokens, spans)          # s.segments / s.block_table / s.src_block_ids
    ... prefill through the kernels (Plan(desc, [s.request(...)], ...)) ...
    c.commit(s.req_id, publish=[(start, length, key, freeze)])
    c.release(s.req_id)
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass

import numpy as np

from . import SxError, lib as _lib

EXPORTED = (
    "sx_cache_pad", "sx_sha256", "sx_cache_virtual_hash", "sx_cache_prefix_hash", "sx_cache_create",
    "sx_cache_destroy", "sx_cache_schedule", "sx_cache_commit", "sx_cache_release", "sx_cache_frozen_add",
    "sx_cache_frozen_delete", "sx_cache_get_stats", "sx_cache_get_block", "sx_cache_free_queue",
)

SX_EFULL = -7
I32, I64, VP, U8P = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.POINTER(ctypes.c_uint8)


class _Piece(ctypes.Structure):
    _fields_ = [("tokens", ctypes.POINTER(I32)), ("n_tokens", I32), ("reuse", I32), ("extra_key", U8P),
                ("extra_key_len", I32)]


class _Span(ctypes.Structure):
    _fields_ = [("start", I32), ("length", I32), ("extra_key", U8P), ("extra_key_len", I32), ("freeze", I32)]


class _Segment(ctypes.Structure):
    _fields_ = [("seq_start", I32), ("length", I32), ("cached", I32), ("old_pos", I32), ("new_pos", I32),
                ("src_block_start", I32)]


class _Info(ctypes.Structure):
    _fields_ = [("request_id", I32), ("n_segments", I32), ("n_blocks", I32), ("n_src_blocks", I32),
                ("n_prefix_hits", I32), ("n_virtual_hits", I32)]


class _Stats(ctypes.Structure):
    _fields_ = [("free", I32), ("in_use", I32), ("frozen", I32), ("idle_frozen", I32), ("prefix_entries", I32),
                ("virtual_entries", I32), ("requests", I32)]


class _Block(ctypes.Structure):
    _fields_ = [("ref", I32), ("frozen", I32), ("in_free_queue", I32), ("n_virtual", I32), ("has_prefix", I32),
                ("hits", I64), ("last_use", I64)]


class CacheFull(SxError):
    pass


_ready = False


def _L():
    global _ready
    L = _lib()
    if not _ready:
        P = ctypes.POINTER
        L.sx_cache_pad.argtypes = [I32, P(_Piece), I32, I32, P(I32), I32, P(I32), P(_Span), I32, P(I32)]
        L.sx_sha256.argtypes = [U8P, I64, U8P]
        L.sx_cache_virtual_hash.argtypes = [P(I32), I32, U8P, I32, U8P]
        L.sx_cache_prefix_hash.argtypes = [U8P, P(I32), I32, U8P, I32, U8P]
        L.sx_cache_create.argtypes = [I32, I32, ctypes.c_double, P(VP)]
        L.sx_cache_destroy.argtypes = [VP]
        L.sx_cache_schedule.argtypes = [VP, P(I32), I32, P(_Span), I32, U8P, I32, P(_Segment), P(I32), P(I32),
                                        P(_Info)]
        L.sx_cache_commit.argtypes = [VP, I32, P(_Span), I32, U8P, I32]
        L.sx_cache_release.argtypes = [VP, I32]
        L.sx_cache_frozen_add.argtypes = [VP, P(I32), I32]
        L.sx_cache_frozen_delete.argtypes = [VP, P(I32), I32]
        L.sx_cache_get_stats.argtypes = [VP, P(_Stats)]
        L.sx_cache_get_block.argtypes = [VP, I32, P(_Block)]
        L.sx_cache_free_queue.argtypes = [VP, P(I32), I32, P(I32)]
        for name in EXPORTED:
            getattr(L, name).restype = I32
        _ready = True
    return L


def _check(st: int) -> None:
    if st != 0:
        msg = _lib().sx_last_error().decode()
        raise (CacheFull if st == SX_EFULL else SxError)(st, msg)


def _ints(xs):
    """(pointer, count) of an int32 copy of xs (token ids and block ids are int32 in the ABI; values
    outside that range raise); the pointer keeps the copy alive."""
    if isinstance(xs, np.ndarray) and xs.dtype == np.int32:
        a = np.ascontiguousarray(xs)
    else:
        wide = np.asarray(xs, dtype=np.int64)
        if wide.size and (wide.min() < -2**31 or wide.max() >= 2**31):
            raise ValueError("value outside the int32 range")
        a = np.ascontiguousarray(wide.astype(np.int32))
    if a.size == 0:
        a = np.zeros(1, np.int32)
        n = 0
    else:
        n = int(a.size)
    ptr = a.ctypes.data_as(ctypes.POINTER(I32))
    ptr._keep = a
    return ptr, n


def _bytes(b: bytes):
    b = bytes(b)
    return (ctypes.c_uint8 * max(len(b), 1)).from_buffer_copy(b + b"\0"), len(b)


def _spans(spans, keep):
    arr = (_Span * max(len(spans), 1))()
    for i, sp in enumerate(spans):
        start, length, key = int(sp[0]), int(sp[1]), bytes(sp[2])
        kb, kn = _bytes(key)
        keep.append(kb)
        arr[i] = _Span(start, length, ctypes.cast(kb, U8P), kn, int(bool(sp[3])) if len(sp) > 3 else 0)
    return arr, len(spans)


def sha256(data: bytes) -> bytes:
    buf, n = _bytes(data)
    out = (ctypes.c_uint8 * 32)()
    _check(_L().sx_sha256(ctypes.cast(buf, U8P), n, out))
    return bytes(out)


def virtual_hash(tokens, extra: bytes) -> bytes:
    t, n = _ints(tokens)
    k, kn = _bytes(extra)
    out = (ctypes.c_uint8 * 32)()
    _check(_L().sx_cache_virtual_hash(t, n, ctypes.cast(k, U8P), kn, out))
    return bytes(out)


def prefix_hash(parent, tokens, extra: bytes = b"") -> bytes:
    t, n = _ints(tokens)
    k, kn = _bytes(extra)
    out = (ctypes.c_uint8 * 32)()
    par = None if parent is None else ctypes.cast(_bytes(parent)[0], U8P)
    _check(_L().sx_cache_prefix_hash(par, t, n, ctypes.cast(k, U8P), kn, out))
    return bytes(out)


def pad(pieces, block_size: int, pad_token: int):
    """Entry padding (sx_cache_pad): pieces [(tokens, reuse, extra_key)] -> (tokens, spans)."""
    keep = []
    arr = (_Piece * max(len(pieces), 1))()
    for i, (toks, reuse, key) in enumerate(pieces):
        t, n = _ints(toks)
        kb, kn = _bytes(key)
        keep += [t, kb]
        arr[i] = _Piece(t, n, int(bool(reuse)), ctypes.cast(kb, U8P), kn)
    nt, ns = I32(), I32()
    L = _L()
    _check(L.sx_cache_pad(int(block_size), arr, len(pieces), int(pad_token), None, 0, ctypes.byref(nt), None, 0,
                          ctypes.byref(ns)))
    out = (I32 * max(nt.value, 1))()
    sp = (_Span * max(ns.value, 1))()
    _check(L.sx_cache_pad(int(block_size), arr, len(pieces), int(pad_token), out, nt.value, ctypes.byref(nt), sp,
                          ns.value, ctypes.byref(ns)))
    spans = [(sp[i].start, sp[i].length, ctypes.string_at(sp[i].extra_key, sp[i].extra_key_len))
             for i in range(ns.value)]
    return list(out[:nt.value]), spans


@dataclass
class Schedule:
    req_id: int
    segments: list              # (seq_start, length, cached, old_pos, new_pos, src_block_start or -1)
    block_table: list
    src_block_ids: list
    n_prefix_hits: int
    n_virtual_hits: int


class BlockCache:
    """One block pool's cache state (sx_cache_create ... sx_cache_destroy)."""

    def __init__(self, n_blocks: int, block_size: int, limit: float = 0.9):
        h = VP()
        _check(_L().sx_cache_create(int(n_blocks), int(block_size), float(limit), ctypes.byref(h)))
        self.handle = h
        self.n_blocks, self.block_size = int(n_blocks), int(block_size)

    def close(self):
        if self.handle:
            _L().sx_cache_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def pad(self, pieces, pad_token: int):
        return pad(pieces, self.block_size, pad_token)

    def schedule(self, tokens, spans=(), prefix_key: bytes = b"") -> Schedule:
        t, T = _ints(tokens)
        keep = []
        sp, ns = _spans(list(spans), keep)
        pk, pn = _bytes(prefix_key)
        nb = max(-(-T // self.block_size), 1)
        segs = (_Segment * nb)()
        table = (I32 * nb)()
        src = (I32 * nb)()
        info = _Info()
        _check(_L().sx_cache_schedule(self.handle, t, T, sp, ns, ctypes.cast(pk, U8P), pn, segs, table, src,
                                      ctypes.byref(info)))
        seg_list = [(g.seq_start, g.length, g.cached, g.old_pos, g.new_pos, g.src_block_start)
                    for g in segs[:info.n_segments]]
        return Schedule(info.request_id, seg_list, list(table[:info.n_blocks]), list(src[:info.n_src_blocks]),
                        info.n_prefix_hits, info.n_virtual_hits)

    def commit(self, req_id: int, publish=(), prefix_key: bytes = b"") -> None:
        keep = []
        sp, ns = _spans(list(publish), keep)
        pk, pn = _bytes(prefix_key)
        _check(_L().sx_cache_commit(self.handle, int(req_id), sp, ns, ctypes.cast(pk, U8P), pn))

    def release(self, req_id: int) -> None:
        _check(_L().sx_cache_release(self.handle, int(req_id)))

    def frozen_add(self, blocks) -> None:
        b, n = _ints(blocks)
        _check(_L().sx_cache_frozen_add(self.handle, b, n))

    def frozen_delete(self, blocks) -> None:
        b, n = _ints(blocks)
        _check(_L().sx_cache_frozen_delete(self.handle, b, n))

    def stats(self) -> dict:
        s = _Stats()
        _check(_L().sx_cache_get_stats(self.handle, ctypes.byref(s)))
        return {f: getattr(s, f) for f, _ in _Stats._fields_}

    def block_info(self, block: int) -> dict:
        s = _Block()
        _check(_L().sx_cache_get_block(self.handle, int(block), ctypes.byref(s)))
        return {f: getattr(s, f) for f, _ in _Block._fields_}

    def free_queue(self) -> list:
        n = I32()
        L = _L()
        _check(L.sx_cache_free_queue(self.handle, None, 0, ctypes.byref(n)))
        out = (I32 * max(n.value, 1))()
        _check(L.sx_cache_free_queue(self.handle, out, n.value, ctypes.byref(n)))
        return list(out[:n.value])
