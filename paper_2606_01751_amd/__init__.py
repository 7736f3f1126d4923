"""Python binding of libsx, the MI355X (gfx950) library of SparseX's per-layer Sparse-KV
Recomputation step (declared in include/sx.h).

The functions below only marshal arguments: they turn torch tensors into device pointers and
call the C entry point of the same name.  Every step of the computation runs in the library's
HIP kernels; there is no fallback.  If libsx.so is missing, loading raises.

Call pattern of one selecting sparse layer (all on one stream):

    plan = Plan(desc, requests, n_dst_blocks, n_src_blocks)
    rope_realign(plan, src_k, src_v, k_cache, v_cache)
    nr, n_nr, max_nr = plan.nonreused_rows()
    kv_scatter(plan, k, v, k_cache, v_cache, rows=nr, n_rows=n_nr, max_rows=max_nr)
    sparseq_score(plan, q, k_cache, scores, lse_in=None)
    topk_select(plan, scores, ratio, rows, n_rows)
    kv_scatter(plan, k, v, k_cache, v_cache, rows=rows, n_rows=n_rows, max_rows=plan.budget(ratio)[1])
    sparse_attn(plan, q, rows, n_rows, plan.budget(ratio)[1], k_cache, v_cache, out)
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

__all__ = [
    "LIB_PATH", "SxError", "lib", "LayerDesc", "Plan", "rope_realign", "kv_scatter", "realign_scatter",
    "realign_scatter_layers", "rows_mask", "realign_scatter_masked", "sparseq_score", "sparseq_score_static",
    "topk_select", "sparse_attn", "full_attn", "gemm_rows", "gemm_rows_split", "rmsnorm_rows", "rope_rows",
    "silu_mul_rows", "F32", "BF16", "ROPE_NEOX", "ROPE_GPTJ", "TOPK_ALL_POSITIONS", "EXPORTED", "use_checked",
    "RELEASE_LIB_PATH", "CHECKED_LIB_PATH",
]

RELEASE_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsx.so")
# same ABI, index arrays in device memory validated on the device (SX_EDEVICE)
CHECKED_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsx_checked.so")
LIB_PATH = RELEASE_LIB_PATH

F32, BF16 = 0, 1
ROPE_NEOX, ROPE_GPTJ = 0, 1
SX_OK, SX_EINVAL, SX_ESHAPE, SX_EUNSUPPORTED, SX_EHIP, SX_EDEVICE, SX_ENOMEM = 0, -1, -2, -3, -4, -5, -6

EXPORTED = (
    "sx_plan_create", "sx_plan_destroy", "sx_plan_get_info", "sx_plan_budget", "sx_plan_nonreused_rows",
    "sx_rope_realign", "sx_kv_scatter", "sx_realign_scatter", "sx_realign_scatter_layers", "sx_rows_mask",
    "sx_realign_scatter_masked", "sx_sparseq_score", "sx_sparseq_score_static", "sx_topk_select",
    "sx_sparse_attn", "sx_full_attn", "sx_gemm_rows", "sx_gemm_rows_split", "sx_rmsnorm_rows", "sx_rope_rows", "sx_silu_mul_rows",
    "sx_last_error", "sx_version",
)


TOPK_ALL_POSITIONS = 1   # sx_layer_desc.flags: Eq. topk over every position


class SxError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"libsx status {status}: {msg}")
        self.status = status


class LayerDesc(ctypes.Structure):
    _fields_ = [
        ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("block_size", ctypes.c_int32), ("dtype", ctypes.c_int32), ("rope_style", ctypes.c_int32),
        ("rope_base", ctypes.c_double), ("softmax_scale", ctypes.c_float), ("flags", ctypes.c_int32),
    ]


class _Segment(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("seq_start", "length", "cached", "old_pos", "new_pos", "src_block_start")]


class _Request(ctypes.Structure):
    _fields_ = [
        ("n_tokens", ctypes.c_int32), ("n_segments", ctypes.c_int32), ("segments", ctypes.POINTER(_Segment)),
        ("block_table", ctypes.POINTER(ctypes.c_int32)), ("src_block_ids", ctypes.POINTER(ctypes.c_int32)),
        ("n_src_block_ids", ctypes.c_int32),
    ]


class _PlanInfo(ctypes.Structure):
    _fields_ = [
        ("total_tokens", ctypes.c_int64), ("n_requests", ctypes.c_int32), ("max_tokens", ctypes.c_int32),
        ("n_reused", ctypes.c_int64), ("n_nonreused", ctypes.c_int64), ("n_probes", ctypes.c_int64),
        ("n_base", ctypes.c_int64), ("max_nonreused", ctypes.c_int32), ("max_probes", ctypes.c_int32),
        ("device_bytes", ctypes.c_int64),
    ]


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded libsx.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_01751_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, I32, I64, D, VP = ctypes.POINTER, ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p
        L.sx_plan_create.argtypes = [P(LayerDesc), P(_Request), I32, I64, I64, P(VP)]
        L.sx_plan_destroy.argtypes = [VP]
        L.sx_plan_get_info.argtypes = [VP, P(_PlanInfo)]
        L.sx_plan_budget.argtypes = [VP, D, P(I64), P(I32)]
        L.sx_plan_nonreused_rows.argtypes = [VP, P(VP), P(VP), P(I32)]
        L.sx_rope_realign.argtypes = [VP, VP, VP, VP, VP, VP]
        L.sx_kv_scatter.argtypes = [VP, VP, VP, VP, VP, I32, VP, VP, VP]
        L.sx_realign_scatter.argtypes = [VP, VP, VP, VP, VP, VP, VP, I32, VP, VP, VP]
        L.sx_realign_scatter_layers.argtypes = [VP, I32, VP, VP, VP, I32, VP]
        L.sx_rows_mask.argtypes = [VP, VP, VP, I32, VP, VP]
        L.sx_realign_scatter_masked.argtypes = [VP, VP, VP, VP, VP, VP, VP, VP, VP]
        L.sx_sparseq_score.argtypes = [VP, VP, VP, VP, VP, VP]
        L.sx_sparseq_score_static.argtypes = [VP, VP, VP, VP, VP, VP]
        L.sx_topk_select.argtypes = [VP, VP, D, VP, VP, VP]
        L.sx_sparse_attn.argtypes = [VP, VP, VP, VP, I32, VP, VP, VP, VP]
        L.sx_full_attn.argtypes = [P(LayerDesc), VP, VP, VP, VP, I32, I32, VP, VP, VP]
        F = ctypes.c_float
        L.sx_gemm_rows.argtypes = [VP, VP, VP, I32, VP, I32, VP, I32, I32, VP, VP, I32, VP]
        L.sx_gemm_rows_split.argtypes = [VP, VP, VP, I32, VP, I32, VP, I32, I32, P(I32), P(VP), I32, VP]
        L.sx_rmsnorm_rows.argtypes = [VP, VP, VP, I32, VP, I32, VP, F, I32, VP, I32, VP]
        L.sx_rope_rows.argtypes = [VP, VP, VP, I32, VP, VP, VP]
        L.sx_silu_mul_rows.argtypes = [VP, VP, I32, VP, I32, VP, VP]
        for name in EXPORTED:
            if name in ("sx_last_error", "sx_version"):
                getattr(L, name).restype = ctypes.c_char_p
                getattr(L, name).argtypes = []
            else:
                getattr(L, name).restype = ctypes.c_int32
        _lib = L
    return _lib


def use_checked(on: bool = True) -> None:
    """Switch every binding to the checked library (libsx_checked.so) or back to the release one.
    Plans belong to the library that made them: switch before creating them."""
    global LIB_PATH, _lib
    LIB_PATH = CHECKED_LIB_PATH if on else RELEASE_LIB_PATH
    _lib = None


def _check(status: int):
    if status != SX_OK:
        raise SxError(status, lib().sx_last_error().decode())


def _ptr(t) -> Optional[int]:
    """Device pointer of a tensor (None stays NULL)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def make_desc(n_q_heads, n_kv_heads, head_dim, dtype, rope_base, rope_style=ROPE_NEOX, block_size=16,
              softmax_scale=0.0, topk_all_positions=False) -> LayerDesc:
    """A layer descriptor; topk_all_positions sets SX_TOPK_ALL_POSITIONS (Eq. topk over every position)."""
    if isinstance(dtype, str):
        dtype = {"f32": F32, "bf16": BF16}[dtype]
    if isinstance(rope_style, str):
        rope_style = {"neox": ROPE_NEOX, "gptj": ROPE_GPTJ}[rope_style]
    return LayerDesc(n_q_heads, n_kv_heads, head_dim, block_size, dtype, rope_style, float(rope_base),
                     float(softmax_scale), TOPK_ALL_POSITIONS if topk_all_positions else 0)


class Plan:
    """Owns an sx_plan.  `requests` are objects with n_tokens, segments (seq_start, length, cached,
    old_pos, new_pos, src_block_start), block_table and src_block_ids (int sequences)."""

    def __init__(self, desc: LayerDesc, requests: Sequence, n_dst_blocks: int, n_src_blocks: int):
        import numpy as np
        self.desc = desc
        self._keep = []
        reqs = (_Request * len(requests))()
        for i, r in enumerate(requests):
            segs = (_Segment * len(r.segments))()
            for j, s in enumerate(r.segments):
                segs[j] = _Segment(int(s.seq_start), int(s.length), int(s.cached), int(s.old_pos),
                                   int(s.new_pos), int(s.src_block_start))
            bt = np.ascontiguousarray(r.block_table, dtype=np.int32)
            src = np.ascontiguousarray(r.src_block_ids, dtype=np.int32)
            if src.size == 0:
                src = np.zeros(1, dtype=np.int32)
            self._keep += [segs, bt, src]
            reqs[i] = _Request(int(r.n_tokens), len(r.segments), segs,
                               bt.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                               src.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                               int(len(r.src_block_ids)))
        h = ctypes.c_void_p()
        _check(lib().sx_plan_create(ctypes.byref(desc), reqs, len(requests), int(n_dst_blocks), int(n_src_blocks),
                                    ctypes.byref(h)))
        self.handle = h
        self._keep = None

    def close(self):
        if getattr(self, "handle", None) is not None and self.handle.value:
            _check(lib().sx_plan_destroy(self.handle))
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def info(self) -> dict:
        inf = _PlanInfo()
        _check(lib().sx_plan_get_info(self.handle, ctypes.byref(inf)))
        return {n: getattr(inf, n) for n, _ in _PlanInfo._fields_}

    def budget(self, ratio: float):
        """(sum of top-k budgets, max_rows bound) for a recompute ratio."""
        k = ctypes.c_int64()
        m = ctypes.c_int32()
        _check(lib().sx_plan_budget(self.handle, float(ratio), ctypes.byref(k), ctypes.byref(m)))
        return k.value, m.value

    def nonreused_rows(self):
        """(rows device pointer, n_rows device pointer, max_rows) of I_nr owned by the plan."""
        rows, n = ctypes.c_void_p(), ctypes.c_void_p()
        m = ctypes.c_int32()
        _check(lib().sx_plan_nonreused_rows(self.handle, ctypes.byref(rows), ctypes.byref(n), ctypes.byref(m)))
        return rows.value, n.value, m.value


def rope_realign(plan: Plan, src_k, src_v, k_cache, v_cache, stream=None):
    _check(lib().sx_rope_realign(plan.handle, _ptr(src_k), _ptr(src_v), _ptr(k_cache), _ptr(v_cache),
                                 _stream(stream)))


def kv_scatter(plan: Plan, k_new, v_new, k_cache, v_cache, rows=None, n_rows=None, max_rows: int = 0,
               stream=None):
    _check(lib().sx_kv_scatter(plan.handle, _ptr(k_new), _ptr(v_new), _ptr(rows), _ptr(n_rows), int(max_rows),
                               _ptr(k_cache), _ptr(v_cache), _stream(stream)))


def realign_scatter(plan: Plan, src_k, src_v, k_new, v_new, rows, n_rows, max_rows: int, k_cache, v_cache,
                    stream=None):
    _check(lib().sx_realign_scatter(plan.handle, _ptr(src_k), _ptr(src_v), _ptr(k_new), _ptr(v_new), _ptr(rows),
                                    _ptr(n_rows), int(max_rows), _ptr(k_cache), _ptr(v_cache), _stream(stream)))


class _LayerKV(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("src_k", "src_v", "k_new", "v_new", "k_cache", "v_cache")]


def realign_scatter_layers(plan: Plan, layers, rows, n_rows, max_rows: int, stream=None):
    """layers: sequence of (src_k, src_v, k_new, v_new, k_cache, v_cache) per layer."""
    arr = (_LayerKV * max(1, len(layers)))()
    for i, t in enumerate(layers):
        arr[i] = _LayerKV(*(_ptr(x) for x in t))
    _check(lib().sx_realign_scatter_layers(plan.handle, len(layers), ctypes.cast(arr, ctypes.c_void_p), _ptr(rows),
                                           _ptr(n_rows), int(max_rows), _stream(stream)))


def rows_mask(plan: Plan, rows, n_rows, max_rows: int, mask, stream=None):
    """mask (uint8, sum T) = 1 on the listed rows, 0 elsewhere."""
    _check(lib().sx_rows_mask(plan.handle, _ptr(rows), _ptr(n_rows), int(max_rows), _ptr(mask), _stream(stream)))


def realign_scatter_masked(plan: Plan, src_k, src_v, k_new, v_new, mask, k_cache, v_cache, stream=None):
    _check(lib().sx_realign_scatter_masked(plan.handle, _ptr(src_k), _ptr(src_v), _ptr(k_new), _ptr(v_new),
                                           _ptr(mask), _ptr(k_cache), _ptr(v_cache), _stream(stream)))


def sparseq_score(plan: Plan, q, k_cache, scores, lse_in=None, stream=None):
    _check(lib().sx_sparseq_score(plan.handle, _ptr(q), _ptr(k_cache), _ptr(lse_in), _ptr(scores), _stream(stream)))


def sparseq_score_static(plan: Plan, q, k_cache, scores, lse_in, stream=None):
    """sparseq_score in one-pass mode with the library's static scratch: allocates nothing."""
    _check(lib().sx_sparseq_score_static(plan.handle, _ptr(q), _ptr(k_cache), _ptr(lse_in), _ptr(scores),
                                         _stream(stream)))


def topk_select(plan: Plan, scores, ratio: float, rows, n_rows, stream=None):
    _check(lib().sx_topk_select(plan.handle, _ptr(scores), float(ratio), _ptr(rows), _ptr(n_rows),
                                _stream(stream)))


def sparse_attn(plan: Plan, q, rows, n_rows, max_rows: int, k_cache, v_cache, out, stream=None):
    _check(lib().sx_sparse_attn(plan.handle, _ptr(q), _ptr(rows), _ptr(n_rows), int(max_rows), _ptr(k_cache),
                                _ptr(v_cache), _ptr(out), _stream(stream)))


def full_attn(desc: LayerDesc, q, k, v, cu_seqlens, n_requests: int, max_seqlen: int, out, lse=None,
              stream=None):
    _check(lib().sx_full_attn(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(cu_seqlens), int(n_requests),
                              int(max_seqlen), _ptr(out), _ptr(lse), _stream(stream)))


# ---- row-sparse layer body (rows of R only; see include/sx.h) ----

def gemm_rows(plan: Plan, rows, n_rows, max_rows: int, x, w, y, residual=None, x_by_token=False,
              y_by_token=False, stream=None):
    """y[row] = x[row] @ w.T (+ residual[row]); w is [n][k]."""
    n, k = int(w.shape[0]), int(w.shape[1])
    _check(lib().sx_gemm_rows(plan.handle, _ptr(rows), _ptr(n_rows), int(max_rows), _ptr(x), int(bool(x_by_token)),
                              _ptr(w), k, n, _ptr(residual), _ptr(y), int(bool(y_by_token)), _stream(stream)))


def gemm_rows_split(plan: Plan, rows, n_rows, max_rows: int, x, w, ys, x_by_token=False, y_by_token=False,
                    stream=None):
    """One launch of y = x @ w.T for a weight of stacked parts: w is [sum n_i][k] and the columns of
    part i go to ys[i] (its last dimension flattened: [..][n_i])."""
    k = int(w.shape[1])
    widths = [int(y.numel() // y.shape[0]) for y in ys]
    if sum(widths) != int(w.shape[0]):
        raise ValueError(f"output widths {widths} do not add up to the weight's {int(w.shape[0])} rows")
    n = len(ys)
    part_n = (ctypes.c_int32 * n)(*widths)
    y_parts = (ctypes.c_void_p * n)(*[_ptr(y) for y in ys])
    _check(lib().sx_gemm_rows_split(plan.handle, _ptr(rows), _ptr(n_rows), int(max_rows), _ptr(x),
                                    int(bool(x_by_token)), _ptr(w), k, n, part_n, y_parts, int(bool(y_by_token)),
                                    _stream(stream)))


def rmsnorm_rows(plan: Plan, rows, n_rows, max_rows: int, x, gamma, eps: float, y, x_by_token=False,
                 y_by_token=False, stream=None):
    h = int(gamma.shape[0])
    _check(lib().sx_rmsnorm_rows(plan.handle, _ptr(rows), _ptr(n_rows), int(max_rows), _ptr(x),
                                 int(bool(x_by_token)), _ptr(gamma), float(eps), h, _ptr(y), int(bool(y_by_token)),
                                 _stream(stream)))


def rope_rows(plan: Plan, rows, n_rows, max_rows: int, q, k, stream=None):
    _check(lib().sx_rope_rows(plan.handle, _ptr(rows), _ptr(n_rows), int(max_rows), _ptr(q), _ptr(k),
                              _stream(stream)))


def silu_mul_rows(plan: Plan, n_rows, max_rows: int, gate_up, y, stream=None):
    f = int(y.shape[-1])
    _check(lib().sx_silu_mul_rows(plan.handle, _ptr(n_rows), int(max_rows), _ptr(gate_up), f, _ptr(y),
                                  _stream(stream)))
