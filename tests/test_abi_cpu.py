"""C-ABI checks that need no GPU: the library loads, exports every function the header declares,
and rejects bad arguments with status codes (validation happens before any device call)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2606_01751_amd as sx
import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions():
    names = set()
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if h.endswith(".h"):
            text = open(os.path.join(ROOT, "include", h)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"\b(sx_[a-z0-9_]+)\s*\(", text))
    return sorted(names)


def test_library_exports_every_declared_function():
    import paper_2606_01751_amd.cache as cache
    L = sx.lib()
    declared = _header_functions()
    assert set(declared) == set(sx.EXPORTED) | set(cache.EXPORTED)
    for name in declared:
        assert hasattr(L, name), name
    assert L.sx_version().decode().startswith("libsx")


def _desc(**kw):
    base = dict(n_q_heads=8, n_kv_heads=2, head_dim=64, dtype="f32", rope_base=1e4)
    base.update(kw)
    return sx.make_desc(**base)


class _Seg:
    def __init__(self, seq_start, length, cached, old_pos=0, new_pos=0, src_block_start=-1):
        self.seq_start, self.length, self.cached = seq_start, length, cached
        self.old_pos, self.new_pos, self.src_block_start = old_pos, new_pos, src_block_start


class _Req:
    def __init__(self, T, segs, bt, src):
        self.n_tokens, self.segments = T, segs
        self.block_table, self.src_block_ids = np.asarray(bt), np.asarray(src)


def _status(desc, reqs, ndst=8, nsrc=8):
    with pytest.raises(sx.SxError) as e:
        sx.Plan(desc, reqs, ndst, nsrc)
    return e.value.status, str(e.value)


def _good():
    return _Req(40, [_Seg(0, 20, 1, 5, 7, 0), _Seg(20, 20, 0, 0, 27)], [0, 1, 2], [3, 4])


def test_plan_rejects_bad_descriptors():
    r = [_good()]
    assert _status(_desc(n_q_heads=6, n_kv_heads=4), r)[0] == sx.SX_ESHAPE
    # more than 64 query heads per KV head: the scoring streams at most 64 columns per chunk
    assert _status(_desc(n_q_heads=65, n_kv_heads=1), r)[0] == sx.SX_EUNSUPPORTED
    assert _status(_desc(n_q_heads=256, n_kv_heads=2), r)[0] == sx.SX_EUNSUPPORTED
    assert _status(_desc(head_dim=96), r)[0] == sx.SX_EUNSUPPORTED
    assert _status(_desc(block_size=32), r)[0] == sx.SX_EUNSUPPORTED
    assert _status(_desc(dtype=7), r)[0] == sx.SX_EUNSUPPORTED
    assert _status(_desc(rope_base=-1.0), r)[0] == sx.SX_EINVAL
    assert _status(_desc(rope_style=5), r)[0] == sx.SX_EINVAL
    d = _desc()
    d.flags = 2                                   # no such flag
    assert _status(d, r)[0] == sx.SX_EINVAL


def test_plan_rejects_bad_segment_tables():
    d = _desc()
    gap = _Req(40, [_Seg(0, 20, 1, 0, 0, 0), _Seg(21, 19, 0)], [0, 1, 2], [3, 4])
    assert _status(d, [gap])[0] == sx.SX_EINVAL
    short = _Req(40, [_Seg(0, 20, 1, 0, 0, 0)], [0, 1, 2], [3, 4])
    assert _status(d, [short])[0] == sx.SX_EINVAL
    zero = _Req(40, [_Seg(0, 0, 1, 0, 0, 0), _Seg(0, 40, 0)], [0, 1, 2], [3])
    assert _status(d, [zero])[0] == sx.SX_EINVAL
    flag = _Req(40, [_Seg(0, 40, 2, 0, 0, 0)], [0, 1, 2], [3, 4, 5])
    assert _status(d, [flag])[0] == sx.SX_EINVAL
    negpos = _Req(40, [_Seg(0, 40, 1, -5, 0, 0)], [0, 1, 2], [3, 4, 5])
    assert _status(d, [negpos])[0] == sx.SX_EINVAL


def test_plan_rejects_bad_block_ids():
    d = _desc()
    oob_dst = _Req(40, [_Seg(0, 20, 1, 0, 0, 0), _Seg(20, 20, 0)], [0, 1, 99], [3, 4])
    assert _status(d, [oob_dst])[0] == sx.SX_ESHAPE
    oob_src = _Req(40, [_Seg(0, 20, 1, 0, 0, 0), _Seg(20, 20, 0)], [0, 1, 2], [3, 40])
    assert _status(d, [oob_src])[0] == sx.SX_ESHAPE
    short_src = _Req(40, [_Seg(0, 20, 1, 0, 0, 1), _Seg(20, 20, 0)], [0, 1, 2], [3, 4])
    assert _status(d, [short_src])[0] == sx.SX_ESHAPE
    dup = [_Req(20, [_Seg(0, 20, 0)], [0, 1], []), _Req(20, [_Seg(0, 20, 0)], [1, 2], [])]
    st, msg = _status(d, dup)
    assert st == sx.SX_EINVAL and "twice" in msg


def test_error_text_is_thread_local_and_set():
    st, msg = _status(_desc(head_dim=96), [_good()])
    assert "head_dim" in msg


def test_null_arguments_are_rejected():
    L = sx.lib()
    assert L.sx_plan_create(None, None, 0, 1, 1, None) == sx.SX_EINVAL
    assert L.sx_rope_realign(None, None, None, None, None, None) == sx.SX_EINVAL
    assert L.sx_sparseq_score(None, None, None, None, None, None) == sx.SX_EINVAL
    assert L.sx_topk_select(None, None, 0.5, None, None, None) == sx.SX_EINVAL
    assert L.sx_sparse_attn(None, None, None, None, 1, None, None, None, None) == sx.SX_EINVAL
    assert L.sx_kv_scatter(None, None, None, None, None, 1, None, None, None) == sx.SX_EINVAL
    assert L.sx_realign_scatter(None, None, None, None, None, None, None, 1, None, None, None) == sx.SX_EINVAL
    assert L.sx_realign_scatter_layers(None, 1, None, None, None, 1, None) == sx.SX_EINVAL
    d = _desc()
    assert L.sx_full_attn(ctypes.byref(d), None, None, None, None, 1, 1, None, None, None) == sx.SX_EINVAL
    assert L.sx_plan_destroy(None) == sx.SX_OK
    assert L.sx_plan_budget(None, 0.5, None, None) == sx.SX_EINVAL


def test_workload_plans_validate_on_host():
    # every named workload passes host validation: the only failure left without a GPU is the
    # device allocation itself
    import torch
    if torch.cuda.is_available():
        pytest.skip("host-only check")
    for i in (1, 2, 3, 4, 5):
        w = W.config(i)
        desc = sx.make_desc(w.n_q_heads, w.n_kv_heads, w.head_dim, w.dtype, w.rope_base, w.rope_style)
        with pytest.raises(sx.SxError) as e:
            sx.Plan(desc, w.requests, w.n_dst_blocks, w.n_src_blocks)
        assert e.value.status in (sx.SX_ENOMEM, sx.SX_EHIP), str(e.value)


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    # no fallback: without the built library every entry point raises instead of computing
    monkeypatch.setattr(sx, "LIB_PATH", str(tmp_path / "libsx.so"))
    monkeypatch.setattr(sx, "_lib", None)
    with pytest.raises(RuntimeError, match="is missing"):
        sx.lib()
    with pytest.raises(RuntimeError, match="is missing"):
        sx.Plan(_desc(), [_good()], 8, 8)
    import paper_2606_01751_amd.cache as C
    monkeypatch.setattr(C, "_ready", False)
    with pytest.raises(RuntimeError, match="is missing"):
        C.sha256(b"abc")


def test_checked_library_exports_the_same_abi():
    # libsx_checked.so: same entry points, device-side validation of index arrays compiled in
    rel = ctypes.CDLL(sx.RELEASE_LIB_PATH)
    chk = ctypes.CDLL(sx.CHECKED_LIB_PATH)
    for name in _header_functions():
        assert hasattr(chk, name), name
    chk.sx_version.restype = rel.sx_version.restype = ctypes.c_char_p
    assert b"device checks" in chk.sx_version() and b"device checks" not in rel.sx_version()
    sx.use_checked(True)
    try:
        # host validation is unchanged in the checked library
        assert _status(_desc(head_dim=96), [_good()])[0] == sx.SX_EUNSUPPORTED
    finally:
        sx.use_checked(False)


def test_plan_rejects_requests_beyond_the_selection_limit():
    # the selection cuts a request into at most 1024 chunks of 2048 tokens
    d = _desc(n_q_heads=2, n_kv_heads=1, head_dim=64, dtype="bf16")
    T = (1 << 21) + 16
    nblk = T // 16
    st, msg = _status(d, [_Req(T, [_Seg(0, T, 0)], np.arange(nblk), [])], ndst=nblk, nsrc=1)
    assert st == sx.SX_EUNSUPPORTED and "per request" in msg
