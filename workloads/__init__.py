"""Seeded synthetic workloads for the Sparse-KV Recomputation step.

This module only builds inputs: segment tables, block tables and random
tensors.  It holds none of the method's arithmetic (no RoPE, no softmax, no
selection), so both the oracle and the HIP path can consume what it makes.

A request is a token sequence of length T cut into contiguous segments
(Section 3.1 and Algorithm 1, input line).  A segment is either *cached* (its
K/V come from an earlier request and sit in a source block pool at their old
RoPE positions) or *uncached* (its tokens form the Sparse-Q rows, Section 3.2).
Fresh per-token Q/K/V stand in for the projections of the current pass and are
drawn for every token; the path reads only the rows it needs.

The five named workloads follow the shapes of the paper's evaluation inputs
(RAG chunks, multi-round chat, agent workflows and a serving batch,
Section 4 and Appendix B).  The datasets themselves are not used: every tensor
is N(0,1) noise with the layout rules documented per builder below.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence

import numpy as np

__all__ = [
    "Segment", "Request", "Workload", "config", "config_names", "custom_workload",
    "random_request", "layer_tensors", "layer_tensors_torch", "round_bf16",
]


@dataclasses.dataclass(frozen=True)
class Segment:
    """One contiguous run of tokens of a request.

    seq_start/length: token indices [seq_start, seq_start+length) of the new sequence.
    cached: True for a reused segment, False for an uncached (Sparse-Q) one.
    old_pos: RoPE position of the first token in the request that cached it (cached only).
    new_pos: RoPE position of the first token in the current request.
    src_block_start: index into Request.src_block_ids of the segment's first source block
                     (cached only, -1 otherwise); the segment starts at slot 0 of that block.
    """
    seq_start: int
    length: int
    cached: bool
    old_pos: int
    new_pos: int
    src_block_start: int = -1


@dataclasses.dataclass
class Request:
    n_tokens: int
    segments: List[Segment]
    block_table: np.ndarray      # int32 [ceil(T/b)]: destination-pool block of each logical block
    src_block_ids: np.ndarray    # int32: source-pool blocks, indexed by Segment.src_block_start
    planted: np.ndarray          # int64 request-local token indices whose cached K row is scaled

    def cached_mask(self) -> np.ndarray:
        m = np.zeros(self.n_tokens, dtype=bool)
        for s in self.segments:
            if s.cached:
                m[s.seq_start:s.seq_start + s.length] = True
        return m


@dataclasses.dataclass
class Workload:
    name: str
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    block_size: int
    dtype: str                   # "f32" or "bf16": storage type of Q/K/V, caches and outputs
    rope_base: float
    rope_style: str              # "neox" (pairs i, i+d/2) or "gptj" (pairs 2i, 2i+1)
    ratios: Sequence[float]      # recompute ratios to run
    n_layers: int
    n_full_layers: int           # layers [0, n_full_layers) run full attention (hybrid threshold)
    requests: List[Request]
    n_dst_blocks: int
    n_src_blocks: int
    plant_scale: float = 4.0
    description: str = ""
    config_id: int = 0

    @property
    def total_tokens(self) -> int:
        return sum(r.n_tokens for r in self.requests)

    @property
    def token_offsets(self) -> np.ndarray:
        off = np.zeros(len(self.requests) + 1, dtype=np.int64)
        off[1:] = np.cumsum([r.n_tokens for r in self.requests])
        return off


# --------------------------------------------------------------------------------------
# Seeding
# --------------------------------------------------------------------------------------

_LAYOUT = 0
_Q, _K, _V, _KSRC, _VSRC = 1, 2, 3, 4, 5


def _rng(*key: int) -> np.random.Generator:
    """Philox stream keyed by (config, layer, request, tensor id, seed)."""
    return np.random.Generator(np.random.Philox(np.random.SeedSequence([int(k) & 0xFFFFFFFF for k in key])))


# --------------------------------------------------------------------------------------
# Request assembly
# --------------------------------------------------------------------------------------

def _assemble(seg_specs, b: int, dst_blocks: np.ndarray, src_alloc, planted=None) -> Request:
    """seg_specs: list of (length, cached, old_pos, new_pos).  new_pos None -> seq_start.

    dst_blocks: destination block ids for the request's logical blocks.
    src_alloc: callable(n_blocks) -> np.ndarray of source block ids (consumed in order).
    """
    segs: List[Segment] = []
    src_ids: List[np.ndarray] = []
    n_src = 0
    t = 0
    for (length, cached, old_pos, new_pos) in seg_specs:
        assert length > 0
        if new_pos is None:
            new_pos = t
        if cached:
            nb = -(-length // b)
            ids = src_alloc(nb)
            src_ids.append(ids)
            segs.append(Segment(t, length, True, int(old_pos), int(new_pos), n_src))
            n_src += nb
        else:
            segs.append(Segment(t, length, False, 0, int(new_pos), -1))
        t += length
    T = t
    nblk = -(-T // b)
    assert len(dst_blocks) >= nblk
    src = np.concatenate(src_ids).astype(np.int32) if src_ids else np.zeros(0, np.int32)
    pl = np.asarray(planted if planted is not None else [], dtype=np.int64)
    return Request(T, segs, np.asarray(dst_blocks[:nblk], dtype=np.int32), src, pl)


class _SrcAllocator:
    def __init__(self, order: np.ndarray):
        self.order = order
        self.used = 0

    def __call__(self, n: int) -> np.ndarray:
        ids = self.order[self.used:self.used + n]
        assert len(ids) == n, "source pool exhausted"
        self.used += n
        return ids


def _planted_positions(rng: np.random.Generator, req_segments, fraction=None, per_segment=None) -> np.ndarray:
    """Token indices of planted high-norm keys inside cached segments."""
    out = []
    for (start, length, cached) in req_segments:
        if not cached:
            continue
        if per_segment is not None:
            n = min(per_segment, length)
        else:
            n = int(math.floor(fraction * length))
        if n > 0:
            out.append(start + np.sort(rng.choice(length, size=n, replace=False)))
    return np.concatenate(out) if out else np.zeros(0, np.int64)


def _fix_sum(units: np.ndarray, target: int, lo: int, hi: int, rng: np.random.Generator) -> np.ndarray:
    """Nudge integer parts by one unit at random indices until they sum to target within [lo, hi]."""
    units = units.copy()
    guard = 0
    while units.sum() != target:
        i = rng.integers(len(units))
        if units.sum() > target and units[i] > lo:
            units[i] -= 1
        elif units.sum() < target and units[i] < hi:
            units[i] += 1
        guard += 1
        assert guard < 10_000_000
    return units


# --------------------------------------------------------------------------------------
# The five named workloads
# --------------------------------------------------------------------------------------

def _c1(seed: int) -> Workload:
    """T=512 fp32 layer, 8/2 heads, d=64, base 1e4, identity block tables.

    Segments in sequence order: cached 128 (old 0, new 64), uncached 64 (new 192),
    cached 192 (old 0, new 300: a +300 shift), uncached 128 (new 492).  Positions
    rise monotonically with a gap 256-299.  Eight planted keys (x4) per cached segment.
    """
    b = 16
    specs = [(128, True, 0, 64), (64, False, 0, 192), (192, True, 0, 300), (128, False, 0, 492)]
    rng = _rng(1, 0, 0, _LAYOUT, seed)
    src = _SrcAllocator(np.arange(20, dtype=np.int32))
    starts = np.cumsum([0] + [s[0] for s in specs[:-1]])
    planted = _planted_positions(rng, [(int(st), s[0], s[1]) for st, s in zip(starts, specs)], per_segment=8)
    req = _assemble(specs, b, np.arange(32, dtype=np.int32), src, planted)
    return Workload("c1", 8, 2, 64, b, "f32", 1e4, "neox", (0.15,), 1, 0, [req], 32, 20,
                    description="T=512 fp32, 8/2 heads, d=64, 4 segments (128c,64u,192c,128u), r=15%",
                    config_id=1)


def _c2(seed: int) -> Workload:
    """Llama-3-8B-shaped RAG layer: T=8192, 32/8/128 bf16, base 5e5.

    [256 uncached system prompt][12 cached 512-token chunks, seeded order, each with its own
    cached start position in [0,4096)][1792 uncached question].  2% planted keys per chunk
    (10 of 512).  Destination blocks: seeded permutation of 512 blocks.
    """
    b = 16
    rng = _rng(2, 0, 0, _LAYOUT, seed)
    chunk_ids = rng.permutation(12)
    old = rng.integers(0, 4096, size=12)
    specs = [(256, False, 0, None)]
    for c in chunk_ids:
        specs.append((512, True, int(old[c]), None))
    specs.append((1792, False, 0, None))
    src = _SrcAllocator(rng.permutation(12 * 32).astype(np.int32))
    starts = np.cumsum([0] + [s[0] for s in specs[:-1]])
    planted = _planted_positions(rng, [(int(st), s[0], s[1]) for st, s in zip(starts, specs)], per_segment=10)
    req = _assemble(specs, b, rng.permutation(512).astype(np.int32), src, planted)
    return Workload("c2", 32, 8, 128, b, "bf16", 5e5, "neox", (0.15,), 1, 0, [req], 512, 384,
                    description="T=8192 bf16 RAG layer, 32/8/128, 12x512 cached chunks, r=15%",
                    config_id=2)


def _c3(seed: int) -> Workload:
    """32-layer hybrid stack, T=32768 multi-round chat, 32/8/128 bf16, base 5e5, threshold 4.

    20 cached history turns (multiples of 16 in [1008,2000], summing to 30720); two uncached
    512-token tool outputs inserted after two seeded turns; a final uncached 1024-token turn.
    A turn's cached position is its offset in the history without the tool outputs, so the
    shift is 0, 512 or 1024.  No planted keys.
    """
    b = 16
    rng = _rng(3, 0, 0, _LAYOUT, seed)
    units = _fix_sum(rng.integers(63, 126, size=20), 1920, 63, 125, rng)
    lens = units * 16
    tool_after = set(int(x) for x in rng.choice(20, size=2, replace=False))
    specs = []
    hist = 0
    for m in range(20):
        specs.append((int(lens[m]), True, hist, None))
        hist += int(lens[m])
        if m in tool_after:
            specs.append((512, False, 0, None))
    specs.append((1024, False, 0, None))
    src = _SrcAllocator(rng.permutation(30720 // 16).astype(np.int32))
    req = _assemble(specs, b, rng.permutation(2048).astype(np.int32), src, None)
    assert req.n_tokens == 32768
    return Workload("c3", 32, 8, 128, b, "bf16", 5e5, "neox", (0.15,), 32, 4, [req], 2048, 1920,
                    description="T=32768 bf16 32-layer hybrid chat stack (4 full + 28 sparse), r=15%",
                    config_id=3)


def _c4(seed: int) -> Workload:
    """Qwen-style agent layer: T=65536, 28/4/128 bf16, base 1e6, ratios 5/10/20 (+15)%.

    48 cached segments (log-uniform 256-4096) from 6 agent sources and 16 uncached segments
    (log-uniform 64-512); lengths rounded to 16 and scaled to total 65536; seeded interleave with
    the last segment cached (tail fallback).  A cached segment's old position is its offset in its
    source's transcript.  1% of cached keys planted.
    """
    b = 16
    T = 65536
    rng = _rng(4, 0, 0, _LAYOUT, seed)
    c_len = np.exp(rng.uniform(np.log(256), np.log(4096), size=48))
    u_len = np.exp(rng.uniform(np.log(64), np.log(512), size=16))
    f = T / (c_len.sum() + u_len.sum())
    c_u = np.maximum(1, np.round(c_len * f / 16)).astype(np.int64)
    u_u = np.maximum(1, np.round(u_len * f / 16)).astype(np.int64)
    c_u = _fix_sum(c_u, T // 16 - int(u_u.sum()), 1, 1 << 30, rng)
    kinds = [("c", i) for i in range(48)] + [("u", i) for i in range(16)]
    order = [kinds[i] for i in rng.permutation(64)]
    if order[-1][0] == "u":
        j = max(i for i, k in enumerate(order[:-1]) if k[0] == "c")
        order[-1], order[j] = order[j], order[-1]
    source = rng.integers(0, 6, size=48)
    # per-source transcript: segments of the source in a seeded order
    old_pos = np.zeros(48, dtype=np.int64)
    for s in range(6):
        mem = np.flatnonzero(source == s)
        mem = mem[rng.permutation(len(mem))]
        off = 0
        for i in mem:
            old_pos[i] = off
            off += int(c_u[i]) * 16
    specs = []
    for kind, i in order:
        if kind == "c":
            specs.append((int(c_u[i]) * 16, True, int(old_pos[i]), None))
        else:
            specs.append((int(u_u[i]) * 16, False, 0, None))
    n_src = int(c_u.sum())
    src = _SrcAllocator(rng.permutation(n_src).astype(np.int32))
    starts = np.cumsum([0] + [s[0] for s in specs[:-1]])
    cached_tok = np.concatenate([np.arange(st, st + s[0]) for st, s in zip(starts, specs) if s[1]])
    planted = np.sort(rng.choice(cached_tok, size=len(cached_tok) // 100, replace=False))
    req = _assemble(specs, b, rng.permutation(T // 16).astype(np.int32), src, planted)
    return Workload("c4", 28, 4, 128, b, "bf16", 1e6, "neox", (0.05, 0.10, 0.20, 0.15), 1, 0, [req],
                    T // 16, n_src,
                    description="T=65536 bf16 agent layer, 28/4/128, 48 cached + 16 uncached segments",
                    config_id=4)


def _dirichlet_units(rng, total_units: int, n: int) -> np.ndarray:
    w = rng.dirichlet(np.ones(n))
    u = np.maximum(1, np.floor(w * total_units)).astype(np.int64)
    return _fix_sum(u, total_units, 1, 1 << 30, rng)


def _c5(seed: int) -> Workload:
    """Serving batch: 8 requests, ~400k tokens, 32/8/128 bf16, base 5e5, 32 layers, threshold 4.

    Request lengths: multiples of 16 in [16384,131072] scaled to 400000 in total.  Each request is
    70-95% cached, split (Dirichlet) into 8-64 cached and 2-8 uncached segments in a seeded order;
    odd-numbered requests end with a cached segment, even-numbered ones with an uncached one.
    A cached segment's old position is its new position minus a shift drawn in [-8192, 8192],
    clipped so the old position stays >= 0.  All requests share one destination pool.
    """
    b = 16
    rng = _rng(5, 0, 0, _LAYOUT, seed)
    n_req = 8
    raw = rng.uniform(16384, 131072, size=n_req)
    units = np.clip(np.round(raw * (400000 / raw.sum()) / 16), 1024, 8192).astype(np.int64)
    units = _fix_sum(units, 400000 // 16, 1024, 8192, rng)
    n_dst = int(units.sum())
    dst_perm = rng.permutation(n_dst).astype(np.int32)
    per_req = []
    n_src = 0
    for r in range(n_req):
        U = int(units[r])
        frac = rng.uniform(0.70, 0.95)
        cu = int(round(frac * U))
        nu = U - cu
        n_c = int(rng.integers(8, 65))
        n_u = int(rng.integers(2, 9))
        cu_parts = _dirichlet_units(rng, cu, n_c)
        nu_parts = _dirichlet_units(rng, nu, n_u)
        kinds = [("c", i) for i in range(n_c)] + [("u", i) for i in range(n_u)]
        order = [kinds[i] for i in rng.permutation(len(kinds))]
        want_last = "c" if r % 2 == 1 else "u"
        if order[-1][0] != want_last:
            j = max(i for i, k in enumerate(order[:-1]) if k[0] == want_last)
            order[-1], order[j] = order[j], order[-1]
        per_req.append((order, cu_parts, nu_parts))
        n_src += int(cu_parts.sum())
    src = _SrcAllocator(rng.permutation(n_src).astype(np.int32))
    reqs = []
    blk = 0
    for r, (order, cu_parts, nu_parts) in enumerate(per_req):
        specs = []
        t = 0
        for kind, i in order:
            if kind == "c":
                L = int(cu_parts[i]) * 16
                shift = int(rng.integers(-8192, 8193))
                old = max(0, t - shift)
                specs.append((L, True, old, None))
            else:
                L = int(nu_parts[i]) * 16
                specs.append((L, False, 0, None))
            t += L
        nb = int(units[r])
        reqs.append(_assemble(specs, b, dst_perm[blk:blk + nb], src, None))
        blk += nb
    assert sum(r.n_tokens for r in reqs) == 400000
    return Workload("c5", 32, 8, 128, b, "bf16", 5e5, "neox", (0.15,), 32, 4, reqs, n_dst, n_src,
                    description="batch of 8 requests (~400k tokens) bf16, 32-layer hybrid stack, r=15%",
                    config_id=5)


_BUILDERS = {1: _c1, 2: _c2, 3: _c3, 4: _c4, 5: _c5}


def config_names():
    return ["c1", "c2", "c3", "c4", "c5"]


def config(i: int, seed: int = 0) -> Workload:
    """Named workload c<i> (i in 1..5)."""
    return _BUILDERS[int(i)](seed)


# --------------------------------------------------------------------------------------
# Small custom layouts for tests
# --------------------------------------------------------------------------------------

def custom_workload(seg_lists, *, n_q_heads=4, n_kv_heads=2, head_dim=64, dtype="f32",
                    rope_base=1e4, rope_style="neox", block_size=16, seed=0, plant_per_segment=0,
                    shuffle_blocks=True, name="custom") -> Workload:
    """Workload from explicit per-request segment specs [(length, cached, old_pos, new_pos|None)]."""
    rng = _rng(99, 0, 0, _LAYOUT, seed)
    b = block_size
    nblks = [-(-sum(s[0] for s in specs) // b) for specs in seg_lists]
    n_dst = int(sum(nblks)) + 3           # a few spare blocks that nothing may touch
    dst = rng.permutation(n_dst).astype(np.int32) if shuffle_blocks else np.arange(n_dst, dtype=np.int32)
    n_src = int(sum(-(-s[0] // b) for specs in seg_lists for s in specs if s[1])) + 2
    src = _SrcAllocator(rng.permutation(n_src).astype(np.int32) if shuffle_blocks
                        else np.arange(n_src, dtype=np.int32))
    reqs = []
    off = 0
    for specs, nb in zip(seg_lists, nblks):
        starts = np.cumsum([0] + [s[0] for s in specs[:-1]])
        planted = _planted_positions(rng, [(int(st), s[0], s[1]) for st, s in zip(starts, specs)],
                                     per_segment=plant_per_segment) if plant_per_segment else None
        reqs.append(_assemble(specs, b, dst[off:off + nb], src, planted))
        off += nb
    return Workload(name, n_q_heads, n_kv_heads, head_dim, b, dtype, rope_base, rope_style, (0.15,),
                    1, 0, reqs, n_dst, n_src, config_id=99)


def random_request_specs(rng: np.random.Generator, T: int, max_seg: int = 96, p_cached: float = 0.6,
                         max_pos: int = 4096):
    """Ragged random segment specs covering exactly T tokens (lengths need not be multiples of 16)."""
    specs = []
    t = 0
    while t < T:
        L = int(min(T - t, rng.integers(1, max_seg + 1)))
        cached = bool(rng.random() < p_cached)
        old = int(rng.integers(0, max_pos)) if cached else 0
        new = t + int(rng.integers(0, 64))
        specs.append((L, cached, old, new))
        t += L
    return specs


def random_request(rng, T, **kw):
    return random_request_specs(rng, T, **kw)


# --------------------------------------------------------------------------------------
# Tensors
# --------------------------------------------------------------------------------------

def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), returned as float32."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).to(torch.float32).numpy()


def _plant_rows(w: Workload):
    """(pool block, slot) of every planted cached key."""
    b = w.block_size
    blks, slots = [], []
    for r in w.requests:
        for t in r.planted:
            seg = next(s for s in r.segments if s.seq_start <= t < s.seq_start + s.length)
            j = int(t) - seg.seq_start
            blks.append(int(r.src_block_ids[seg.src_block_start + j // b]))
            slots.append(j % b)
    return np.asarray(blks, dtype=np.int64), np.asarray(slots, dtype=np.int64)


def layer_tensors(w: Workload, layer: int = 0, seed: int = 0) -> dict:
    """Host tensors of one layer (float32, bf16-exact for bf16 workloads).

    q [sum T][Hq][d], k/v [sum T][Hkv][d]: fresh post-RoPE rows of every token.
    k_src/v_src [n_src_blocks][Hkv][b][d]: source pool holding the cached segments at their old
    positions; planted rows are scaled by plant_scale.
    """
    Ttot = w.total_tokens
    Hq, Hkv, d, b = w.n_q_heads, w.n_kv_heads, w.head_dim, w.block_size
    cid = w.config_id

    def draw(tid, shape):
        return _rng(cid, layer, 0, tid, seed).standard_normal(size=shape, dtype=np.float32)

    out = {
        "q": draw(_Q, (Ttot, Hq, d)),
        "k": draw(_K, (Ttot, Hkv, d)),
        "v": draw(_V, (Ttot, Hkv, d)),
        "k_src": draw(_KSRC, (w.n_src_blocks, Hkv, b, d)),
        "v_src": draw(_VSRC, (w.n_src_blocks, Hkv, b, d)),
    }
    pb, ps = _plant_rows(w)
    if len(pb):
        out["k_src"][pb, :, ps, :] *= np.float32(w.plant_scale)
    if w.dtype == "bf16":
        out = {k: round_bf16(v) for k, v in out.items()}
    return out


def request_tensors(w: Workload, layer: int, r: int, seed: int = 0) -> dict:
    """Host tensors of request r of one layer, drawn from the request's own streams (keyed by
    (config, layer, 1 + r, tensor id, seed)), so that one request of a large batch can be checked on
    the CPU without drawing the whole batch there.

    q [T_r][Hq][d], k/v [T_r][Hkv][d]: the request's fresh rows.  src_blocks: the sorted source-pool
    block ids its cached segments read; k_src/v_src [len(src_blocks)][Hkv][b][d] their contents
    (planted rows of the request scaled by plant_scale).  Same distributions as layer_tensors;
    float32, bf16-exact for bf16 workloads.  A device batch drawn by layer_tensors_torch takes
    these values by overwriting the request's rows and blocks."""
    req = w.requests[r]
    T = req.n_tokens
    Hq, Hkv, d, b = w.n_q_heads, w.n_kv_heads, w.head_dim, w.block_size
    cid = w.config_id

    def draw(tid, shape):
        return _rng(cid, layer, 1 + r, tid, seed).standard_normal(size=shape, dtype=np.float32)

    blocks = np.unique(np.asarray(req.src_block_ids, dtype=np.int64))
    out = {
        "q": draw(_Q, (T, Hq, d)),
        "k": draw(_K, (T, Hkv, d)),
        "v": draw(_V, (T, Hkv, d)),
        "k_src": draw(_KSRC, (len(blocks), Hkv, b, d)),
        "v_src": draw(_VSRC, (len(blocks), Hkv, b, d)),
    }
    where = {int(x): i for i, x in enumerate(blocks)}
    for t in np.asarray(req.planted, dtype=np.int64):
        seg = next(s for s in req.segments if s.seq_start <= t < s.seq_start + s.length)
        j = int(t) - seg.seq_start
        out["k_src"][where[int(req.src_block_ids[seg.src_block_start + j // b])], :, j % b, :] *= np.float32(w.plant_scale)
    if w.dtype == "bf16":
        out = {k: round_bf16(v) for k, v in out.items()}
    out["src_blocks"] = blocks
    return out


def request_pools(w: Workload, r: int, rt: dict) -> tuple:
    """Full-size source pools [n_src_blocks][Hkv][b][d] (zeros) holding request r's source blocks
    from request_tensors, for the oracle's re-alignment of that request."""
    shape = (w.n_src_blocks, w.n_kv_heads, w.block_size, w.head_dim)
    ks = np.zeros(shape, np.float32)
    vs = np.zeros(shape, np.float32)
    ks[rt["src_blocks"]] = rt["k_src"]
    vs[rt["src_blocks"]] = rt["v_src"]
    return ks, vs


def layer_tensors_torch(w: Workload, layer: int = 0, seed: int = 0, device="cuda", which=None) -> dict:
    """Device tensors of one layer, drawn with torch's generator (for sizes too big to draw on
    the host).  Same distributions and planting as layer_tensors, different random stream.
    Returned in the workload's storage dtype."""
    import torch
    Ttot = w.total_tokens
    Hq, Hkv, d, b = w.n_q_heads, w.n_kv_heads, w.head_dim, w.block_size
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    shapes = {
        "q": (_Q, (Ttot, Hq, d)), "k": (_K, (Ttot, Hkv, d)), "v": (_V, (Ttot, Hkv, d)),
        "k_src": (_KSRC, (w.n_src_blocks, Hkv, b, d)), "v_src": (_VSRC, (w.n_src_blocks, Hkv, b, d)),
    }
    out = {}
    for name, (tid, shape) in shapes.items():
        if which is not None and name not in which:
            continue
        g = torch.Generator(device=device)
        g.manual_seed(int(np.random.SeedSequence([w.config_id, layer, 0, tid, seed]).generate_state(1)[0]))
        x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
        if name == "k_src":
            pb, ps = _plant_rows(w)
            if len(pb):
                pbt = torch.as_tensor(pb, device=device)
                pst = torch.as_tensor(ps, device=device)
                x[pbt, :, pst, :] *= w.plant_scale
        out[name] = x.to(dt)
    return out
