"""Plain CPU oracle of SparseX's per-layer Sparse-KV Recomputation step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this package: only the
tests, the smoke check and the benchmark's CPU-baseline leg use it.  It shares no code with the
HIP library (no kernels, headers, tables or helpers); the only thing both sides consume is the
seeded input generator in ``workloads``.

Everything here is a direct, slow transcription of the paper's definitions:

* RoPE re-alignment (Section 3.1): a cached key at old position n moves to n' by the
  incremental rotation R_{n'-n}; values are copied unchanged.
* Sparse-Q scoring (Section 3.2, Eq. sparseq-attn and Eq. sparseq-score): softmax attention
  of the non-reused query rows over all causally visible keys, summed per key over rows and,
  at the implementation level, over attention heads.
* Key selection (Eq. topk), overflow (Section 3.3), tail fallback (Section 3.2, last
  paragraph) and the recompute set R (Algorithm 1, step 17).
* KV write of recomputed rows (Algorithm 1, steps 19-20) and sparse causal attention of the
  rows of R over the mixed cache (Algorithm 1, step 21).
* Plain causal attention for the layers before the hybrid threshold (Section 3.4,
  Algorithm 1 steps 7-10).

Precision: scores and attention are computed in float64 from the stored input values.  The
re-aligned key is a stored value, so the decision of what gets stored is taken in the precision
the storing kernel uses: the rotation is evaluated in float32 (each product and sum rounded
once, no fused multiply-add) from float32 cos/sin of a float64 angle, then rounded to the storage
type (round-to-nearest-even for bfloat16).

Readings of points the paper leaves open (pair layout, sign, candidates of the top-k, rounding
of k, tie order, overflow width, tail trigger) are listed in the design notes; each function
states the one it uses.

Parity status: every function below is pinned by the oracle self-tests (closed forms,
invariants, brute force on tiny inputs and the hand-derived sets of the 512-token workload).
"""
from __future__ import annotations

import math
from typing import Iterable, List, Sequence

import numpy as np

__all__ = [
    "token_layout", "nonreuse_positions", "reuse_positions", "rope_frequencies", "rope_pairs",
    "rope_rotate", "to_bf16", "store", "realign_request", "scatter_rows", "gather_tokens",
    "tail_fallback", "overflow_positions", "probe_positions", "budget", "topk_keys",
    "recompute_set", "sparseq_scores", "attention_rows", "full_attention", "softmax_scale",
    "sparse_layer", "rmsnorm", "linear", "rope_at_positions", "silu_mul", "layer_body",
]


# ---------------------------------------------------------------------------------------------
# Token layout (Section 3.2: reuse / non-reuse index sets; Algorithm 1 steps 3-5)
# ---------------------------------------------------------------------------------------------

def token_layout(n_tokens: int, segments) -> tuple:
    """Per-token (cached flag, RoPE position in the new sequence, segment index).

    The segments must tile [0, n_tokens) in order.  Causal order is the sequence index; the
    position is only used by RoPE.
    """
    cached = np.zeros(n_tokens, dtype=bool)
    pos = np.zeros(n_tokens, dtype=np.int64)
    seg_of = np.full(n_tokens, -1, dtype=np.int64)
    t = 0
    for m, s in enumerate(segments):
        if s.seq_start != t or s.length <= 0:
            raise ValueError("segments must tile the sequence in order")
        for j in range(s.length):
            cached[t + j] = bool(s.cached)
            pos[t + j] = s.new_pos + j
            seg_of[t + j] = m
        t += s.length
    if t != n_tokens:
        raise ValueError("segments do not cover the sequence")
    return cached, pos, seg_of


def nonreuse_positions(n_tokens: int, segments) -> np.ndarray:
    """I_nr: token indices of uncached segments (the Sparse-Q rows)."""
    cached, _, _ = token_layout(n_tokens, segments)
    return np.flatnonzero(~cached)


def reuse_positions(n_tokens: int, segments) -> np.ndarray:
    """I_reuse: token indices of cached segments."""
    cached, _, _ = token_layout(n_tokens, segments)
    return np.flatnonzero(cached)


# ---------------------------------------------------------------------------------------------
# RoPE re-alignment (Section 3.1)
# ---------------------------------------------------------------------------------------------

def rope_frequencies(head_dim: int, base: float) -> np.ndarray:
    """theta_i = base^(-2i/d), i = 0 .. d/2-1, in float64."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    return np.power(float(base), -2.0 * i / head_dim)


def rope_pairs(head_dim: int, style: str) -> tuple:
    """Index pairs (first, second) that RoPE rotates together with frequency i.

    "neox": (i, i + d/2); "gptj": (2i, 2i + 1).  The paper only says RoPE has a two-dimensional
    block structure; which two coordinates form a block is a property of the checkpoint.
    """
    h = head_dim // 2
    i = np.arange(h)
    if style == "neox":
        return i, i + h
    if style == "gptj":
        return 2 * i, 2 * i + 1
    raise ValueError(style)


def rope_rotate(k: np.ndarray, delta: int, base: float, style: str = "neox") -> np.ndarray:
    """R_delta applied to the last axis of float32 keys, evaluated in float32.

    Each pair (x1, x2) with frequency theta_i becomes
        x1' = x1*cos(phi) - x2*sin(phi),   x2' = x2*cos(phi) + x1*sin(phi),   phi = delta*theta_i,
    the standard RoPE rotation (Section 3.1: k_{n'} = R_{n'-n} k_n).  phi and its cos/sin are
    float64, then rounded to float32; every product and sum below is one rounded float32 op.
    """
    k = np.asarray(k, dtype=np.float32)
    d = k.shape[-1]
    phi = float(delta) * rope_frequencies(d, base)
    c = np.cos(phi).astype(np.float32)
    s = np.sin(phi).astype(np.float32)
    a, b = rope_pairs(d, style)
    x1 = k[..., a]
    x2 = k[..., b]
    out = np.empty_like(k)
    out[..., a] = (x1 * c) - (x2 * s)
    out[..., b] = (x2 * c) + (x1 * s)
    return out


def to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16, ties to even; returned as float32 values."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def store(x: np.ndarray, dtype: str) -> np.ndarray:
    """Value written to a cache of the given storage type."""
    x = np.asarray(x, dtype=np.float32)
    return to_bf16(x) if dtype == "bf16" else x.copy()


def _src_slots(req, seg, b):
    j = np.arange(seg.length)
    blk = np.asarray(req.src_block_ids)[seg.src_block_start + j // b]
    return blk.astype(np.int64), (j % b).astype(np.int64)


def _dst_slots(req, tokens, b):
    tokens = np.asarray(tokens, dtype=np.int64)
    return np.asarray(req.block_table)[tokens // b].astype(np.int64), tokens % b


def realign_request(req, w, k_src_pool, v_src_pool, k_dst_pool, v_dst_pool) -> None:
    """Algorithm 1 step 6 for one layer: for every cached segment with shift
    delta = new_pos - old_pos, write R_delta K_old into the segment's destination slots and
    copy V_old unchanged.  Pools are [blocks][Hkv][b][d]; segment token j sits in source block
    src_block_ids[src_block_start + j // b], slot j % b, and goes to destination block
    block_table[t // b], slot t % b with t = seq_start + j."""
    b = w.block_size
    for seg in req.segments:
        if not seg.cached:
            continue
        delta = seg.new_pos - seg.old_pos
        sb, so = _src_slots(req, seg, b)
        db, do = _dst_slots(req, np.arange(seg.seq_start, seg.seq_start + seg.length), b)
        k_old = k_src_pool[sb, :, so, :]
        v_old = v_src_pool[sb, :, so, :]
        k_dst_pool[db, :, do, :] = store(rope_rotate(k_old, delta, w.rope_base, w.rope_style), w.dtype)
        v_dst_pool[db, :, do, :] = v_old


def scatter_rows(req, w, rows, k_new, v_new, k_pool, v_pool) -> None:
    """Algorithm 1 step 19 (KV write): fresh K/V of token t go to its destination slot.
    k_new/v_new are the request's own [T][Hkv][d] rows."""
    rows = np.asarray(rows, dtype=np.int64)
    if len(rows) == 0:
        return
    db, do = _dst_slots(req, rows, w.block_size)
    k_pool[db, :, do, :] = k_new[rows]
    v_pool[db, :, do, :] = v_new[rows]


def gather_tokens(req, w, pool) -> np.ndarray:
    """Token-order view [T][Hkv][d] of a request's destination slots."""
    db, do = _dst_slots(req, np.arange(req.n_tokens), w.block_size)
    return pool[db, :, do, :]


# ---------------------------------------------------------------------------------------------
# Probe set, overflow, tail fallback, top-k and R (Sections 3.2-3.3, Algorithm 1 steps 14-17)
# ---------------------------------------------------------------------------------------------

def tail_fallback(n_tokens: int, segments, tail: int = 64) -> np.ndarray:
    """S_tail: if the last token belongs to a cached segment, the last min(64, len) tokens of
    that segment; otherwise empty (Section 3.2, fallback paragraph; Algorithm 1 step 16)."""
    last = None
    for s in segments:
        if s.seq_start <= n_tokens - 1 < s.seq_start + s.length:
            last = s
    if last is None or not last.cached:
        return np.zeros(0, dtype=np.int64)
    lo = max(last.seq_start, n_tokens - tail)
    return np.arange(lo, n_tokens, dtype=np.int64)


def overflow_positions(n_tokens: int, segments, block: int) -> np.ndarray:
    """S_ov: for every maximal run [a, e) of non-reused tokens, the `block` positions on each
    side, [a-block, a) and [e, e+block), clipped to the sequence (Section 3.3;
    Algorithm 1 step 15)."""
    cached, _, _ = token_layout(n_tokens, segments)
    out = set()
    t = 0
    while t < n_tokens:
        if cached[t]:
            t += 1
            continue
        a = t
        while t < n_tokens and not cached[t]:
            t += 1
        e = t
        out.update(range(max(0, a - block), a))
        out.update(range(e, min(n_tokens, e + block)))
    return np.array(sorted(out), dtype=np.int64)


def probe_positions(n_tokens: int, segments) -> np.ndarray:
    """Query rows that probe the keys: I_nr plus the tail-fallback rows (the fallback makes the
    tail act as last-Q probes, Section 3.2)."""
    return np.union1d(nonreuse_positions(n_tokens, segments), tail_fallback(n_tokens, segments))


def budget(n_candidates: int, ratio: float) -> int:
    """Top-k budget from a recompute ratio: k = min(n, floor(ratio * n + 1/2)), float64."""
    if not (0.0 <= ratio <= 1.0):
        raise ValueError("ratio must lie in [0, 1]")
    return int(min(n_candidates, math.floor(float(ratio) * float(n_candidates) + 0.5)))


def topk_keys(scores: np.ndarray, candidates: np.ndarray, k: int) -> np.ndarray:
    """Eq. topk over the candidate positions: the k positions with the largest score, ties
    broken towards the lower index (total order on (-s_j, j))."""
    cand = [int(j) for j in candidates]
    cand.sort(key=lambda j: (-float(scores[j]), j))
    return np.array(sorted(cand[:k]), dtype=np.int64)


def recompute_set(n_tokens: int, segments, scores: np.ndarray, ratio: float, block: int,
                  candidates: str = "reused") -> dict:
    """Algorithm 1 step 17: R = I_nr U S_key U S_ov U S_tail, sorted.  Candidates of the top-k
    are the reused positions, with k = budget(|I_reuse|, ratio); candidates="all" takes Eq. topk
    as printed, over every position (k = budget(T, ratio))."""
    i_nr = nonreuse_positions(n_tokens, segments)
    i_reuse = reuse_positions(n_tokens, segments)
    cand = i_reuse if candidates == "reused" else np.arange(n_tokens, dtype=np.int64)
    k = budget(len(cand), ratio)
    s_key = topk_keys(scores, cand, k)
    s_ov = overflow_positions(n_tokens, segments, block)
    s_tail = tail_fallback(n_tokens, segments)
    R = np.union1d(np.union1d(i_nr, s_key), np.union1d(s_ov, s_tail)).astype(np.int64)
    return {"R": R, "S_key": s_key, "S_ov": s_ov, "S_tail": s_tail, "I_nr": i_nr, "k": k}


# ---------------------------------------------------------------------------------------------
# Sparse-Q scores (Eq. sparseq-attn and Eq. sparseq-score; cross-head sum of Section 3.2)
# ---------------------------------------------------------------------------------------------

def softmax_scale(head_dim: int) -> float:
    return 1.0 / math.sqrt(head_dim)


def _masked_softmax_rows(z: np.ndarray, rows: np.ndarray) -> np.ndarray:
    """Row-wise softmax of z [len(rows)][T] under the causal mask M[i, j] = -inf for j > i."""
    T = z.shape[1]
    mask = np.arange(T)[None, :] > rows[:, None]
    z = np.where(mask, -np.inf, z)
    m = z.max(axis=1, keepdims=True)
    e = np.exp(z - m)
    return e / e.sum(axis=1, keepdims=True)


def sparseq_scores(q: np.ndarray, k: np.ndarray, probes: np.ndarray, scale: float,
                   chunk: int = 256) -> np.ndarray:
    """s_j = sum over query heads h and probe rows i of softmax_j(q_{i,h} K^T * scale + M_causal).

    q: [T][Hq][d], k: [T][Hkv][d] (token order, the keys the layer sees).  Query head h reads key
    head h // (Hq / Hkv).  Returns float64 [T]."""
    T, Hq, d = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    probes = np.asarray(probes, dtype=np.int64)
    s = np.zeros(T, dtype=np.float64)
    kf = np.asarray(k, dtype=np.float64)
    for c0 in range(0, len(probes), chunk):
        rows = probes[c0:c0 + chunk]
        qr = np.asarray(q[rows], dtype=np.float64)
        for h in range(Hq):
            z = (qr[:, h, :] @ kf[:, h // G, :].T) * scale
            s += _masked_softmax_rows(z, rows).sum(axis=0)
    return s


# ---------------------------------------------------------------------------------------------
# Attention (Algorithm 1 step 21; full causal attention for the hybrid layers)
# ---------------------------------------------------------------------------------------------

def attention_rows(q: np.ndarray, k: np.ndarray, v: np.ndarray, rows: np.ndarray, scale: float,
                   chunk: int = 256) -> np.ndarray:
    """SparseAttn(Q[R], K[1:T], V[1:T], M_causal) in matrix form: for the listed rows,
    softmax(Q[R] K^T * scale + M_causal[R, :]) V, per query head.  Returns float64
    [len(rows)][Hq][d]."""
    T, Hq, d = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    rows = np.asarray(rows, dtype=np.int64)
    out = np.zeros((len(rows), Hq, v.shape[2]), dtype=np.float64)
    kf = np.asarray(k, dtype=np.float64)
    vf = np.asarray(v, dtype=np.float64)
    for c0 in range(0, len(rows), chunk):
        r = rows[c0:c0 + chunk]
        qr = np.asarray(q[r], dtype=np.float64)
        for h in range(Hq):
            a = _masked_softmax_rows((qr[:, h, :] @ kf[:, h // G, :].T) * scale, r)
            out[c0:c0 + len(r), h, :] = a @ vf[:, h // G, :]
    return out


def full_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float, rows=None) -> np.ndarray:
    """Plain causal attention written per row without a mask matrix: row i attends to keys
    0..i only.  An independent formulation from attention_rows.  Returns float64
    [len(rows)][Hq][d] (all T rows if rows is None)."""
    T, Hq, d = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    rows = np.arange(T) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.zeros((len(rows), Hq, v.shape[2]), dtype=np.float64)
    for n, i in enumerate(rows):
        kk = np.asarray(k[:i + 1], dtype=np.float64)
        vv = np.asarray(v[:i + 1], dtype=np.float64)
        for g in range(Hkv):
            qg = np.asarray(q[i, g * G:(g + 1) * G, :], dtype=np.float64)    # [G][d]
            z = (kk[:, g, :] @ qg.T) * scale                                  # [i+1][G]
            w = np.exp(z - z.max(axis=0))
            w /= w.sum(axis=0)
            out[n, g * G:(g + 1) * G, :] = w.T @ vv[:, g, :]
    return out


# ---------------------------------------------------------------------------------------------
# One layer, end to end
# ---------------------------------------------------------------------------------------------

def _empty_pool(w):
    return np.zeros((w.n_dst_blocks, w.n_kv_heads, w.block_size, w.head_dim), dtype=np.float32)


def sparse_layer(w, tensors: dict, ratio: float, *, scores_from=None, R_from=None,
                 attn_rows_sample=None, skip_attention=False, k_pool=None, v_pool=None) -> dict:
    """The selecting sparse layer for every request of the workload.

    1. realign cached segments into the destination pool (Section 3.1);
    2. write the fresh K/V of I_nr (the rows every layer computes);
    3. Sparse-Q scores over the mixed keys (fresh on I_nr, re-aligned cached elsewhere);
    4. R = I_nr U top-k U overflow U tail;
    5. write fresh K/V of R (Algorithm 1 step 19; rows outside R keep the re-aligned values);
    6. sparse causal attention of the rows of R over the cache (Algorithm 1 step 21).

    scores_from / R_from let a caller reuse per-request scores or sets (for layers after the
    boundary, which reuse R).  attn_rows_sample: per-request index arrays into R to evaluate
    (row sampling for very large inputs; each output row is independent of the others).
    Returns per-request lists plus the final pools.
    """
    scale = softmax_scale(w.head_dim)
    kp = _empty_pool(w) if k_pool is None else k_pool
    vp = _empty_pool(w) if v_pool is None else v_pool
    offs = w.token_offsets
    res = {"scores": [], "sets": [], "out": [], "k_realigned": None}
    for r, req in enumerate(w.requests):
        realign_request(req, w, tensors["k_src"], tensors["v_src"], kp, vp)
    res["k_realigned"] = kp.copy()
    res["v_realigned"] = vp.copy()
    for r, req in enumerate(w.requests):
        o0, o1 = offs[r], offs[r + 1]
        q, k, v = tensors["q"][o0:o1], tensors["k"][o0:o1], tensors["v"][o0:o1]
        T = req.n_tokens
        scatter_rows(req, w, nonreuse_positions(T, req.segments), k, v, kp, vp)
        if R_from is not None:
            sets = R_from[r]
            sc = None
        else:
            if scores_from is not None:
                sc = scores_from[r]
            else:
                sc = sparseq_scores(q, gather_tokens(req, w, kp), probe_positions(T, req.segments), scale)
            sets = recompute_set(T, req.segments, sc, ratio, w.block_size)
        res["scores"].append(sc)
        res["sets"].append(sets)
        scatter_rows(req, w, sets["R"], k, v, kp, vp)
        if skip_attention:
            res["out"].append(None)
            continue
        R = sets["R"]
        sel = np.arange(len(R)) if attn_rows_sample is None else np.asarray(attn_rows_sample[r])
        res["out"].append(attention_rows(q, gather_tokens(req, w, kp), gather_tokens(req, w, vp), R[sel], scale))
    res["k_pool"] = kp
    res["v_pool"] = vp
    return res


# ---------------------------------------------------------------------------------------------
# Row-sparse layer body (Algorithm 1 step 19: project Q/K/V only for the tokens of R; step 22:
# update the hidden states only on R, then the output projection, residual path, normalisation
# and feed-forward module on those rows).  The paper does not fix the block architecture; the
# reading used is the Llama-3 block of the workloads: pre-normalisation with RMSNorm, linear
# maps without bias, RoPE on the fresh queries and keys at their positions in the new sequence,
# and a SwiGLU feed-forward module.  Everything is float64 from the stored input values; where a
# result is stored (bfloat16), `store` rounds it.
# ---------------------------------------------------------------------------------------------

def rmsnorm(x: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * gamma over the last axis, float64."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gamma, dtype=np.float64)


def linear(x: np.ndarray, w: np.ndarray, residual=None) -> np.ndarray:
    """x w^T (+ residual) with w stored [out][in] (a linear layer's weight), float64."""
    y = np.asarray(x, dtype=np.float64) @ np.asarray(w, dtype=np.float64).T
    return y if residual is None else y + np.asarray(residual, dtype=np.float64)


def rope_at_positions(x: np.ndarray, positions, base: float, style: str = "neox") -> np.ndarray:
    """RoPE of fresh rows [n][H][d] at their positions: row i is rotated by R_{positions[i]}
    (the rotation of rope_rotate with shift = position, i.e. from position 0), float32."""
    x = np.asarray(x, dtype=np.float32)
    out = np.empty_like(x)
    for i, p in enumerate(np.asarray(positions, dtype=np.int64)):
        out[i] = rope_rotate(x[i], int(p), base, style)
    return out


def silu_mul(gate_up: np.ndarray) -> np.ndarray:
    """SwiGLU: silu(g) * u for rows [g (f) | u (f)], silu(g) = g / (1 + e^-g), float64."""
    gu = np.asarray(gate_up, dtype=np.float64)
    f = gu.shape[-1] // 2
    g, u = gu[..., :f], gu[..., f:]
    return g / (1.0 + np.exp(-g)) * u


def layer_body(w, hidden: np.ndarray, R: np.ndarray, weights: dict, src_k, src_v, eps: float) -> dict:
    """One sparse layer of a single request on the rows of R (Algorithm 1 steps 19-22).

    hidden: the request's [T][H] input hidden states; weights: ln1 [H], wq [Hq d][H],
    wk / wv [Hkv d][H], wo [H][Hq d], ln2 [H], wgu [2F][H], wd [H][F].  The cache of the layer
    holds the re-aligned cached K/V of reused tokens (step 20) and the freshly projected K/V of
    the rows of R (step 19).  Intermediates are stored in the workload's type (bfloat16) where
    the GPU path stores them.  Returns the new hidden states of R and the intermediates."""
    req = w.requests[0]
    T = req.n_tokens
    Hq, Hkv, d = w.n_q_heads, w.n_kv_heads, w.head_dim
    R = np.asarray(R, dtype=np.int64)
    dt = w.dtype
    x1 = store(rmsnorm(hidden[R], weights["ln1"], eps), dt)
    q = store(linear(x1, weights["wq"]), dt).reshape(len(R), Hq, d)
    k = store(linear(x1, weights["wk"]), dt).reshape(len(R), Hkv, d)
    v = store(linear(x1, weights["wv"]), dt).reshape(len(R), Hkv, d)
    _, pos, _ = token_layout(T, req.segments)
    q = store(rope_at_positions(q, pos[R], w.rope_base, w.rope_style), dt)
    k = store(rope_at_positions(k, pos[R], w.rope_base, w.rope_style), dt)
    kp, vp = _empty_pool(w), _empty_pool(w)
    realign_request(req, w, src_k, src_v, kp, vp)
    k_tok = np.zeros((T, Hkv, d), np.float32)
    v_tok = np.zeros((T, Hkv, d), np.float32)
    k_tok[R], v_tok[R] = k, v
    scatter_rows(req, w, R, k_tok, v_tok, kp, vp)
    q_tok = np.zeros((T, Hq, d), np.float32)
    q_tok[R] = q
    att = store(attention_rows(q_tok, gather_tokens(req, w, kp), gather_tokens(req, w, vp), R,
                               softmax_scale(d)), dt).reshape(len(R), Hq * d)
    h1 = store(linear(att, weights["wo"], hidden[R]), dt)
    x2 = store(rmsnorm(h1, weights["ln2"], eps), dt)
    gu = store(linear(x2, weights["wgu"]), dt)
    a = store(silu_mul(gu), dt)
    h2 = store(linear(a, weights["wd"], h1), dt)
    return {"x1": x1, "q": q, "k": k, "v": v, "att": att, "h1": h1, "x2": x2, "gu": gu, "a": a, "h2": h2,
            "k_pool": kp, "v_pool": vp}
