"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

None of these tests re-types an oracle formula: each compares the oracle with a closed form,
an invariant, an independent formulation (complex-number RoPE, per-element loops, a library
routine) or the hand-derived index sets of the 512-token workload.
"""
import cmath
import math
import os

import numpy as np
import pytest

import oracle as O
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------------------------------------
# RoPE re-alignment (Section 3.1)
# ----------------------------------------------------------------------------------------------

def _rope_complex(k, pos, base, style):
    """Absolute RoPE written as complex multiplication: pair (x1, x2) is the complex number
    x1 + i*x2, multiplied by exp(i * pos * base^(-2i/d)).  float64."""
    k = np.asarray(k, dtype=np.float64)
    d = k.shape[-1]
    out = np.empty_like(k)
    for i in range(d // 2):
        a, b = (i, i + d // 2) if style == "neox" else (2 * i, 2 * i + 1)
        theta = base ** (-2.0 * i / d)
        z = (k[..., a] + 1j * k[..., b]) * cmath.exp(1j * pos * theta)
        out[..., a] = z.real
        out[..., b] = z.imag
    return out


@pytest.mark.parametrize("style", ["neox", "gptj"])
def test_rope_zero_delta_is_identity(style):
    rng = np.random.default_rng(1)
    k = rng.standard_normal((7, 3, 64)).astype(np.float32)
    assert np.array_equal(O.rope_rotate(k, 0, 1e4, style), k)
    kb = O.to_bf16(k)
    assert np.array_equal(O.store(O.rope_rotate(kb, 0, 5e5, style), "bf16"), kb)


def test_rope_closed_form_d4():
    # d = 4, base 1e4: theta_0 = 1, theta_1 = 0.01.  NeoX pairs (0,2), (1,3); GPT-J pairs (0,1), (2,3).
    c1, s1, c2, s2 = math.cos(1.0), math.sin(1.0), math.cos(0.01), math.sin(0.01)
    e = np.eye(4, dtype=np.float32)
    got = O.rope_rotate(e, 1, 1e4, "neox").astype(np.float64)
    want = np.array([[c1, 0, s1, 0], [0, c2, 0, s2], [-s1, 0, c1, 0], [0, -s2, 0, c2]])
    np.testing.assert_allclose(got, want, atol=1e-7)
    got = O.rope_rotate(e, 1, 1e4, "gptj").astype(np.float64)
    want = np.array([[c1, s1, 0, 0], [-s1, c1, 0, 0], [0, 0, c2, s2], [0, 0, -s2, c2]])
    np.testing.assert_allclose(got, want, atol=1e-7)
    # negative shift rotates the other way
    got = O.rope_rotate(e[:1], -1, 1e4, "neox").astype(np.float64)
    np.testing.assert_allclose(got, [[c1, 0, -s1, 0]], atol=1e-7)


@pytest.mark.parametrize("style", ["neox", "gptj"])
@pytest.mark.parametrize("a,b,base", [(64, 300, 1e4), (-4000, 12345, 5e5), (131000, -70000, 1e6)])
def test_rope_composes_additively(style, a, b, base):
    rng = np.random.default_rng(2)
    k = (4 * rng.standard_normal((16, 128))).astype(np.float32)
    two = O.rope_rotate(O.rope_rotate(k, a, base, style), b, base, style)
    one = O.rope_rotate(k, a + b, base, style)
    bound = 1e-6 * np.abs(k).max()
    assert np.abs(two - one).max() <= bound
    back = O.rope_rotate(O.rope_rotate(k, a, base, style), -a, base, style)
    assert np.abs(back - k).max() <= bound


def test_rope_preserves_pair_norms():
    rng = np.random.default_rng(3)
    k = rng.standard_normal((32, 128)).astype(np.float32)
    r = O.rope_rotate(k, 777, 5e5, "neox").astype(np.float64)
    kd = k.astype(np.float64)
    n0 = kd[:, :64] ** 2 + kd[:, 64:] ** 2
    n1 = r[:, :64] ** 2 + r[:, 64:] ** 2
    np.testing.assert_allclose(n1, n0, rtol=1e-6, atol=1e-7)


@pytest.mark.parametrize("style", ["neox", "gptj"])
def test_rope_relative_property(style):
    # K written at old position p is R_p k; re-aligned to p' it must equal R_{p'} k, and
    # <R_m q, R_n k> = <q, R_{n-m} k>.
    rng = np.random.default_rng(4)
    base = 5e5
    kraw = rng.standard_normal((10, 64))
    q = rng.standard_normal((10, 64))
    p, p2 = 1234, 4321
    k_old = _rope_complex(kraw, p, base, style).astype(np.float32)
    got = O.rope_rotate(k_old, p2 - p, base, style).astype(np.float64)
    want = _rope_complex(kraw, p2, base, style)
    assert np.abs(got - want).max() < 2e-5
    m, n = 50, 20
    lhs = np.sum(_rope_complex(q, m, base, style) * _rope_complex(kraw, n, base, style), axis=-1)
    rel = O.rope_rotate(kraw.astype(np.float32), n - m, base, style).astype(np.float64)
    rhs = np.sum(q * rel, axis=-1)
    np.testing.assert_allclose(lhs, rhs, atol=2e-5)


def test_to_bf16_rounding():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, 1.0 + 2 ** -8 + 2 ** -20,
                  -2.5, 3.0e-3], dtype=np.float32)
    got = O.to_bf16(x)
    want = np.array([1.0, 1.0, 1.0 + 2 ** -6, 1.0, 1.0 + 2 ** -7, -2.5, 0.0029907227], dtype=np.float32)
    np.testing.assert_array_equal(got[:6], want[:6])
    assert abs(got[6] - 3.0e-3) <= 2 ** -8 * 3.0e-3
    import torch
    r = np.random.default_rng(5).standard_normal(10000).astype(np.float32) * 10
    ref = torch.from_numpy(r).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(O.to_bf16(r), ref)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_realign_request_moves_keys_to_new_positions(dtype):
    # Source keys are R_old k_raw; after re-alignment the destination slot of every reused token
    # must hold R_new k_raw (complex RoPE, independent), values bit-exact, other slots untouched.
    specs = [(37, True, 100, 5), (20, False, 0, 42), (50, True, 0, 62), (9, True, 7000, 112)]
    w = W.custom_workload([specs], n_q_heads=2, n_kv_heads=2, head_dim=64, dtype=dtype, rope_base=1e4)
    req = w.requests[0]
    rng = np.random.default_rng(6)
    b = w.block_size
    kraw = rng.standard_normal((req.n_tokens, 2, 64))
    v_tok = rng.standard_normal((req.n_tokens, 2, 64)).astype(np.float32)
    k_src = np.zeros((w.n_src_blocks, 2, b, 64), np.float32)
    v_src = np.zeros_like(k_src)
    _, pos, _ = O.token_layout(req.n_tokens, req.segments)
    for s in req.segments:
        if not s.cached:
            continue
        for j in range(s.length):
            blk = req.src_block_ids[s.src_block_start + j // b]
            k_src[blk, :, j % b] = _rope_complex(kraw[s.seq_start + j], s.old_pos + j, 1e4, "neox")
            v_src[blk, :, j % b] = v_tok[s.seq_start + j]
    if dtype == "bf16":
        k_src = O.to_bf16(k_src)
    kd = np.full((w.n_dst_blocks, 2, b, 64), 7.0, np.float32)
    vd = kd.copy()
    O.realign_request(req, w, k_src, v_src, kd, vd)
    tol = 2e-5 if dtype == "f32" else 0.06
    touched = set()
    for t in range(req.n_tokens):
        blk, sl = req.block_table[t // b], t % b
        seg = [s for s in req.segments if s.seq_start <= t < s.seq_start + s.length][0]
        if seg.cached:
            touched.add((blk, sl))
            want = _rope_complex(kraw[t], pos[t], 1e4, "neox")
            assert np.abs(kd[blk, :, sl] - want).max() < tol * max(1.0, np.abs(want).max())
            assert np.array_equal(vd[blk, :, sl], v_tok[t])
    for blk in range(w.n_dst_blocks):
        for sl in range(b):
            if (blk, sl) not in touched:
                assert np.all(kd[blk, :, sl] == 7.0) and np.all(vd[blk, :, sl] == 7.0)


# ----------------------------------------------------------------------------------------------
# Sparse-Q scores (Eq. sparseq-attn, Eq. sparseq-score, cross-head aggregation)
# ----------------------------------------------------------------------------------------------

def _scores_loops(q, k, probes, scale):
    T, Hq, d = q.shape
    G = Hq // k.shape[1]
    s = [0.0] * T
    for i in probes:
        for h in range(Hq):
            z = [sum(float(q[i, h, x]) * float(k[j, h // G, x]) for x in range(d)) * scale for j in range(i + 1)]
            m = max(z)
            e = [math.exp(v - m) for v in z]
            tot = sum(e)
            for j in range(i + 1):
                s[j] += e[j] / tot
    return np.array(s)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_scores_match_loops_on_tiny_inputs(seed):
    rng = np.random.default_rng(10 + seed)
    T, Hq, Hkv, d = 19, 4, 2, 8
    q = rng.standard_normal((T, Hq, d)) * 2
    k = rng.standard_normal((T, Hkv, d)) * 2
    probes = np.sort(rng.choice(T, size=6, replace=False))
    got = O.sparseq_scores(q, k, probes, 0.35)
    want = _scores_loops(q, k, probes, 0.35)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-14)


def test_scores_row_sums_and_causality():
    rng = np.random.default_rng(11)
    T, Hq, Hkv, d = 300, 8, 2, 32
    q = rng.standard_normal((T, Hq, d))
    k = rng.standard_normal((T, Hkv, d)) * 3
    probes = np.array([3, 50, 51, 52, 199, 200, 241])
    s = O.sparseq_scores(q, k, probes, 1 / math.sqrt(d), chunk=4)
    assert abs(s.sum() - Hq * len(probes)) < 1e-9
    assert np.all(s[probes.max() + 1:] == 0.0)
    assert np.all(s[: probes.max() + 1] > 0.0)


def test_scores_zero_query_closed_form():
    T, Hq, Hkv, d = 64, 6, 3, 16
    q = np.zeros((T, Hq, d))
    k = np.random.default_rng(12).standard_normal((T, Hkv, d))
    probes = np.array([0, 5, 17, 40, 63])
    s = O.sparseq_scores(q, k, probes, 0.25)
    want = np.array([Hq * sum(1.0 / (i + 1) for i in probes if i >= j) for j in range(T)])
    np.testing.assert_allclose(s, want, rtol=1e-13)


def test_scores_single_probe_is_softmax_row():
    from scipy.special import softmax
    rng = np.random.default_rng(13)
    T, d = 40, 16
    q = rng.standard_normal((T, 1, d))
    k = rng.standard_normal((T, 1, d))
    i = 29
    s = O.sparseq_scores(q, k, np.array([i]), 0.5)
    want = np.zeros(T)
    want[: i + 1] = softmax(0.5 * (k[: i + 1, 0] @ q[i, 0]))
    np.testing.assert_allclose(s, want, rtol=1e-12, atol=1e-15)


def test_scores_query_head_reads_its_group_kv_head():
    # Hq=4, Hkv=2: heads 0,1 read KV head 0 (random keys), heads 2,3 read KV head 1 (zero keys,
    # uniform attention).  A head -> KV-head mapping by h % Hkv would mix the two.
    from scipy.special import softmax
    rng = np.random.default_rng(14)
    T, d = 30, 8
    q = rng.standard_normal((T, 4, d))
    k = np.zeros((T, 2, d))
    k[:, 0] = rng.standard_normal((T, d)) * 2
    probes = np.array([9, 29])
    s = O.sparseq_scores(q, k, probes, 1.0)
    want = np.zeros(T)
    for i in probes:
        for h in (0, 1):
            want[: i + 1] += softmax(k[: i + 1, 0] @ q[i, h])
        want[: i + 1] += 2.0 / (i + 1)
    np.testing.assert_allclose(s, want, rtol=1e-12)


# ----------------------------------------------------------------------------------------------
# Selection, overflow, tail fallback, R (Eq. topk; Section 3.3; Algorithm 1 steps 14-17)
# ----------------------------------------------------------------------------------------------

def _parse_ranges(tokens):
    out = []
    for t in tokens:
        a, b = t.split("-")
        out.extend(range(int(a), int(b) + 1))
    return np.array(out, dtype=np.int64)


def test_c1_sets_match_hand_derivation():
    golden = {}
    with open(os.path.join(GOLDEN, "c1_sets.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            parts = line.split()
            golden[parts[0]] = parts[1:]
    w = W.config(1)
    req = w.requests[0]
    T = req.n_tokens
    np.testing.assert_array_equal(O.nonreuse_positions(T, req.segments), _parse_ranges(golden["I_nr"]))
    np.testing.assert_array_equal(O.overflow_positions(T, req.segments, 16), _parse_ranges(golden["S_ov"]))
    np.testing.assert_array_equal(O.tail_fallback(T, req.segments), _parse_ranges(golden["S_tail"]))
    assert O.budget(len(O.reuse_positions(T, req.segments)), 0.15) == int(golden["k"][0])


def test_budget_rounding():
    assert O.budget(320, 0.15) == 48
    assert O.budget(6144, 0.15) == 922
    assert O.budget(30, 0.05) == 2          # 1.5 rounds up
    assert O.budget(10, 0.0) == 0
    assert O.budget(10, 1.0) == 10
    assert O.budget(0, 0.5) == 0
    with pytest.raises(ValueError):
        O.budget(10, 1.5)


@pytest.mark.parametrize("seed", range(5))
def test_topk_matches_rank_count(seed):
    rng = np.random.default_rng(20 + seed)
    T = 60
    scores = rng.integers(0, 6, size=T).astype(np.float64)     # many ties
    cand = np.sort(rng.choice(T, size=35, replace=False))
    for k in (0, 1, 7, 20, 35):
        got = O.topk_keys(scores, cand, k)
        want = [j for j in cand
                if sum(1 for j2 in cand if scores[j2] > scores[j] or (scores[j2] == scores[j] and j2 < j)) < k]
        np.testing.assert_array_equal(got, np.array(want, dtype=np.int64))


def _seg(specs):
    w = W.custom_workload([specs], n_q_heads=1, n_kv_heads=1, head_dim=8)
    return w.requests[0]


@pytest.mark.parametrize("seed", range(3))
def test_recompute_set_over_all_positions(seed):
    """Eq. topk as printed (candidates = every position): S_key holds the k = floor(r T + 1/2)
    positions that a rank count over all T positions puts first; the other parts of R are those of
    the default reading, and with every position a candidate R can only grow with the ratio."""
    rng = np.random.default_rng(40 + seed)
    r = _seg([(48, True, 0, None), (16, False, 0, None), (64, True, 5, None), (32, False, 0, None)])
    T = 160
    scores = rng.integers(0, 8, size=T).astype(np.float64)
    prev = None
    for ratio in (0.0, 0.1, 0.25, 0.5, 1.0):
        got = O.recompute_set(T, r.segments, scores, ratio, 16, candidates="all")
        base = O.recompute_set(T, r.segments, scores, ratio, 16)
        k = int(np.floor(ratio * T + 0.5))
        assert got["k"] == k and len(got["S_key"]) == k
        rank = np.array([sum(1 for j2 in range(T) if scores[j2] > scores[j] or (scores[j2] == scores[j] and j2 < j))
                         for j in range(T)])
        np.testing.assert_array_equal(got["S_key"], np.flatnonzero(rank < k))
        for part in ("I_nr", "S_ov", "S_tail"):
            np.testing.assert_array_equal(got[part], base[part])
        np.testing.assert_array_equal(got["R"], np.union1d(base["I_nr"], np.union1d(got["S_key"], np.union1d(
            base["S_ov"], base["S_tail"]))))
        if prev is not None:
            assert set(prev) <= set(got["R"])
        prev = got["R"]
    assert len(prev) == T


def test_overflow_edge_layouts():
    # uncached run at the start: only a right-hand block
    r = _seg([(20, False, 0, None), (40, True, 0, None)])
    np.testing.assert_array_equal(O.overflow_positions(60, r.segments, 16), np.arange(20, 36))
    # uncached run at the end: only a left-hand block
    r = _seg([(40, True, 0, None), (20, False, 0, None)])
    np.testing.assert_array_equal(O.overflow_positions(60, r.segments, 16), np.arange(24, 40))
    # adjacent uncached segments form one run; a cached gap shorter than a block is covered
    r = _seg([(30, True, 0, None), (5, False, 0, None), (6, False, 0, None), (10, True, 0, None),
              (4, False, 0, None), (40, True, 0, None)])
    # runs [30, 41) and [51, 55): blocks [14, 30), [41, 57), [35, 51), [55, 71)
    want = sorted(set(range(14, 30)) | set(range(41, 57)) | set(range(35, 51)) | set(range(55, 71)))
    np.testing.assert_array_equal(O.overflow_positions(95, r.segments, 16), np.array(want))
    # no uncached tokens at all: no overflow
    r = _seg([(50, True, 0, None)])
    assert len(O.overflow_positions(50, r.segments, 16)) == 0


def test_tail_fallback_layouts():
    r = _seg([(30, False, 0, None), (100, True, 0, None)])
    np.testing.assert_array_equal(O.tail_fallback(130, r.segments), np.arange(66, 130))
    r = _seg([(30, False, 0, None), (40, True, 0, None)])
    np.testing.assert_array_equal(O.tail_fallback(70, r.segments), np.arange(30, 70))
    r = _seg([(30, True, 0, None), (40, False, 0, None)])
    assert len(O.tail_fallback(70, r.segments)) == 0
    # the fallback rows also probe (they act as last-Q rows)
    r = _seg([(30, False, 0, None), (100, True, 0, None)])
    np.testing.assert_array_equal(O.probe_positions(130, r.segments),
                                  np.concatenate([np.arange(30), np.arange(66, 130)]))


def test_recompute_set_extremes():
    w = W.config(1)
    req = w.requests[0]
    T = req.n_tokens
    s = np.random.default_rng(30).random(T)
    base = np.union1d(O.nonreuse_positions(T, req.segments), O.overflow_positions(T, req.segments, 16))
    np.testing.assert_array_equal(O.recompute_set(T, req.segments, s, 0.0, 16)["R"], base)
    np.testing.assert_array_equal(O.recompute_set(T, req.segments, s, 1.0, 16)["R"], np.arange(T))
    sets = O.recompute_set(T, req.segments, s, 0.15, 16)
    assert len(sets["S_key"]) == 48
    assert set(sets["S_key"]).issubset(set(O.reuse_positions(T, req.segments)))
    assert len(sets["R"]) == len(np.union1d(base, sets["S_key"]))


def test_token_layout_rejects_bad_tables():
    from workloads import Segment
    with pytest.raises(ValueError):
        O.token_layout(10, [Segment(0, 4, True, 0, 0, 0), Segment(5, 5, False, 0, 5)])
    with pytest.raises(ValueError):
        O.token_layout(10, [Segment(0, 4, True, 0, 0, 0)])


# ----------------------------------------------------------------------------------------------
# Attention (Algorithm 1 step 21 and the full layers)
# ----------------------------------------------------------------------------------------------

def test_attention_matches_loops_on_tiny_inputs():
    rng = np.random.default_rng(40)
    T, Hq, Hkv, d = 13, 4, 2, 6
    q, k, v = (rng.standard_normal((T, h, d)) for h in (Hq, Hkv, Hkv))
    rows = np.array([0, 4, 12])
    got = O.attention_rows(q, k, v, rows, 0.4)
    for n, i in enumerate(rows):
        for h in range(Hq):
            z = [0.4 * float(np.dot(q[i, h], k[j, h // 2])) for j in range(i + 1)]
            m = max(z)
            e = [math.exp(x - m) for x in z]
            want = sum(e[j] * v[j, h // 2] for j in range(i + 1)) / sum(e)
            np.testing.assert_allclose(got[n, h], want, rtol=1e-12, atol=1e-14)


def test_full_attention_matches_torch_sdpa():
    import torch
    rng = np.random.default_rng(41)
    T, Hq, Hkv, d = 70, 8, 2, 16
    q, k, v = (rng.standard_normal((T, h, d)) for h in (Hq, Hkv, Hkv))
    # the oracle's own scale against torch's default 1/sqrt(d) (pins softmax_scale too)
    got = O.full_attention(q, k, v, O.softmax_scale(d))
    tq = torch.from_numpy(q).permute(1, 0, 2)
    tk = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(Hq // Hkv, dim=0)
    tv = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(Hq // Hkv, dim=0)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True).permute(1, 0, 2).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(O.attention_rows(q, k, v, np.arange(T), 1 / math.sqrt(d)), got, rtol=1e-10, atol=1e-12)


def test_attention_zero_keys_is_prefix_mean():
    rng = np.random.default_rng(42)
    T, d = 50, 8
    q = rng.standard_normal((T, 2, d))
    k = np.zeros((T, 1, d))
    v = rng.standard_normal((T, 1, d))
    rows = np.array([0, 9, 49])
    got = O.attention_rows(q, k, v, rows, 1.0)
    for n, i in enumerate(rows):
        for h in range(2):
            np.testing.assert_allclose(got[n, h], v[: i + 1, 0].mean(axis=0), rtol=1e-12, atol=1e-14)


def test_ratio_one_equals_full_attention():
    w = W.config(1)
    t = W.layer_tensors(w, 0)
    res = O.sparse_layer(w, t, 1.0)
    R = res["sets"][0]["R"]
    np.testing.assert_array_equal(R, np.arange(512))
    full = O.full_attention(t["q"], t["k"], t["v"], O.softmax_scale(64))
    np.testing.assert_allclose(res["out"][0], full, rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("ratio", [0.0, 0.15, 0.6])
def test_zero_deviation_sparse_equals_full(ratio):
    # If the fresh K/V of reused tokens equal their re-aligned cached values, recomputation
    # changes nothing: every row of R must equal plain causal attention on the fresh tensors.
    w = W.config(1)
    t = W.layer_tensors(w, 0)
    req = w.requests[0]
    kp = np.zeros((w.n_dst_blocks, 2, 16, 64), np.float32)
    vp = np.zeros_like(kp)
    O.realign_request(req, w, t["k_src"], t["v_src"], kp, vp)
    cached = req.cached_mask()
    k_al = O.gather_tokens(req, w, kp)
    v_al = O.gather_tokens(req, w, vp)
    t = dict(t)
    t["k"] = np.where(cached[:, None, None], k_al, t["k"])
    t["v"] = np.where(cached[:, None, None], v_al, t["v"])
    res = O.sparse_layer(w, t, ratio)
    R = res["sets"][0]["R"]
    full = O.full_attention(t["q"], t["k"], t["v"], O.softmax_scale(64), rows=R)
    np.testing.assert_allclose(res["out"][0], full, rtol=1e-10, atol=1e-12)


def test_selecting_layer_scores_fresh_nonreused_and_realigned_cached_keys():
    # Section 3.2 with Algorithm 1 steps 6 and 11-12: in the selecting layer the Sparse-Q rows score
    # against the current context -- their own fresh keys on I_nr and the cached keys moved to their
    # new positions on I_reuse.  The key matrix is built here on its own: each cached token's source
    # row (read from the pool by block id) rotated by its segment's shift with complex-number RoPE,
    # each uncached token's fresh key.  Probes are the uncached tokens plus the whole final cached
    # segment (30 tokens, shorter than the 64-token fallback).  Scores: scipy's softmax per probe row
    # and head over the visible keys, summed.
    from scipy.special import softmax
    specs = [(40, True, 300, None), (24, False, 0, None), (56, True, 5, None), (17, False, 0, None),
             (30, True, 900, None)]
    base = 1e4
    w = W.custom_workload([specs], n_q_heads=4, n_kv_heads=2, head_dim=16, dtype="f32", rope_base=base, seed=8)
    t = W.layer_tensors(w, 0)
    req = w.requests[0]
    T, b, G = req.n_tokens, w.block_size, 2
    keys = np.empty((T, 2, 16))
    probes = []
    for s in req.segments:
        for j in range(s.length):
            tok = s.seq_start + j
            if s.cached:
                blk = req.src_block_ids[s.src_block_start + j // b]
                keys[tok] = _rope_complex(t["k_src"][blk, :, j % b, :], s.new_pos - s.old_pos, base, "neox")
            else:
                keys[tok] = t["k"][tok]
                probes.append(tok)
    probes += list(range(T - 30, T))
    scale = 1.0 / math.sqrt(16)
    want = np.zeros(T)
    for i in probes:
        for h in range(4):
            want[: i + 1] += softmax(keys[: i + 1, h // G, :] @ t["q"][i, h].astype(np.float64) * scale)
    got = O.sparse_layer(w, t, 0.3, skip_attention=True)["scores"][0]
    np.testing.assert_allclose(got, want, rtol=1e-5, atol=1e-12)


def test_scatter_is_exact_and_local():
    specs = [(40, True, 0, None), (25, False, 0, None), (30, True, 9, None)]
    w = W.custom_workload([specs], n_q_heads=2, n_kv_heads=1, head_dim=8)
    req = w.requests[0]
    rng = np.random.default_rng(50)
    k_new = rng.standard_normal((95, 1, 8)).astype(np.float32)
    v_new = rng.standard_normal((95, 1, 8)).astype(np.float32)
    kp = np.full((w.n_dst_blocks, 1, 16, 8), -3.0, np.float32)
    vp = kp.copy()
    rows = np.array([0, 17, 40, 64, 94])
    O.scatter_rows(req, w, rows, k_new, v_new, kp, vp)
    gk = O.gather_tokens(req, w, kp)
    gv = O.gather_tokens(req, w, vp)
    assert np.array_equal(gk[rows], k_new[rows]) and np.array_equal(gv[rows], v_new[rows])
    others = np.setdiff1d(np.arange(95), rows)
    assert np.all(gk[others] == -3.0) and np.all(gv[others] == -3.0)
    assert (kp != -3.0).sum() == len(rows) * 8


# ----------------------------------------------------------------------------------------------
# Row-sparse layer body (Algorithm 1 steps 19 and 22)
# ----------------------------------------------------------------------------------------------

def test_rmsnorm_closed_form_and_invariants():
    # [3, 4]: mean square 12.5, so the row becomes [3, 4] / sqrt(12.5)
    y = O.rmsnorm(np.array([[3.0, 4.0]]), np.array([1.0, 1.0]), 0.0)
    np.testing.assert_allclose(y, [[0.8485281374238571, 1.1313708498984762]], rtol=1e-15)
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 64))
    g = rng.standard_normal(64)
    # scale invariance without eps, mean square 1 with unit gamma, gamma multiplies elementwise
    np.testing.assert_allclose(O.rmsnorm(7.5 * x, g, 0.0), O.rmsnorm(x, g, 0.0), rtol=1e-12)
    np.testing.assert_allclose(np.mean(O.rmsnorm(x, np.ones(64), 0.0) ** 2, axis=1), 1.0, rtol=1e-12)
    np.testing.assert_allclose(O.rmsnorm(x, 2.0 * g, 0.0), 2.0 * O.rmsnorm(x, g, 0.0), rtol=1e-12)
    # eps bounds a zero row
    assert np.all(O.rmsnorm(np.zeros((1, 8)), np.ones(8), 1e-6) == 0.0)


def test_linear_matches_loops_and_identity():
    rng = np.random.default_rng(1)
    x = rng.integers(-5, 6, size=(3, 7)).astype(np.float64)
    w = rng.integers(-5, 6, size=(4, 7)).astype(np.float64)
    r = rng.integers(-5, 6, size=(3, 4)).astype(np.float64)
    loops = np.zeros((3, 4))
    for i in range(3):
        for j in range(4):
            for kk in range(7):
                loops[i, j] += x[i, kk] * w[j, kk]
    assert np.array_equal(O.linear(x, w), loops)
    assert np.array_equal(O.linear(x, w, r), loops + r)
    assert np.array_equal(O.linear(x, np.eye(7)), x)


@pytest.mark.parametrize("style", ["neox", "gptj"])
def test_rope_at_positions_absolute_and_relative(style):
    rng = np.random.default_rng(2)
    d, base = 64, 1e4
    x = rng.standard_normal((3, 2, d)).astype(np.float32)
    # position 0 is the identity; a position p matches the complex-number absolute RoPE
    assert np.array_equal(O.rope_at_positions(x, [0, 0, 0], base, style), x)
    pos = [5, 300, 4097]
    got = O.rope_at_positions(x, pos, base, style)
    for i, p in enumerate(pos):
        np.testing.assert_allclose(got[i], _rope_complex(x[i], p, base, style), atol=2e-5)
    # relative property: <R_a q, R_b k> depends on a - b only
    q = x[0, 0][None, None]
    k = x[1, 0][None, None]
    def dot(a, b):
        return float(np.dot(O.rope_at_positions(q, [a], base, style)[0, 0].astype(np.float64),
                            O.rope_at_positions(k, [b], base, style)[0, 0].astype(np.float64)))
    assert abs(dot(10, 3) - dot(1010, 1003)) < 1e-4
    assert abs(dot(10, 3) - dot(3, 10)) > 1e-3   # the rotation has a direction


def test_silu_mul_closed_forms():
    g = np.array([0.0, 1.0, 30.0, -30.0])
    y = O.silu_mul(np.concatenate([g, np.ones(4)])[None])[0]
    np.testing.assert_allclose(y[:2], [0.0, 1.0 / (1.0 + math.exp(-1.0))], rtol=1e-15)
    np.testing.assert_allclose(y[2], 30.0, rtol=1e-12)      # silu(g) -> g for large g
    assert abs(y[3]) < 1e-11                                 # -> 0 for very negative g
    u = np.array([2.0, -3.0, 0.5, 4.0])
    np.testing.assert_allclose(O.silu_mul(np.concatenate([g, u])[None])[0], y * u, rtol=1e-15)


def _dense_block(hidden, wts, w, eps):
    """The same Llama block written densely over every token, attention by the per-row causal
    formulation (independent of the row-list routing of layer_body)."""
    T = hidden.shape[0]
    Hq, Hkv, d = w.n_q_heads, w.n_kv_heads, w.head_dim
    st = lambda a: O.store(a, w.dtype)
    x1 = st(O.rmsnorm(hidden, wts["ln1"], eps))
    q = st(O.linear(x1, wts["wq"])).reshape(T, Hq, d)
    k = st(O.linear(x1, wts["wk"])).reshape(T, Hkv, d)
    v = st(O.linear(x1, wts["wv"])).reshape(T, Hkv, d)
    pos = np.arange(T)
    q = st(O.rope_at_positions(q, pos, w.rope_base, w.rope_style))
    k = st(O.rope_at_positions(k, pos, w.rope_base, w.rope_style))
    att = st(O.full_attention(q, k, v, O.softmax_scale(d))).reshape(T, Hq * d)
    h1 = st(O.linear(att, wts["wo"], hidden))
    x2 = st(O.rmsnorm(h1, wts["ln2"], eps))
    a = st(O.silu_mul(st(O.linear(x2, wts["wgu"]))))
    return st(O.linear(a, wts["wd"], h1))


def _body_weights(rng, H, Hq, Hkv, d, F):
    def m(o, i):
        return O.to_bf16((rng.standard_normal((o, i)) / math.sqrt(i)).astype(np.float32))
    return {"ln1": O.to_bf16((1 + 0.1 * rng.standard_normal(H)).astype(np.float32)), "wq": m(Hq * d, H),
            "wk": m(Hkv * d, H), "wv": m(Hkv * d, H), "wo": m(H, Hq * d),
            "ln2": O.to_bf16((1 + 0.1 * rng.standard_normal(H)).astype(np.float32)), "wgu": m(2 * F, H),
            "wd": m(H, F)}


def test_layer_body_with_every_row_equals_dense_block():
    """No cached segment and R = every token: the row-sparse body is the plain dense block."""
    specs = [[(40, False, 0, None)]]
    w = W.custom_workload(specs, n_q_heads=4, n_kv_heads=2, head_dim=16, dtype="bf16", rope_base=1e4, seed=5,
                          name="body-dense")
    T, H = 40, 64
    rng = np.random.default_rng(3)
    hidden = O.to_bf16(rng.standard_normal((T, H)).astype(np.float32))
    wts = _body_weights(rng, H, 4, 2, 16, 96)
    t = W.layer_tensors(w, 0)
    body = O.layer_body(w, hidden, np.arange(T), wts, t["k_src"], t["v_src"], 1e-5)
    dense = _dense_block(hidden, wts, w, 1e-5)
    np.testing.assert_allclose(body["h2"], dense, atol=1e-6)


def test_layer_body_rows_depend_only_on_their_own_inputs_and_the_cache():
    """A row of R is computed from its own hidden state and the cache: dropping other rows of R
    from the set changes nothing for it as long as the cache is the same (here every token is
    cached, so rows outside R read re-aligned keys either way -- except the dropped rows' own
    slots, which is why only rows before the dropped ones are compared)."""
    specs = [[(32, True, 3, None), (16, False, 0, None), (32, True, 50, None)]]
    w = W.custom_workload(specs, n_q_heads=4, n_kv_heads=2, head_dim=16, dtype="bf16", rope_base=1e4, seed=6,
                          name="body-local")
    T, H = 80, 64
    rng = np.random.default_rng(4)
    hidden = O.to_bf16(rng.standard_normal((T, H)).astype(np.float32))
    wts = _body_weights(rng, H, 4, 2, 16, 96)
    t = W.layer_tensors(w, 0)
    R = np.array([2, 7, 32, 40, 47, 60, 70])
    full = O.layer_body(w, hidden, R, wts, t["k_src"], t["v_src"], 1e-5)
    part = O.layer_body(w, hidden, R[:4], wts, t["k_src"], t["v_src"], 1e-5)
    np.testing.assert_array_equal(full["h2"][:4], part["h2"])
