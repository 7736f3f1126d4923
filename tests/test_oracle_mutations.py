"""The oracle's pins catch plausible mistakes: each case plants one mistake in the oracle (on the
CPU, by replacing one of its functions for the duration of the case) and runs the pins that
should notice it; at least one of them must fail."""
import math

import numpy as np
import pytest

import oracle as O
import test_oracle_pins as P


def _fails(checks):
    for fn, args in checks:
        try:
            fn(*args)
        except Exception:   # an assertion (or a shape error the mistake causes)
            return True
    return False


def _bad_rope_rotate_sign(k, delta, base, style="neox"):
    k = np.asarray(k, dtype=np.float32)
    d = k.shape[-1]
    phi = float(delta) * O.rope_frequencies(d, base)
    c, s = np.cos(phi).astype(np.float32), np.sin(phi).astype(np.float32)
    a, b = O.rope_pairs(d, style)
    out = np.empty_like(k)
    out[..., a] = k[..., a] * c + k[..., b] * s
    out[..., b] = k[..., b] * c - k[..., a] * s
    return out


def _bad_frequencies(head_dim, base):
    i = np.arange(head_dim // 2, dtype=np.float64)
    return np.power(float(base), -1.0 * i / head_dim)


def _bad_pairs(head_dim, style):
    h = head_dim // 2
    i = np.arange(h)
    return (2 * i, 2 * i + 1) if style == "neox" else (i, i + h)


_orig = {name: getattr(O, name) for name in ("budget", "overflow_positions", "tail_fallback", "topk_keys",
                                              "realign_request", "softmax_scale", "rmsnorm", "silu_mul",
                                              "rope_at_positions", "linear", "attention_rows", "sparse_layer")}


def _bad_budget(n, ratio):
    return min(n, int(math.floor(ratio * n)))


def _bad_overflow(n_tokens, segments, block):
    return _orig["overflow_positions"](n_tokens, segments, block // 2)


def _bad_tail(n_tokens, segments, tail=64):
    return _orig["tail_fallback"](n_tokens, segments, 32)


def _bad_topk(scores, candidates, k):
    c = np.asarray(candidates, dtype=np.int64)
    order = np.lexsort((-c, -np.asarray(scores, dtype=np.float64)[c]))   # ties: higher index first
    return np.sort(c[order[:k]])


def _bad_realign(req, w, k_src_pool, v_src_pool, k_dst_pool, v_dst_pool):
    b = w.block_size
    for seg in req.segments:
        if not seg.cached:
            continue
        delta = seg.old_pos - seg.new_pos
        sb, so = O._src_slots(req, seg, b)
        db, do = O._dst_slots(req, np.arange(seg.seq_start, seg.seq_start + seg.length), b)
        k_dst_pool[db, :, do, :] = O.store(O.rope_rotate(k_src_pool[sb, :, so, :], delta, w.rope_base,
                                                         w.rope_style), w.dtype)
        v_dst_pool[db, :, do, :] = v_src_pool[sb, :, so, :]


def _bad_scale(head_dim):
    return 1.0 / head_dim


def _bad_rmsnorm_no_gamma(x, gamma, eps):
    return _orig["rmsnorm"](x, np.ones_like(np.asarray(gamma, dtype=np.float64)), eps)


def _bad_rmsnorm_sum(x, gamma, eps):
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.sum(x * x, axis=-1, keepdims=True) + eps) * gamma


def _bad_silu(gate_up):
    gu = np.asarray(gate_up, dtype=np.float64)
    f = gu.shape[-1] // 2
    g, u = gu[..., :f], gu[..., f:]
    return g / (1.0 + np.exp(g)) * u


def _bad_rope_positions(x, positions, base, style="neox"):
    return _orig["rope_at_positions"](x, np.asarray(positions) + 1, base, style)


def _bad_linear_no_residual(x, w, residual=None):
    return _orig["linear"](x, w)


def _bad_attention_head_map(q, k, v, rows, scale, chunk=256):
    Hq, Hkv = q.shape[1], k.shape[1]
    if Hq == Hkv:
        return _orig["attention_rows"](q, k, v, rows, scale, chunk)
    # query head h reads KV head h mod Hkv instead of h / (Hq / Hkv)
    perm = np.array([h % Hkv for h in range(Hq)])
    G = Hq // Hkv
    k2 = np.repeat(k, G, axis=1)[:, [p * G for p in perm]]
    v2 = np.repeat(v, G, axis=1)[:, [p * G for p in perm]]
    return _orig["attention_rows"](q, k2, v2, rows, scale, chunk)


def _bad_sparse_layer_scores_first(w, tensors, ratio, **kw):
    # the Sparse-Q scores are taken before the fresh keys of I_nr are written, so the uncached rows
    # score against whatever their cache slots held (Algorithm 1 steps 11-12 out of order)
    kp = O._empty_pool(w)
    vp = O._empty_pool(w)
    offs = w.token_offsets
    scores = []
    for r, req in enumerate(w.requests):
        O.realign_request(req, w, tensors["k_src"], tensors["v_src"], kp, vp)
        q = tensors["q"][offs[r]:offs[r + 1]]
        scores.append(O.sparseq_scores(q, O.gather_tokens(req, w, kp), O.probe_positions(req.n_tokens, req.segments),
                                       O.softmax_scale(w.head_dim)))
    return _orig["sparse_layer"](w, tensors, ratio, scores_from=scores, **kw)


CASES = [
    ("rope sign", "rope_rotate", _bad_rope_rotate_sign,
     [(P.test_rope_closed_form_d4, ()), (P.test_rope_relative_property, ("neox",))]),
    ("rope frequency exponent", "rope_frequencies", _bad_frequencies,
     [(P.test_rope_closed_form_d4, ()), (P.test_rope_relative_property, ("neox",))]),
    ("rope pair layout", "rope_pairs", _bad_pairs,
     [(P.test_rope_closed_form_d4, ()), (P.test_rope_relative_property, ("neox",))]),
    ("budget rounding", "budget", _bad_budget, [(P.test_budget_rounding, ()), (P.test_c1_sets_match_hand_derivation, ())]),
    ("overflow width", "overflow_positions", _bad_overflow,
     [(P.test_overflow_edge_layouts, ()), (P.test_c1_sets_match_hand_derivation, ())]),
    ("tail length", "tail_fallback", _bad_tail, [(P.test_tail_fallback_layouts, ())]),
    ("tie order", "topk_keys", _bad_topk, [(P.test_topk_matches_rank_count, (0,)), (P.test_topk_matches_rank_count, (1,))]),
    ("shift direction", "realign_request", _bad_realign,
     [(P.test_realign_request_moves_keys_to_new_positions, ("f32",))]),
    ("softmax scale", "softmax_scale", _bad_scale,
     [(P.test_full_attention_matches_torch_sdpa, ()), (P.test_attention_matches_loops_on_tiny_inputs, ())]),
    ("attention head map", "attention_rows", _bad_attention_head_map,
     [(P.test_attention_matches_loops_on_tiny_inputs, ()), (P.test_ratio_one_equals_full_attention, ())]),
    ("rmsnorm without gamma", "rmsnorm", _bad_rmsnorm_no_gamma, [(P.test_rmsnorm_closed_form_and_invariants, ())]),
    ("rmsnorm sum for mean", "rmsnorm", _bad_rmsnorm_sum, [(P.test_rmsnorm_closed_form_and_invariants, ())]),
    ("silu sign", "silu_mul", _bad_silu, [(P.test_silu_mul_closed_forms, ())]),
    ("rope position off by one", "rope_at_positions", _bad_rope_positions,
     [(P.test_rope_at_positions_absolute_and_relative, ("neox",))]),
    ("missing residual", "linear", _bad_linear_no_residual,
     [(P.test_linear_matches_loops_and_identity, ())]),
    ("scores before the I_nr write", "sparse_layer", _bad_sparse_layer_scores_first,
     [(P.test_selecting_layer_scores_fresh_nonreused_and_realigned_cached_keys, ())]),
]


@pytest.mark.parametrize("name,target,bad,checks", CASES, ids=[c[0] for c in CASES])
def test_planted_mistake_fails_a_pin(monkeypatch, name, target, bad, checks):
    monkeypatch.setattr(O, target, bad)
    assert _fails(checks), f"no pin notices the planted mistake: {name}"


def test_pins_pass_on_the_true_oracle():
    for _, _, _, checks in CASES:
        assert not _fails(checks)
