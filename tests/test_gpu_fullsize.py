"""Parity at the full sizes of the named workloads, in the launch configuration the benchmark uses.

* c3 (32768 tokens, 32/8/128): the boundary full layer (its attention also yields the softmax
  denominators that the one-pass scoring uses), the selection on it and the first sparse layer.  Scores and recompute sets are compared with the oracle's (stored by
  tests/golden/make_golden.py from the same seeded inputs); attention on sampled rows (every
  output row depends only on its own query row and the cache, so each sampled row is an exact
  check).
* c4 (65536 tokens, 28/4/128): the selecting layer at every recompute ratio of the workload.
* c5 (8 requests, 400000 tokens): properties that hold at any size (every softmax row sums to one,
  so per request sum_j s_j = Hq |P|; zero scores after the last probe), the selection exact on the
  GPU's own scores, re-aligned cache and KV write bit-exact, attention exact on sampled rows.
"""
import os

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from sxgpu import desc_of, dev, host, log, rows_per_request, tie_band_ok

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

try:
    import paper_2606_01751_amd as sx
except Exception:  # pragma: no cover
    sx = None


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    sx.lib()


def _layout_hash(w):
    import importlib.util
    spec = importlib.util.spec_from_file_location("make_golden", os.path.join(GOLDEN, "make_golden.py"))
    m = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(m)
    return m.layout_hash(w)


def _pool(w, dt):
    return torch.zeros((w.n_dst_blocks, w.n_kv_heads, w.block_size, w.head_dim), dtype=dt, device="cuda")


def _check_scores(gs, s_o, label):
    big = s_o >= 1e-3 * s_o.max()
    rel = (np.abs(gs - s_o)[big] / s_o[big]).max()
    log(f"[{label}] score rel err max {rel:.3g}")
    assert np.all(gs[s_o == 0] == 0)
    assert rel < 1e-4


def test_c3_boundary_selection_and_layers():
    w = W.config(3)
    g = np.load(os.path.join(GOLDEN, "c3_boundary.npz"))
    assert str(g["layout"]) == _layout_hash(w), "golden file does not match the workload layout"
    req = w.requests[0]
    T = req.n_tokens
    ratio = 0.15
    dt = torch.bfloat16
    plan = sx.Plan(desc_of(w), w.requests, w.n_dst_blocks, w.n_src_blocks)
    k_total, max_rows = plan.budget(ratio)
    scale = O.softmax_scale(w.head_dim)
    rng = np.random.default_rng(3)

    # boundary full layer: KV write of every row + full attention, then the selection on it
    layer = int(g["layer"])
    log(f"[c3] generating layer {layer}")
    t = W.layer_tensors(w, layer)
    q, k, v = dev(t["q"], w), dev(t["k"], w), dev(t["v"], w)
    kc, vc = _pool(w, dt), _pool(w, dt)
    out = torch.zeros_like(q)
    cu = torch.tensor([0, T], dtype=torch.int32, device="cuda")
    scores = torch.zeros(T, dtype=torch.float32, device="cuda")
    rows = torch.zeros(T, dtype=torch.int32, device="cuda")
    n_rows = torch.zeros(1, dtype=torch.int32, device="cuda")
    lse = torch.zeros((T, w.n_q_heads), dtype=torch.float32, device="cuda")
    sx.kv_scatter(plan, k, v, kc, vc)
    sx.full_attn(desc_of(w), q, k, v, cu, 1, T, out, lse)
    sx.sparseq_score(plan, q, kc, scores, lse_in=lse)     # one pass: the boundary layer's denominators
    sx.topk_select(plan, scores, ratio, rows, n_rows)
    torch.cuda.synchronize()
    gs = host(scores).astype(np.float64)
    _check_scores(gs, g["scores"], "c3")
    R = rows_per_request(w, rows, n_rows)[0]
    np.testing.assert_array_equal(R, O.recompute_set(T, req.segments, gs, ratio, w.block_size)["R"])
    ok, nd, detail = tie_band_ok(R, g["R"], g["scores"], req.cached_mask(), int(g["k"]))
    log(f"[c3] |R| gpu {len(R)} oracle {len(g['R'])}, differing {nd}")
    assert ok, detail
    assert len(R) <= max_rows
    sample = np.unique(np.concatenate([[0, T - 1], rng.choice(T, size=126, replace=False)]))
    ref = O.attention_rows(t["q"], t["k"], t["v"], sample, scale)
    err = np.abs(host(out)[sample] - ref).max()
    log(f"[c3] full attention max-abs on {len(sample)} rows {err:.3g}")
    assert err <= 2e-2
    del q, k, v, kc, vc, out, t

    # first sparse layer as the stack runs it: one-pass re-alignment + KV write of R, sparse attention of R
    layer += 1
    log(f"[c3] generating layer {layer}")
    t = W.layer_tensors(w, layer)
    q, k, v, ks, vs = (dev(t[n], w) for n in ("q", "k", "v", "k_src", "v_src"))
    kc, vc = _pool(w, dt), _pool(w, dt)
    out = torch.zeros_like(q)
    mask = torch.zeros(T, dtype=torch.uint8, device="cuda")
    sx.rows_mask(plan, rows, n_rows, max_rows, mask)
    sx.realign_scatter_masked(plan, ks, vs, k, v, mask, kc, vc)
    sx.sparse_attn(plan, q, rows, n_rows, max_rows, kc, vc, out)
    torch.cuda.synchronize()
    kp = np.zeros((w.n_dst_blocks, w.n_kv_heads, w.block_size, w.head_dim), np.float32)
    vp = np.zeros_like(kp)
    O.realign_request(req, w, t["k_src"], t["v_src"], kp, vp)
    O.scatter_rows(req, w, R, t["k"], t["v"], kp, vp)
    assert np.array_equal(host(kc), kp) and np.array_equal(host(vc), vp)
    sample = np.unique(np.concatenate([[0, len(R) - 1], rng.choice(len(R), size=126, replace=False)]))
    ref = O.attention_rows(t["q"], O.gather_tokens(req, w, kp), O.gather_tokens(req, w, vp), R[sample], scale)
    err = np.abs(host(out)[sample] - ref).max()
    log(f"[c3] sparse attention max-abs on {len(sample)} rows of R {err:.3g}")
    assert err <= 2e-2
    plan.close()


def test_c4_selecting_layer_all_ratios():
    w = W.config(4)
    g = np.load(os.path.join(GOLDEN, "c4_layer.npz"))
    assert str(g["layout"]) == _layout_hash(w), "golden file does not match the workload layout"
    req = w.requests[0]
    T = req.n_tokens
    dt = torch.bfloat16
    scale = O.softmax_scale(w.head_dim)
    log("[c4] generating")
    t = W.layer_tensors(w, 0)
    plan = sx.Plan(desc_of(w), w.requests, w.n_dst_blocks, w.n_src_blocks)
    q, k, v, ks, vs = (dev(t[n], w) for n in ("q", "k", "v", "k_src", "v_src"))
    kc, vc = _pool(w, dt), _pool(w, dt)
    scores = torch.zeros(T, dtype=torch.float32, device="cuda")
    rows = torch.zeros(T, dtype=torch.int32, device="cuda")
    n_rows = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = torch.zeros_like(q)
    sx.rope_realign(plan, ks, vs, kc, vc)
    nr, n_nr, m_nr = plan.nonreused_rows()
    sx.kv_scatter(plan, k, v, kc, vc, rows=nr, n_rows=n_nr, max_rows=m_nr)
    sx.sparseq_score(plan, q, kc, scores)
    torch.cuda.synchronize()
    gs = host(scores).astype(np.float64)
    _check_scores(gs, g["scores"], "c4")
    kp = np.zeros((w.n_dst_blocks, w.n_kv_heads, w.block_size, w.head_dim), np.float32)
    vp = np.zeros_like(kp)
    O.realign_request(req, w, t["k_src"], t["v_src"], kp, vp)
    O.scatter_rows(req, w, O.nonreuse_positions(T, req.segments), t["k"], t["v"], kp, vp)
    assert np.array_equal(host(kc), kp) and np.array_equal(host(vc), vp)
    cand = req.cached_mask()
    for ratio in w.ratios:
        sx.topk_select(plan, scores, ratio, rows, n_rows)
        torch.cuda.synchronize()
        R = rows_per_request(w, rows, n_rows)[0]
        np.testing.assert_array_equal(R, O.recompute_set(T, req.segments, gs, ratio, w.block_size)["R"])
        Ro = g[f"R_{int(round(ratio * 100))}"]
        k_r = O.budget(int(cand.sum()), ratio)
        ok, nd, detail = tie_band_ok(R, Ro, g["scores"], cand, k_r)
        log(f"[c4] ratio {ratio}: |R| gpu {len(R)} oracle {len(Ro)}, differing {nd}")
        assert ok, detail
    # attention at the last ratio (15 %)
    max_rows = plan.budget(w.ratios[-1])[1]
    sx.kv_scatter(plan, k, v, kc, vc, rows=rows, n_rows=n_rows, max_rows=max_rows)
    sx.sparse_attn(plan, q, rows, n_rows, max_rows, kc, vc, out)
    torch.cuda.synchronize()
    O.scatter_rows(req, w, R, t["k"], t["v"], kp, vp)
    assert np.array_equal(host(kc), kp) and np.array_equal(host(vc), vp)
    rng = np.random.default_rng(4)
    sample = np.unique(np.concatenate([[0, len(R) - 1], rng.choice(len(R), size=126, replace=False)]))
    ref = O.attention_rows(t["q"], O.gather_tokens(req, w, kp), O.gather_tokens(req, w, vp), R[sample], scale)
    err = np.abs(host(out)[sample] - ref).max()
    log(f"[c4] sparse attention max-abs on {len(sample)} rows {err:.3g}")
    assert err <= 2e-2
    plan.close()


def test_c5_batch_sparse_layer_properties():
    w = W.config(5)
    layer = w.n_full_layers          # first sparse layer
    ratio = 0.15
    dt = torch.bfloat16
    scale = O.softmax_scale(w.head_dim)
    log("[c5] generating on the device")
    t = W.layer_tensors_torch(w, layer)
    plan = sx.Plan(desc_of(w), w.requests, w.n_dst_blocks, w.n_src_blocks)
    tot = w.total_tokens
    kc, vc = _pool(w, dt), _pool(w, dt)
    scores = torch.zeros(tot, dtype=torch.float32, device="cuda")
    rows = torch.zeros(tot, dtype=torch.int32, device="cuda")
    n_rows = torch.zeros(len(w.requests), dtype=torch.int32, device="cuda")
    out = torch.zeros_like(t["q"])
    k_total, max_rows = plan.budget(ratio)
    sx.rope_realign(plan, t["k_src"], t["v_src"], kc, vc)
    nr, n_nr, m_nr = plan.nonreused_rows()
    sx.kv_scatter(plan, t["k"], t["v"], kc, vc, rows=nr, n_rows=n_nr, max_rows=m_nr)
    sx.sparseq_score(plan, t["q"], kc, scores)
    sx.topk_select(plan, scores, ratio, rows, n_rows)
    sx.kv_scatter(plan, t["k"], t["v"], kc, vc, rows=rows, n_rows=n_rows, max_rows=max_rows)
    sx.sparse_attn(plan, t["q"], rows, n_rows, max_rows, kc, vc, out)
    torch.cuda.synchronize()
    log("[c5] checking")
    gs = host(scores).astype(np.float64)
    Rs = rows_per_request(w, rows, n_rows)
    offs = w.token_offsets
    h = {n: host(t[n]) for n in ("k", "v", "k_src", "v_src")}
    kp = np.zeros((w.n_dst_blocks, w.n_kv_heads, w.block_size, w.head_dim), np.float32)
    vp = np.zeros_like(kp)
    for r, req in enumerate(w.requests):
        O.realign_request(req, w, h["k_src"], h["v_src"], kp, vp)
    rng = np.random.default_rng(5)
    for r, req in enumerate(w.requests):
        T = req.n_tokens
        s = gs[offs[r]:offs[r + 1]]
        P = O.probe_positions(T, req.segments)
        assert np.all(s >= 0) and np.all(s[P.max() + 1:] == 0)
        rel = abs(s.sum() - w.n_q_heads * len(P)) / (w.n_q_heads * len(P))
        assert rel < 1e-5, rel
        np.testing.assert_array_equal(Rs[r], O.recompute_set(T, req.segments, s, ratio, w.block_size)["R"])
        sl = slice(offs[r], offs[r + 1])
        O.scatter_rows(req, w, O.nonreuse_positions(T, req.segments), h["k"][sl], h["v"][sl], kp, vp)
        O.scatter_rows(req, w, Rs[r], h["k"][sl], h["v"][sl], kp, vp)
    assert np.array_equal(host(kc), kp) and np.array_equal(host(vc), vp)
    worst = 0.0
    for r, req in enumerate(w.requests):
        R = Rs[r]
        sample = np.unique(np.concatenate([[len(R) - 1], rng.choice(len(R), size=31, replace=False)]))
        qr = host(t["q"][offs[r]:offs[r + 1]])
        ref = O.attention_rows(qr, O.gather_tokens(req, w, kp), O.gather_tokens(req, w, vp), R[sample], scale)
        got = host(out[offs[r]:offs[r] + len(R)])[sample]
        worst = max(worst, np.abs(got - ref).max())
    log(f"[c5] {len(w.requests)} requests, |R| total {sum(len(x) for x in Rs)}, sparse attention max-abs {worst:.3g}")
    assert worst <= 2e-2
    plan.close()
