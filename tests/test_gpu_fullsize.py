"""Parity at the full sizes of the named workloads, in the launch configuration the benchmark uses.

* c3 (32768 tokens, 32/8/128): the boundary full layer (its attention also yields the softmax
  denominators that the one-pass scoring uses), the selection on it and the first sparse layer.  Scores and recompute sets are compared with the oracle's (stored by
  tests/golden/make_golden.py from the same seeded inputs); attention on sampled rows (every
  output row depends only on its own query row and the cache, so each sampled row is an exact
  check).
* c4 (65536 tokens, 28/4/128): the selecting layer at every recompute ratio of the workload.
* c5 (8 requests, 400000 tokens, one shared pool) in both modes it runs: the selecting layer
  (two-pass scoring on mixed keys) and the hybrid stack (the boundary full layer through cu_seqlens
  with its log-sum-exp output, one-pass scoring, byte mask of R, one-pass re-alignment + KV write
  and sparse attention of the next layer).  The batch is drawn on the device; requests 4 (ends
  uncached) and 7 (ends cached: the tail fallback probes) take host-drawn inputs whose oracle scores
  and recompute sets tests/golden/make_golden.py stored.  Every request is also checked by
  properties that hold at any size (every softmax row sums to one, so sum_j s_j = Hq |P|; zero
  scores after the last probe), the selection exactly on the GPU's own scores, caches bit-exact and
  attention on sampled rows (the first and last rows of the longest request included).
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

    # the next two sparse layers as the stack runs them: the byte mask of R built once, then per layer
    # the one-pass re-alignment + KV write of R and the sparse attention of R (own inputs and caches)
    mask = torch.zeros(T, dtype=torch.uint8, device="cuda")
    sx.rows_mask(plan, rows, n_rows, max_rows, mask)
    for _ in range(2):
        layer += 1
        log(f"[c3] generating layer {layer}")
        t = W.layer_tensors(w, layer)
        q, k, v, ks, vs = (dev(t[n], w) for n in ("q", "k", "v", "k_src", "v_src"))
        kc, vc = _pool(w, dt), _pool(w, dt)
        out = torch.zeros_like(q)
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
        log(f"[c3] layer {layer}: sparse attention max-abs on {len(sample)} rows of R {err:.3g}")
        assert err <= 2e-2
        del q, k, v, ks, vs, kc, vc, out, t
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


C5_REQUESTS = (4, 7)   # the requests tests/golden/make_golden.py stores (c5_requests.npz)


def _c5_layer(w, layer):
    """Device tensors of one c5 layer: drawn on the device, with the host-drawn inputs of the stored
    requests written over their rows and source blocks."""
    log(f"[c5] drawing layer {layer}")
    t = W.layer_tensors_torch(w, layer)
    offs = w.token_offsets
    for r in C5_REQUESTS:
        rt = W.request_tensors(w, layer, r)
        for n in ("q", "k", "v"):
            t[n][offs[r]:offs[r + 1]] = torch.from_numpy(rt[n]).to("cuda").to(torch.bfloat16)
        blocks = torch.from_numpy(rt["src_blocks"]).to("cuda")
        t["k_src"][blocks] = torch.from_numpy(rt["k_src"]).to("cuda").to(torch.bfloat16)
        t["v_src"][blocks] = torch.from_numpy(rt["v_src"]).to("cuda").to(torch.bfloat16)
    return t


def _c5_golden(w):
    g = np.load(os.path.join(GOLDEN, "c5_requests.npz"))
    assert str(g["layout"]) == _layout_hash(w), "golden file does not match the workload layout"
    return g


def _c5_scores_and_sets(w, gs, Rs, g, mode, ratio):
    """Per request: score properties, selection exact on the GPU's scores; for the stored requests,
    scores and R against the oracle's."""
    offs = w.token_offsets
    for r, req in enumerate(w.requests):
        T = req.n_tokens
        s = gs[offs[r]:offs[r + 1]]
        P = O.probe_positions(T, req.segments)
        assert np.all(s >= 0) and np.all(s[P.max() + 1:] == 0)
        rel = abs(s.sum() - w.n_q_heads * len(P)) / (w.n_q_heads * len(P))
        assert rel < 1e-5, rel
        np.testing.assert_array_equal(Rs[r], O.recompute_set(T, req.segments, s, ratio, w.block_size)["R"])
    for r in C5_REQUESTS:
        req = w.requests[r]
        so = g[f"{mode}_{r}_scores"].astype(np.float64)
        _check_scores(gs[offs[r]:offs[r + 1]], so, f"c5 {mode} request {r}")
        ok, nd, detail = tie_band_ok(Rs[r], g[f"{mode}_{r}_R"].astype(np.int64), so, req.cached_mask(),
                                     int(g[f"{mode}_{r}_k"]))
        log(f"[c5 {mode}] request {r}: |R| gpu {len(Rs[r])} oracle {len(g[f'{mode}_{r}_R'])}, differing {nd}")
        assert ok, detail


def _attention_sample(w, rng, t, out, rows_of, kp=None, vp=None, n_rand=6):
    """Max-abs error of sampled attention rows against the oracle.  rows_of[r]: the request's row list
    (token indices; out holds row n of request r at off_r + n).  Keys and values: the oracle pools
    (kp, vp) when given, else the fresh tensors.  The first and last rows of the longest request are
    always in the sample."""
    offs = w.token_offsets
    scale = O.softmax_scale(w.head_dim)
    longest = int(np.argmax([r.n_tokens for r in w.requests]))
    worst = 0.0
    for r, req in enumerate(w.requests):
        T = req.n_tokens
        R = rows_of[r]
        pick = rng.choice(len(R), size=min(n_rand, len(R)), replace=False)
        if r == longest:
            pick = np.concatenate([pick, [0, len(R) - 1]])
        pick = np.unique(pick)
        toks = R[pick]
        o0 = int(offs[r])
        q = np.zeros((T, w.n_q_heads, w.head_dim), np.float32)
        q[toks] = host(t["q"][o0 + torch.from_numpy(toks).to("cuda")])
        if kp is None:
            k, v = host(t["k"][o0:o0 + T]), host(t["v"][o0:o0 + T])
        else:
            k, v = O.gather_tokens(req, w, kp), O.gather_tokens(req, w, vp)
        ref = O.attention_rows(q, k, v, toks, scale)
        got = host(out[o0 + torch.from_numpy(pick).to("cuda")])
        worst = max(worst, float(np.abs(got - ref).max()))
    return worst


@pytest.mark.timeout(900)
def test_c5_batch_selecting_layer():
    """The selecting layer on the whole batch (two-pass scoring over mixed keys)."""
    w = W.config(5)
    g = _c5_golden(w)
    layer = 4
    ratio = 0.15
    dt = torch.bfloat16
    t = _c5_layer(w, layer)
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
    log("[c5 mixed] checking")
    gs = host(scores).astype(np.float64)
    Rs = rows_per_request(w, rows, n_rows)
    _c5_scores_and_sets(w, gs, Rs, g, "mixed", ratio)
    offs = w.token_offsets
    h = {n: host(t[n]) for n in ("k", "v", "k_src", "v_src")}
    kp = np.zeros((w.n_dst_blocks, w.n_kv_heads, w.block_size, w.head_dim), np.float32)
    vp = np.zeros_like(kp)
    for r, req in enumerate(w.requests):
        O.realign_request(req, w, h["k_src"], h["v_src"], kp, vp)
        sl = slice(offs[r], offs[r + 1])
        O.scatter_rows(req, w, O.nonreuse_positions(req.n_tokens, req.segments), h["k"][sl], h["v"][sl], kp, vp)
        O.scatter_rows(req, w, Rs[r], h["k"][sl], h["v"][sl], kp, vp)
    assert np.array_equal(host(kc), kp) and np.array_equal(host(vc), vp)
    del h
    worst = _attention_sample(w, np.random.default_rng(5), t, out, Rs, kp, vp)
    log(f"[c5 mixed] {len(w.requests)} requests, |R| total {sum(len(x) for x in Rs)}, sparse attention max-abs "
        f"{worst:.3g}")
    assert worst <= 2e-2
    plan.close()


@pytest.mark.timeout(900)
def test_c5_batch_hybrid_stack():
    """The hybrid stack on the whole batch: the boundary full layer (every row's KV write, full attention
    of the 8 requests through cu_seqlens with the log-sum-exp output), the one-pass selection on its
    fresh keys, then the next (sparse) layer from the byte mask of R.  Scores and attention are also run
    twice and compared bit for bit (determinism at full size)."""
    w = W.config(5)
    g = _c5_golden(w)
    ratio = 0.15
    dt = torch.bfloat16
    plan = sx.Plan(desc_of(w), w.requests, w.n_dst_blocks, w.n_src_blocks)
    tot = w.total_tokens
    offs = w.token_offsets
    k_total, max_rows = plan.budget(ratio)
    rng = np.random.default_rng(6)

    t = _c5_layer(w, 3)
    kc, vc = _pool(w, dt), _pool(w, dt)
    out = torch.zeros_like(t["q"])
    lse = torch.zeros((tot, w.n_q_heads), dtype=torch.float32, device="cuda")
    cu = torch.from_numpy(offs.astype(np.int32)).to("cuda")
    max_T = max(r.n_tokens for r in w.requests)
    scores = torch.zeros(tot, dtype=torch.float32, device="cuda")
    scores2 = torch.zeros_like(scores)
    rows = torch.zeros(tot, dtype=torch.int32, device="cuda")
    n_rows = torch.zeros(len(w.requests), dtype=torch.int32, device="cuda")
    mask = torch.full((tot,), 0x55, dtype=torch.uint8, device="cuda")
    sx.kv_scatter(plan, t["k"], t["v"], kc, vc)
    sx.full_attn(desc_of(w), t["q"], t["k"], t["v"], cu, len(w.requests), max_T, out, lse)
    sx.sparseq_score(plan, t["q"], kc, scores, lse_in=lse)
    sx.sparseq_score(plan, t["q"], kc, scores2, lse_in=lse)
    sx.topk_select(plan, scores, ratio, rows, n_rows)
    sx.rows_mask(plan, rows, n_rows, max_rows, mask)
    torch.cuda.synchronize()
    log("[c5 stack] checking the boundary layer")
    assert torch.equal(scores, scores2), "scores differ between two runs"
    gs = host(scores).astype(np.float64)
    Rs = rows_per_request(w, rows, n_rows)
    _c5_scores_and_sets(w, gs, Rs, g, "fresh", ratio)
    want_mask = np.zeros(tot, np.uint8)
    for r in range(len(w.requests)):
        want_mask[offs[r] + Rs[r]] = 1
    assert np.array_equal(mask.cpu().numpy(), want_mask)
    hk, hv = host(t["k"]), host(t["v"])
    kp = np.zeros((w.n_dst_blocks, w.n_kv_heads, w.block_size, w.head_dim), np.float32)
    vp = np.zeros_like(kp)
    for r, req in enumerate(w.requests):
        sl = slice(offs[r], offs[r + 1])
        O.scatter_rows(req, w, np.arange(req.n_tokens), hk[sl], hv[sl], kp, vp)
    assert np.array_equal(host(kc), kp) and np.array_equal(host(vc), vp)
    del hk, hv, kp, vp
    every = [np.arange(r.n_tokens) for r in w.requests]
    worst = _attention_sample(w, rng, t, out, every)
    log(f"[c5 stack] full attention of {len(w.requests)} requests, max-abs on sampled rows {worst:.3g}")
    assert worst <= 2e-2
    del t, out, lse, kc, vc

    t = _c5_layer(w, 4)
    kc = torch.full((w.n_dst_blocks, w.n_kv_heads, w.block_size, w.head_dim), -7.0, dtype=dt, device="cuda")
    vc = torch.full_like(kc, -7.0)
    out = torch.zeros_like(t["q"])
    out2 = torch.zeros_like(t["q"])
    sx.realign_scatter_masked(plan, t["k_src"], t["v_src"], t["k"], t["v"], mask, kc, vc)
    sx.sparse_attn(plan, t["q"], rows, n_rows, max_rows, kc, vc, out)
    sx.sparse_attn(plan, t["q"], rows, n_rows, max_rows, kc, vc, out2)
    torch.cuda.synchronize()
    log("[c5 stack] checking the first sparse layer")
    assert torch.equal(out, out2), "sparse attention differs between two runs"
    del out2
    h = {n: host(t[n]) for n in ("k", "v", "k_src", "v_src")}
    kp = np.full((w.n_dst_blocks, w.n_kv_heads, w.block_size, w.head_dim), -7.0, np.float32)
    vp = kp.copy()
    for r, req in enumerate(w.requests):
        O.realign_request(req, w, h["k_src"], h["v_src"], kp, vp)
        sl = slice(offs[r], offs[r + 1])
        O.scatter_rows(req, w, Rs[r], h["k"][sl], h["v"][sl], kp, vp)
    assert np.array_equal(host(kc), kp) and np.array_equal(host(vc), vp)
    del h
    worst = _attention_sample(w, rng, t, out, Rs, kp, vp)
    log(f"[c5 stack] sparse attention, |R| total {sum(len(x) for x in Rs)}, max-abs on sampled rows {worst:.3g}")
    assert worst <= 2e-2
    plan.close()
