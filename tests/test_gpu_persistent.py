"""Persistent attention grids: results do not depend on how the row tiles are shared out.

Sparse attention takes its row tiles from work queues held in the plan, full attention from
queue slots held by the library, and every launch must leave its counters at zero for the next.
These tests replay captured graphs (sparse attention keeps its plan counters under capture; full
attention switches to one workgroup per row tile), interleave eager calls of other sizes between
the replays, and run full attention on two streams at once, comparing every result with the first
eager one bit for bit (each row tile is computed by one workgroup with the same arithmetic,
whichever workgroup takes it).
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu

try:
    import paper_2606_01751_amd as sx
    from sxgpu import GpuLayer, desc_of, dev, log
except Exception:  # pragma: no cover - collected without the library
    sx = None


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    sx.lib()


def _workload():
    """Three requests (700, 257 and 1300 tokens), 8 query heads over 2 KV heads, d = 128, bf16."""
    rng = np.random.default_rng(11)
    specs = [W.random_request_specs(rng, T, max_seg=90) for T in (700, 257, 1300)]
    return W.custom_workload(specs, n_q_heads=8, n_kv_heads=2, head_dim=128, dtype="bf16", rope_base=1e4,
                             rope_style="neox", seed=11, plant_per_segment=3, name="persist")


def test_full_attention_graph_replays_and_two_streams():
    w = _workload()
    log("[persistent] full attention: eager, 3 graph replays, two streams")
    t = W.layer_tensors(w, 0)
    q, k, v = dev(t["q"], w), dev(t["k"], w), dev(t["v"], w)
    cu = torch.tensor(w.token_offsets, dtype=torch.int32, device="cuda")
    n_req, max_t = len(w.requests), max(r.n_tokens for r in w.requests)
    # the first request alone: a launch of another size between the replays
    cu1 = torch.tensor(w.token_offsets[:2], dtype=torch.int32, device="cuda")
    t1 = w.requests[0].n_tokens

    def run(out, stream=None):
        sx.full_attn(desc_of(w), q, k, v, cu, n_req, max_t, out, stream=stream)

    want = torch.zeros_like(q)
    run(want)
    torch.cuda.synchronize()
    assert torch.isfinite(want.float()).all()
    out_g = torch.zeros_like(q)
    side = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        run(out_g)
    other, first = torch.zeros_like(q), torch.zeros_like(q)
    for i in range(3):
        out_g.zero_()
        other.zero_()
        first.zero_()
        run(other)
        sx.full_attn(desc_of(w), q, k, v, cu1, 1, t1, first)
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out_g, want), f"replay {i}"
        assert torch.equal(other, want), f"eager call before replay {i}"
        assert torch.equal(first[:t1], want[:t1]), f"one-request call before replay {i}"
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    o1, o2 = torch.zeros_like(q), torch.zeros_like(q)
    torch.cuda.synchronize()
    with torch.cuda.stream(s1):
        run(o1)
    with torch.cuda.stream(s2):
        run(o2)
    torch.cuda.synchronize()
    assert torch.equal(o1, want) and torch.equal(o2, want)


def test_sparse_attention_graph_replays_and_fewer_rows():
    w = _workload()
    log("[persistent] sparse attention: eager, 3 graph replays, calls with fewer rows between them")
    g = GpuLayer(w, W.layer_tensors(w, 0))
    ratio = 0.3
    g.realign()
    g.scatter_nonreused()
    g.score()
    g.select(ratio)
    g.scatter_rows(ratio)
    m = g.plan.budget(ratio)[1]

    def run(out, n_rows, stream=None):
        sx.sparse_attn(g.plan, g.t["q"], g.rows, n_rows, m, g.k_cache, g.v_cache, out, stream=stream)

    want = torch.zeros_like(g.out)
    run(want, g.n_rows)
    torch.cuda.synchronize()
    n = g.n_rows.cpu().numpy()
    offs = w.token_offsets
    assert n.min() > 2
    half = torch.from_numpy((n // 2).astype(np.int32)).to("cuda")
    out_g = torch.zeros_like(g.out)
    side = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        run(out_g, g.n_rows)
    fewer = torch.zeros_like(g.out)
    for i in range(3):
        out_g.zero_()
        fewer.zero_()
        run(fewer, half)
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out_g, want), f"replay {i}"
        for r in range(len(w.requests)):
            a, b = offs[r], offs[r] + int(n[r] // 2)
            assert torch.equal(fewer[a:b], want[a:b]), f"request {r} with half its rows before replay {i}"
            assert not fewer[b:offs[r] + int(n[r])].any(), f"request {r}: rows past the bound written"


def test_sparse_attention_planned_tile_order():
    """sx_rows_mask plans the order in which sx_sparse_attn takes its row tiles for the same row list;
    the result must not change, also when n_rows changes at the same address after the plan was
    made (the attention then sees a different tile count and keeps the queue's own order)."""
    w = _workload()
    log("[persistent] sparse attention with the planned tile order of sx_rows_mask")
    g = GpuLayer(w, W.layer_tensors(w, 0))
    ratio = 0.3
    g.realign()
    g.scatter_nonreused()
    g.score()
    g.select(ratio)
    g.scatter_rows(ratio)
    m = g.plan.budget(ratio)[1]
    want = torch.zeros_like(g.out)
    sx.sparse_attn(g.plan, g.t["q"], g.rows, g.n_rows, m, g.k_cache, g.v_cache, want)
    mask = torch.zeros(w.total_tokens, dtype=torch.uint8, device="cuda")
    sx.rows_mask(g.plan, g.rows, g.n_rows, m, mask)
    for i in range(2):
        out = torch.zeros_like(g.out)
        sx.sparse_attn(g.plan, g.t["q"], g.rows, g.n_rows, m, g.k_cache, g.v_cache, out)
        torch.cuda.synchronize()
        assert torch.equal(out, want), f"planned order, call {i}"
    n = g.n_rows.cpu().numpy()
    g.n_rows.copy_(torch.from_numpy((n // 2).astype(np.int32)))
    out = torch.zeros_like(g.out)
    sx.sparse_attn(g.plan, g.t["q"], g.rows, g.n_rows, m, g.k_cache, g.v_cache, out)
    torch.cuda.synchronize()
    offs = w.token_offsets
    for r in range(len(w.requests)):
        a, b = offs[r], offs[r] + int(n[r] // 2)
        assert torch.equal(out[a:b], want[a:b]), f"request {r} with half its rows after the plan"
        assert not out[b:offs[r] + int(n[r])].any()


def test_many_launches_cycle_every_queue_slot():
    """70 full-attention launches (more than the 64 library queue slots, so every slot is reused)
    of three sizes in turn, and 30 sparse-attention launches on one plan with three row counts in
    turn: every result is bit-identical to the first one of its size, so each launch left its
    counters at zero."""
    w = _workload()
    log("[persistent] 70 full-attention and 30 sparse-attention launches in turn")
    t = W.layer_tensors(w, 0)
    q, k, v = dev(t["q"], w), dev(t["k"], w), dev(t["v"], w)
    offs = w.token_offsets
    n_req = len(w.requests)
    # full attention over the first 1, 2 and 3 requests
    sizes = [(torch.tensor(offs[:i + 2], dtype=torch.int32, device="cuda"), i + 1,
              max(r.n_tokens for r in w.requests[:i + 1])) for i in range(n_req)]
    want = []
    for cu, nr, mx in sizes:
        o = torch.zeros_like(q)
        sx.full_attn(desc_of(w), q, k, v, cu, nr, mx, o)
        want.append(o)
    torch.cuda.synchronize()
    outs = []
    for i in range(70):
        cu, nr, mx = sizes[i % n_req]
        o = torch.zeros_like(q)
        sx.full_attn(desc_of(w), q, k, v, cu, nr, mx, o)
        outs.append(o)
    torch.cuda.synchronize()
    for i, o in enumerate(outs):
        assert torch.equal(o, want[i % n_req]), f"full-attention launch {i}"
    g = GpuLayer(w, t)
    ratio = 0.3
    g.realign()
    g.scatter_nonreused()
    g.score()
    g.select(ratio)
    g.scatter_rows(ratio)
    m = g.plan.budget(ratio)[1]
    n = g.n_rows.cpu().numpy()
    counts = [torch.from_numpy(np.maximum(n // d, 1).astype(np.int32)).to("cuda") for d in (1, 2, 3)]
    ref = []
    for c in counts:
        o = torch.zeros_like(g.out)
        sx.sparse_attn(g.plan, g.t["q"], g.rows, c, m, g.k_cache, g.v_cache, o)
        ref.append(o)
    torch.cuda.synchronize()
    outs = []
    for i in range(30):
        o = torch.zeros_like(g.out)
        sx.sparse_attn(g.plan, g.t["q"], g.rows, counts[i % 3], m, g.k_cache, g.v_cache, o)
        outs.append(o)
    torch.cuda.synchronize()
    for i, o in enumerate(outs):
        assert torch.equal(o, ref[i % 3]), f"sparse-attention launch {i}"
