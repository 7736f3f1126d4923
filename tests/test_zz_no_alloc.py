"""The allocation-free scoring entry point (sx_sparseq_score_static) against sx_sparseq_score.

Both run the same kernels in the same fixed summation order, so the scores must be bit-identical;
two calls in a row on different plans (the second smaller, so it reads what the first left in the
shared static scratch), bfloat16 and float32, plus the oracle on the small case and the size
limit."""
import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from sxgpu import GpuLayer, desc_of, host, log

pytestmark = pytest.mark.gpu

try:
    import paper_2606_01751_amd as sx
except Exception:  # pragma: no cover
    sx = None


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    sx.lib()


def _one_pass(w, t):
    g = GpuLayer(w, t)
    offs = w.token_offsets
    sx.kv_scatter(g.plan, g.t["k"], g.t["v"], g.k_cache, g.v_cache)
    cu = torch.tensor(offs, dtype=torch.int32, device="cuda")
    out = torch.zeros_like(g.t["q"])
    lse = torch.zeros((w.total_tokens, w.n_q_heads), dtype=torch.float32, device="cuda")
    sx.full_attn(desc_of(w), g.t["q"], g.t["k"], g.t["v"], cu, len(w.requests),
                 max(r.n_tokens for r in w.requests), out, lse)
    ref = torch.full((w.total_tokens,), -1.0, dtype=torch.float32, device="cuda")
    got = torch.full((w.total_tokens,), -2.0, dtype=torch.float32, device="cuda")
    sx.sparseq_score(g.plan, g.t["q"], g.k_cache, ref, lse_in=lse)
    sx.sparseq_score_static(g.plan, g.t["q"], g.k_cache, got, lse)
    torch.cuda.synchronize()
    return g, ref, got


def test_static_scratch_scores_equal_plan_scratch_scores():
    small_specs = [[(37, False, 0, None), (250, True, 900, None), (5, False, 0, None), (100, True, 3, None)],
                   [(20, True, 0, 50), (300, False, 0, 70)]]
    cases = [
        ("8192-token RAG layer (bf16, 32/8/128)", W.config(2)),
        ("two small requests (bf16, 8/1/128)", W.custom_workload(small_specs, n_q_heads=8, n_kv_heads=1,
                                                                 head_dim=128, dtype="bf16", rope_base=5e5,
                                                                 seed=7, name="small")),
        ("two small requests (f32, 8/2/64)", W.custom_workload(small_specs, n_q_heads=8, n_kv_heads=2,
                                                               head_dim=64, dtype="f32", seed=9, name="small32")),
    ]
    for label, w in cases:
        log(f"[static scratch] {label}")
        t = W.layer_tensors(w, 0)
        g, ref, got = _one_pass(w, t)
        assert torch.equal(ref, got), f"{label}: static-scratch scores differ from the plan-scratch scores"
        if w.total_tokens < 2000:
            s = host(got).astype(np.float64)
            offs = w.token_offsets
            for r, req in enumerate(w.requests):
                sl = slice(offs[r], offs[r + 1])
                s_o = O.sparseq_scores(t["q"][sl], t["k"][sl], O.probe_positions(req.n_tokens, req.segments),
                                       O.softmax_scale(w.head_dim))
                big = s_o >= 1e-3 * s_o.max()
                assert np.all(s[sl][s_o == 0] == 0)
                assert (np.abs(s[sl] - s_o)[big] / s_o[big]).max() < 1e-4
        g.plan.close()


def test_static_scratch_rejects_oversized_plans():
    # 64 query heads on one KV head and 4096 uncached tokens: the gathered probe queries alone need
    # 4160 x 64 x 128 x 2 bytes (68 MB), beyond the 32 MiB static scratch
    w = W.custom_workload([[(4096, False, 0, None)]], n_q_heads=64, n_kv_heads=1, head_dim=128, dtype="bf16",
                          seed=3, name="big")
    plan = sx.Plan(desc_of(w), w.requests, w.n_dst_blocks, w.n_src_blocks)
    q = torch.zeros((4096, 64, 128), dtype=torch.bfloat16, device="cuda")
    kc = torch.zeros((w.n_dst_blocks, 1, 16, 128), dtype=torch.bfloat16, device="cuda")
    lse = torch.zeros((4096, 64), dtype=torch.float32, device="cuda")
    scores = torch.zeros(4096, dtype=torch.float32, device="cuda")
    with pytest.raises(sx.SxError) as e:
        sx.sparseq_score_static(plan, q, kc, scores, lse)
    assert e.value.status == sx.SX_EUNSUPPORTED and "static scratch" in str(e.value)
    plan.close()
