"""GPU parity of the row-sparse layer body (Algorithm 1 steps 19 and 22) against the oracle.

Each operation runs on seeded inputs through the C ABI with ragged multi-request row lists,
both row addressings (slot / token) and a canary in every row that is not listed; then a whole
sparse layer (RMSNorm, Q/K/V projections, RoPE, one-pass KV write, sparse attention, output
projection + residual, RMSNorm, SwiGLU feed-forward + residual) against oracle.layer_body.
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_01751_amd as sx
import workloads as W
from sxgpu import CANARY, desc_of, dev, host, log

pytestmark = pytest.mark.gpu
BF16_ULP = 2.0 ** -8     # bfloat16 relative spacing (8 stored mantissa bits)


def _ragged_workload(seed=11):
    rng = np.random.default_rng(seed)
    specs = [W.random_request_specs(rng, T) for T in (700, 257, 40)]
    return W.custom_workload(specs, n_q_heads=8, n_kv_heads=2, head_dim=128, dtype="bf16", rope_base=5e5,
                             seed=seed, name="layer-ragged")


def _rows(w, rng, frac):
    """A sorted random subset of every request's tokens (at least one row), row-list layout."""
    per = [np.sort(rng.choice(r.n_tokens, size=max(1, int(frac * r.n_tokens)), replace=False)) for r in w.requests]
    rows = np.zeros(w.total_tokens, np.int32)
    n = np.zeros(len(w.requests), np.int32)
    for r, R in enumerate(per):
        rows[w.token_offsets[r]:w.token_offsets[r] + len(R)] = R
        n[r] = len(R)
    return per, torch.from_numpy(rows).cuda(), torch.from_numpy(n).cuda(), int(n.max())


def _bf16(rng, shape, scale=1.0):
    return O.to_bf16((scale * rng.standard_normal(shape)).astype(np.float32))


def _index(w, per, r, by_token):
    off = w.token_offsets[r]
    return off + per[r] if by_token else off + np.arange(len(per[r]))


@pytest.mark.parametrize("x_tok,y_tok,with_res", [(False, False, False), (True, False, True), (False, True, True),
                                                  (True, True, False)])
def test_gemm_rows_matches_oracle(x_tok, y_tok, with_res):
    log(f"[gemm_rows] x_tok={x_tok} y_tok={y_tok} residual={with_res}")
    w = _ragged_workload()
    rng = np.random.default_rng(12)
    per, rows, n_rows, m = _rows(w, rng, 0.6)
    K, N, tot = 384, 512, w.total_tokens
    x = _bf16(rng, (tot, K))
    wt = _bf16(rng, (N, K), 1 / math.sqrt(K))
    res = _bf16(rng, (tot, N)) if with_res else None
    plan = sx.Plan(desc_of(w), w.requests, w.n_dst_blocks, w.n_src_blocks)
    y = torch.full((tot, N), CANARY, dtype=torch.bfloat16, device="cuda")
    sx.gemm_rows(plan, rows, n_rows, m, dev(x, w), dev(wt, w), y, residual=None if res is None else dev(res, w),
                 x_by_token=x_tok, y_by_token=y_tok)
    torch.cuda.synchronize()
    got = host(y)
    touched = np.zeros(tot, bool)
    worst = 0.0
    for r in range(len(w.requests)):
        xi, yi = _index(w, per, r, x_tok), _index(w, per, r, y_tok)
        ref = O.linear(x[xi], wt, None if res is None else res[yi])
        # bound: the float32 accumulation (k terms) plus one rounding of the bfloat16 result
        mag = np.abs(x[xi]).astype(np.float64) @ np.abs(wt).astype(np.float64).T
        tol = BF16_ULP * np.abs(ref) + 1e-5 * mag + 1e-6
        err = np.abs(got[yi] - ref)
        worst = max(worst, float((err / tol).max()))
        assert np.all(err <= tol), f"request {r}: max err {err.max():.3g}"
        touched[yi] = True
    assert np.all(got[~touched] == CANARY), "rows that are not listed were written"
    log(f"  worst error / bound {worst:.3f}")
    plan.close()


def test_gemm_rows_full_tiles_and_k_tail_shapes():
    """Row counts that end exactly on and just past a 256-row tile; k = 64 (one stage), 128 (two)
    and 1024; n = 256 (one feature tile) and 768."""
    specs = [[(512, False, 0, None)], [(257, False, 0, None)]]
    w = W.custom_workload(specs, n_q_heads=8, n_kv_heads=2, head_dim=128, dtype="bf16", rope_base=5e5, seed=3,
                          name="gemm-edges")
    rng = np.random.default_rng(13)
    per = [np.arange(512), np.arange(257)]
    rows = torch.from_numpy(np.concatenate([per[0], per[1]]).astype(np.int32)).cuda()
    n_rows = torch.tensor([512, 257], dtype=torch.int32, device="cuda")
    for K, N in ((64, 256), (128, 512), (1024, 768)):
        x = _bf16(rng, (w.total_tokens, K))
        wt = _bf16(rng, (N, K), 1 / math.sqrt(K))
        plan = sx.Plan(desc_of(w), w.requests, w.n_dst_blocks, w.n_src_blocks)
        y = torch.full((w.total_tokens, N), CANARY, dtype=torch.bfloat16, device="cuda")
        sx.gemm_rows(plan, rows, n_rows, 512, dev(x, w), dev(wt, w), y)
        torch.cuda.synchronize()
        ref = O.linear(x, wt)
        mag = np.abs(x).astype(np.float64) @ np.abs(wt).astype(np.float64).T
        assert np.all(np.abs(host(y) - ref) <= BF16_ULP * np.abs(ref) + 1e-5 * mag + 1e-6), (K, N)
        plan.close()


@pytest.mark.parametrize("x_tok,y_tok", [(True, True), (False, False)])
def test_gemm_rows_split_matches_oracle(x_tok, y_tok):
    """Stacked query / key / value weights in one launch: each output part equals the product with
    its own block of rows of the weight."""
    log(f"[gemm_rows_split] x_tok={x_tok} y_tok={y_tok}")
    w = _ragged_workload()
    rng = np.random.default_rng(14)
    per, rows, n_rows, m = _rows(w, rng, 0.5)
    K, widths, tot = 256, (512, 256, 256), w.total_tokens
    x = _bf16(rng, (tot, K))
    wt = _bf16(rng, (sum(widths), K), 1 / math.sqrt(K))
    plan = sx.Plan(desc_of(w), w.requests, w.n_dst_blocks, w.n_src_blocks)
    ys = [torch.full((tot, n), CANARY, dtype=torch.bfloat16, device="cuda") for n in widths]
    sx.gemm_rows_split(plan, rows, n_rows, m, dev(x, w), dev(wt, w), ys, x_by_token=x_tok, y_by_token=y_tok)
    torch.cuda.synchronize()
    start = 0
    for n, y in zip(widths, ys):
        got = host(y)
        wp = wt[start:start + n]
        touched = np.zeros(tot, bool)
        for r in range(len(w.requests)):
            xi, yi = _index(w, per, r, x_tok), _index(w, per, r, y_tok)
            ref = O.linear(x[xi], wp)
            mag = np.abs(x[xi]).astype(np.float64) @ np.abs(wp).astype(np.float64).T
            err = np.abs(got[yi] - ref)
            assert np.all(err <= BF16_ULP * np.abs(ref) + 1e-5 * mag + 1e-6), f"part at {start}, request {r}"
            touched[yi] = True
        assert np.all(got[~touched] == CANARY), "rows that are not listed were written"
        start += n
    plan.close()


def test_gemm_rows_split_rejects_bad_parts():
    w = _ragged_workload()
    plan = sx.Plan(desc_of(w), w.requests, w.n_dst_blocks, w.n_src_blocks)
    rows = torch.zeros(w.total_tokens, dtype=torch.int32, device="cuda")
    n_rows = torch.zeros(3, dtype=torch.int32, device="cuda")
    x = torch.zeros((w.total_tokens, 128), dtype=torch.bfloat16, device="cuda")
    wt = torch.zeros((384, 128), dtype=torch.bfloat16, device="cuda")
    ys = [torch.zeros((w.total_tokens, n), dtype=torch.bfloat16, device="cuda") for n in (256, 128)]
    with pytest.raises(sx.SxError) as e:
        sx.gemm_rows_split(plan, rows, n_rows, 10, x, wt, ys)   # a part 128 wide
    assert e.value.status == sx.SX_EUNSUPPORTED
    with pytest.raises(ValueError):
        sx.gemm_rows_split(plan, rows, n_rows, 10, x, wt[:256], ys)   # widths add up to 384, w has 256 rows
    plan.close()


def test_gemm_rows_rejects_unsupported_shapes():
    w = _ragged_workload()
    plan = sx.Plan(desc_of(w), w.requests, w.n_dst_blocks, w.n_src_blocks)
    rows = torch.zeros(w.total_tokens, dtype=torch.int32, device="cuda")
    n_rows = torch.zeros(3, dtype=torch.int32, device="cuda")
    x = torch.zeros((w.total_tokens, 96), dtype=torch.bfloat16, device="cuda")
    wt = torch.zeros((256, 96), dtype=torch.bfloat16, device="cuda")
    y = torch.zeros((w.total_tokens, 256), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(sx.SxError) as e:
        sx.gemm_rows(plan, rows, n_rows, 10, x, wt, y)   # k = 96 is not a multiple of 64
    assert e.value.status == sx.SX_EUNSUPPORTED
    plan.close()


@pytest.mark.parametrize("x_tok,y_tok", [(True, False), (False, True)])
def test_rmsnorm_rows_matches_oracle(x_tok, y_tok):
    w = _ragged_workload()
    rng = np.random.default_rng(14)
    per, rows, n_rows, m = _rows(w, rng, 0.5)
    H, tot, eps = 1024, w.total_tokens, 1e-5
    x = _bf16(rng, (tot, H), 2.0)
    gamma = O.to_bf16((1 + 0.2 * rng.standard_normal(H)).astype(np.float32))
    plan = sx.Plan(desc_of(w), w.requests, w.n_dst_blocks, w.n_src_blocks)
    y = torch.full((tot, H), CANARY, dtype=torch.bfloat16, device="cuda")
    sx.rmsnorm_rows(plan, rows, n_rows, m, dev(x, w), dev(gamma, w), eps, y, x_by_token=x_tok, y_by_token=y_tok)
    torch.cuda.synchronize()
    got = host(y)
    touched = np.zeros(tot, bool)
    for r in range(len(w.requests)):
        xi, yi = _index(w, per, r, x_tok), _index(w, per, r, y_tok)
        ref = O.rmsnorm(x[xi], gamma, eps)
        assert np.all(np.abs(got[yi] - ref) <= 2 * BF16_ULP * np.abs(ref) + 1e-6), f"request {r}"
        touched[yi] = True
    assert np.all(got[~touched] == CANARY)
    plan.close()


@pytest.mark.parametrize("style", ["neox", "gptj"])
def test_rope_rows_matches_oracle(style):
    rng = np.random.default_rng(15)
    specs = [W.random_request_specs(rng, T, max_pos=120000) for T in (300, 90)]
    w = W.custom_workload(specs, n_q_heads=8, n_kv_heads=2, head_dim=128, dtype="bf16", rope_base=5e5,
                          rope_style=style, seed=15, name="rope-rows")
    per, rows, n_rows, m = _rows(w, rng, 0.4)
    tot = w.total_tokens
    q = _bf16(rng, (tot, 8, 128))
    k = _bf16(rng, (tot, 2, 128))
    plan = sx.Plan(desc_of(w), w.requests, w.n_dst_blocks, w.n_src_blocks)
    qd, kd = dev(q, w), dev(k, w)
    sx.rope_rows(plan, rows, n_rows, m, qd, kd)
    torch.cuda.synchronize()
    gq, gk = host(qd), host(kd)
    worst, exact, total = 0.0, 0, 0
    listed = np.zeros(tot, bool)
    for r, req in enumerate(w.requests):
        _, pos, _ = O.token_layout(req.n_tokens, req.segments)
        ti = w.token_offsets[r] + per[r]
        for got, src in ((gq, q), (gk, k)):
            ref = O.store(O.rope_at_positions(src[ti], pos[per[r]], w.rope_base, style), "bf16")
            worst = max(worst, float(np.abs(got[ti] - ref).max()))
            exact += int(np.sum(got[ti] == ref))
            total += ref.size
        listed[ti] = True
    log(f"[rope_rows] {style}: max-abs {worst:.3g}, bit-identical {exact}/{total}")
    assert worst <= 1e-2
    assert np.array_equal(gq[~listed], q[~listed]) and np.array_equal(gk[~listed], k[~listed])
    plan.close()


def test_silu_mul_rows_matches_oracle():
    w = _ragged_workload()
    rng = np.random.default_rng(16)
    per, rows, n_rows, m = _rows(w, rng, 0.7)
    F, tot = 1024, w.total_tokens
    gu = _bf16(rng, (tot, 2 * F), 3.0)
    plan = sx.Plan(desc_of(w), w.requests, w.n_dst_blocks, w.n_src_blocks)
    y = torch.full((tot, F), CANARY, dtype=torch.bfloat16, device="cuda")
    sx.silu_mul_rows(plan, n_rows, m, dev(gu, w), y)
    torch.cuda.synchronize()
    got = host(y)
    touched = np.zeros(tot, bool)
    for r in range(len(w.requests)):
        si = _index(w, per, r, False)
        ref = O.silu_mul(gu[si])
        assert np.all(np.abs(got[si] - ref) <= 2 * BF16_ULP * np.abs(ref) + 1e-6), f"request {r}"
        touched[si] = True
    assert np.all(got[~touched] == CANARY)
    plan.close()


def layer_weights(rng, H, Hq, Hkv, d, F):
    def m(o, i):
        return _bf16(rng, (o, i), 1 / math.sqrt(i))
    return {"ln1": O.to_bf16((1 + 0.1 * rng.standard_normal(H)).astype(np.float32)), "wq": m(Hq * d, H),
            "wk": m(Hkv * d, H), "wv": m(Hkv * d, H), "wo": m(H, Hq * d),
            "ln2": O.to_bf16((1 + 0.1 * rng.standard_normal(H)).astype(np.float32)), "wgu": m(2 * F, H),
            "wd": m(H, F)}


def run_layer_body(plan, w, rows, n_rows, max_rows, hidden, wd, src_k, src_v, kc, vc, eps, bufs):
    """One sparse layer on the device through the C ABI (the call sequence bench.py times)."""
    Hq, Hkv, d = w.n_q_heads, w.n_kv_heads, w.head_dim
    b = bufs
    sx.rmsnorm_rows(plan, rows, n_rows, max_rows, hidden, wd["ln1"], eps, b["x1"], x_by_token=True)
    # the query, key and value projections in one launch (wd["wqkv"] stacks wq, wk, wv)
    sx.gemm_rows_split(plan, rows, n_rows, max_rows, b["x1"], wd["wqkv"], [b["q"], b["k"], b["v"]],
                       y_by_token=True)
    sx.rope_rows(plan, rows, n_rows, max_rows, b["q"], b["k"])
    sx.rows_mask(plan, rows, n_rows, max_rows, b["mask"])
    sx.realign_scatter_masked(plan, src_k, src_v, b["k"], b["v"], b["mask"], kc, vc)
    sx.sparse_attn(plan, b["q"], rows, n_rows, max_rows, kc, vc, b["att"])
    sx.gemm_rows(plan, rows, n_rows, max_rows, b["att"].view(-1, Hq * d), wd["wo"], b["h1"], residual=hidden,
                 y_by_token=True)
    sx.rmsnorm_rows(plan, rows, n_rows, max_rows, b["h1"], wd["ln2"], eps, b["x2"], x_by_token=True)
    sx.gemm_rows(plan, rows, n_rows, max_rows, b["x2"], wd["wgu"], b["gu"])
    sx.silu_mul_rows(plan, n_rows, max_rows, b["gu"], b["a"])
    sx.gemm_rows(plan, rows, n_rows, max_rows, b["a"], wd["wd"], b["h2"], residual=b["h1"], y_by_token=True)


def layer_buffers(tot, H, Hq, Hkv, d, F):
    z = lambda *s: torch.zeros(s, dtype=torch.bfloat16, device="cuda")
    return {"x1": z(tot, H), "q": z(tot, Hq, d), "k": z(tot, Hkv, d), "v": z(tot, Hkv, d),
            "mask": torch.zeros(tot, dtype=torch.uint8, device="cuda"), "att": z(tot, Hq, d), "h1": z(tot, H),
            "x2": z(tot, H), "gu": z(tot, 2 * F), "a": z(tot, F), "h2": z(tot, H)}


def test_layer_body_matches_oracle():
    """One sparse layer of a request with cached and uncached segments (R = I_nr, the overflow
    rows and a random third of the reused tokens) against oracle.layer_body."""
    specs = [[(96, True, 0, None), (48, False, 0, None), (160, True, 700, None), (64, False, 0, None),
              (144, True, 40, None)]]
    w = W.custom_workload(specs, n_q_heads=8, n_kv_heads=2, head_dim=128, dtype="bf16", rope_base=5e5, seed=21,
                          name="layer-body")
    req = w.requests[0]
    T = req.n_tokens
    Hq, Hkv, d, H, F, eps = 8, 2, 128, 1024, 1024, 1e-5
    rng = np.random.default_rng(22)
    base = O.recompute_set(T, req.segments, np.zeros(T), 0.0, w.block_size)["R"]
    extra = rng.choice(O.reuse_positions(T, req.segments), size=T // 3, replace=False)
    R = np.unique(np.concatenate([base, extra]))
    hidden = _bf16(rng, (T, H))
    wts = layer_weights(rng, H, Hq, Hkv, d, F)
    t = W.layer_tensors(w, 0)
    ref = O.layer_body(w, hidden, R, wts, t["k_src"], t["v_src"], eps)

    plan = sx.Plan(desc_of(w), w.requests, w.n_dst_blocks, w.n_src_blocks)
    rows = torch.zeros(T, dtype=torch.int32, device="cuda")
    rows[:len(R)] = torch.from_numpy(R.astype(np.int32)).cuda()
    n_rows = torch.tensor([len(R)], dtype=torch.int32, device="cuda")
    wd = {kk: dev(v, w) for kk, v in wts.items()}
    wd["wqkv"] = dev(np.concatenate([wts["wq"], wts["wk"], wts["wv"]]), w)
    shape = (w.n_dst_blocks, Hkv, w.block_size, d)
    kc = torch.full(shape, CANARY, dtype=torch.bfloat16, device="cuda")
    vc = torch.full(shape, CANARY, dtype=torch.bfloat16, device="cuda")
    bufs = layer_buffers(T, H, Hq, Hkv, d, F)
    run_layer_body(plan, w, rows, n_rows, len(R), dev(hidden, w), wd, dev(t["k_src"], w), dev(t["v_src"], w), kc, vc,
                   eps, bufs)
    torch.cuda.synchronize()
    n = len(R)
    checks = [("x1", host(bufs["x1"])[:n]), ("q", host(bufs["q"])[R]), ("k", host(bufs["k"])[R]),
              ("h1", host(bufs["h1"])[R]), ("h2", host(bufs["h2"])[R])]
    for name, got in checks:
        want = ref[name]
        err = np.abs(got.reshape(want.shape) - want)
        rel = err / np.maximum(np.abs(want), 1.0)
        log(f"[layer_body] {name}: max-abs {err.max():.3g}, relative to max(|x|, 1): max {rel.max():.3g}, "
            f"rms {math.sqrt(float(np.mean(rel ** 2))):.3g}")
    # Bound derived from the arithmetic: the chain stores eight bfloat16 intermediates; where the
    # GPU's float32 summation order puts a value on the other side of a rounding boundary, that
    # intermediate differs by one step (each operation alone is within one or two steps of the
    # oracle, tested above), and later matrix products sum many such one-step differences.  So a
    # few elements of the last outputs sit several steps away while the typical deviation stays
    # below one step: the bar is 8 steps of max(|x|, 1) per element and an RMS deviation below one
    # step.  A wiring mistake (a residual dropped, a row mixed up, a wrong RoPE position) moves
    # elements by whole units.
    for name, got in checks:
        want = ref[name]
        rel = np.abs(got.reshape(want.shape) - want) / np.maximum(np.abs(want), 1.0)
        assert rel.max() <= 8 * BF16_ULP, (name, rel.max())
        assert math.sqrt(float(np.mean(rel ** 2))) <= BF16_ULP, (name, math.sqrt(float(np.mean(rel ** 2))))
    # the request's cache slots (the spare blocks hold the canary on the device, zeros in the oracle)
    kt = O.gather_tokens(req, w, host(kc))
    want_k = O.gather_tokens(req, w, ref["k_pool"])
    assert np.all(np.abs(kt - want_k) <= 8 * BF16_ULP * np.maximum(np.abs(want_k), 1.0))
    assert np.array_equal(O.gather_tokens(req, w, host(vc))[np.setdiff1d(np.arange(T), R)],
                          O.gather_tokens(req, w, ref["v_pool"])[np.setdiff1d(np.arange(T), R)])
    plan.close()


def test_layer_body_full_size_sampled_rows():
    """The layer body at the benchmark's size and launch configuration (the 32768-token chat stack:
    32/8/128 heads, hidden 4096, feed-forward 14336, the 6712 rows of its stored recompute set),
    each operation checked on 64 sampled rows against the oracle fed with the GPU's own inputs to
    that operation (a row of every output depends only on that row of the inputs and the weights,
    so a sampled row is an exact check).  The attention output is replaced by seeded values: the
    attention kernels have their own full-size tests."""
    import os
    w = W.config(3)
    req = w.requests[0]
    T = req.n_tokens
    Hq, Hkv, d, H, F, eps = w.n_q_heads, w.n_kv_heads, w.head_dim, 4096, 14336, 1e-5
    R = np.load(os.path.join(os.path.dirname(__file__), "golden", "c3_boundary.npz"))["R"].astype(np.int64)
    log(f"[layer_body full size] T={T} |R|={len(R)} hidden={H} ffn={F}")
    rng = np.random.default_rng(31)
    hidden = _bf16(rng, (T, H))
    att = _bf16(rng, (T, Hq * d))
    wts = {"ln1": O.to_bf16((1 + 0.1 * rng.standard_normal(H)).astype(np.float32)),
           "wqkv": _bf16(rng, ((Hq + 2 * Hkv) * d, H), 1 / math.sqrt(H)),
           "wo": _bf16(rng, (H, Hq * d), 1 / math.sqrt(Hq * d)),
           "ln2": O.to_bf16((1 + 0.1 * rng.standard_normal(H)).astype(np.float32)),
           "wgu": _bf16(rng, (2 * F, H), 1 / math.sqrt(H)),
           "wd": _bf16(rng, (H, F), 1 / math.sqrt(F))}
    plan = sx.Plan(desc_of(w), w.requests, w.n_dst_blocks, w.n_src_blocks)
    rows = torch.zeros(T, dtype=torch.int32, device="cuda")
    rows[:len(R)] = torch.from_numpy(R.astype(np.int32)).cuda()
    n_rows = torch.tensor([len(R)], dtype=torch.int32, device="cuda")
    m = len(R)
    z = lambda *s: torch.zeros(s, dtype=torch.bfloat16, device="cuda")
    wd = {k: dev(v, w) for k, v in wts.items()}
    hid, atd = dev(hidden, w), dev(att, w)
    x1, q, k, v, h1, x2, gu, a = z(T, H), z(T, Hq, d), z(T, Hkv, d), z(T, Hkv, d), z(T, H), z(T, H), z(T, 2 * F), z(T, F)
    sx.rmsnorm_rows(plan, rows, n_rows, m, hid, wd["ln1"], eps, x1, x_by_token=True)
    sx.gemm_rows_split(plan, rows, n_rows, m, x1, wd["wqkv"], [q, k, v], y_by_token=True)
    qk_pre = (host(q), host(k))
    sx.rope_rows(plan, rows, n_rows, m, q, k)
    sx.gemm_rows(plan, rows, n_rows, m, atd, wd["wo"], h1, residual=hid, y_by_token=True)
    sx.rmsnorm_rows(plan, rows, n_rows, m, h1, wd["ln2"], eps, x2, x_by_token=True)
    sx.gemm_rows(plan, rows, n_rows, m, x2, wd["wgu"], gu)
    sx.silu_mul_rows(plan, n_rows, m, gu, a)
    h1_before = host(h1)
    sx.gemm_rows(plan, rows, n_rows, m, a, wd["wd"], hid, residual=h1, y_by_token=True)
    torch.cuda.synchronize()

    pick = np.unique(np.concatenate([[0, 1, m - 2, m - 1], rng.choice(m, 60, replace=False)]))
    tok = R[pick]          # token rows of the sampled slots
    g = {n: host(t) for n, t in (("x1", x1), ("q", q), ("k", k), ("x2", x2), ("gu", gu), ("a", a), ("h2", hid))}

    def gemm_ok(name, xin, wt, got, res=None):
        ref = O.linear(xin, wt, res)
        mag = np.abs(xin).astype(np.float64) @ np.abs(wt).astype(np.float64).T
        bound = BF16_ULP * np.abs(ref) + 1e-5 * mag + 1e-6
        worst = float((np.abs(got - ref) / bound).max())
        log(f"  {name}: worst error / bound {worst:.3f}")
        assert worst <= 1.0, name

    # RMSNorm of the hidden states (token rows in, slot rows out)
    ref = O.rmsnorm(hidden[tok], wts["ln1"], eps)
    assert np.all(np.abs(g["x1"][pick] - ref) <= 2 * BF16_ULP * np.abs(ref) + 1e-6)
    # stacked Q/K/V (slot rows in, token rows out), before RoPE
    n_q = Hq * d
    gemm_ok("q|k|v", g["x1"][pick], wts["wqkv"],
            np.concatenate([qk_pre[0][tok].reshape(len(tok), -1), qk_pre[1][tok].reshape(len(tok), -1),
                            host(v)[tok].reshape(len(tok), -1)], axis=1))
    # RoPE at the tokens' positions in the new sequence, bit for bit
    _, pos, _ = O.token_layout(T, req.segments)
    for got, pre in ((g["q"], qk_pre[0]), (g["k"], qk_pre[1])):
        want = O.store(O.rope_at_positions(pre[tok], pos[tok], w.rope_base, w.rope_style), "bf16")
        assert np.array_equal(got[tok], want)
    # output projection + residual, RMSNorm, gate|up, SwiGLU, down projection + residual
    gemm_ok("o + residual", att[pick], wts["wo"], h1_before[tok], res=hidden[tok])
    ref = O.rmsnorm(h1_before[tok], wts["ln2"], eps)
    assert np.all(np.abs(g["x2"][pick] - ref) <= 2 * BF16_ULP * np.abs(ref) + 1e-6)
    gemm_ok("gate|up", g["x2"][pick], wts["wgu"], g["gu"][pick])
    ref = O.silu_mul(g["gu"][pick])
    assert np.all(np.abs(g["a"][pick] - ref) <= 2 * BF16_ULP * np.abs(ref) + 1e-6)
    gemm_ok("down + residual", g["a"][pick], wts["wd"], g["h2"][tok], res=h1_before[tok])
    # rows outside R keep their hidden state
    others = np.setdiff1d(np.arange(T), R)[:: max(1, (T - m) // 512)]
    assert np.array_equal(g["h2"][others], hidden[others])
    plan.close()


def test_layer_ops_with_an_empty_request():
    """A request whose row list is empty (n_rows = 0) between two that have rows: nothing of it is
    read or written, the others are computed as usual (GEMM, split GEMM, RMSNorm, RoPE, SwiGLU)."""
    w = _ragged_workload(seed=17)
    rng = np.random.default_rng(18)
    per, rows, n_rows, m = _rows(w, rng, 0.5)
    per[1] = per[1][:0]
    n_rows[1] = 0
    tot, K, N, F = w.total_tokens, 256, 512, 256
    x = _bf16(rng, (tot, K))
    wt = _bf16(rng, (N, K), 1 / math.sqrt(K))
    gamma = O.to_bf16((1 + 0.2 * rng.standard_normal(K)).astype(np.float32))
    gu = _bf16(rng, (tot, 2 * F), 2.0)
    q = _bf16(rng, (tot, 8, 128))
    k = _bf16(rng, (tot, 2, 128))
    plan = sx.Plan(desc_of(w), w.requests, w.n_dst_blocks, w.n_src_blocks)
    full = lambda n: torch.full((tot, n), CANARY, dtype=torch.bfloat16, device="cuda")
    y, y1, y2, xn, a = full(N), full(256), full(256), full(K), full(F)
    qd, kd = dev(q, w), dev(k, w)
    sx.gemm_rows(plan, rows, n_rows, m, dev(x, w), dev(wt, w), y, x_by_token=True, y_by_token=True)
    sx.gemm_rows_split(plan, rows, n_rows, m, dev(x, w), dev(wt, w), [y1, y2], x_by_token=True, y_by_token=True)
    sx.rmsnorm_rows(plan, rows, n_rows, m, dev(x, w), dev(gamma, w), 1e-5, xn, x_by_token=True, y_by_token=True)
    sx.silu_mul_rows(plan, n_rows, m, dev(gu, w), a)
    sx.rope_rows(plan, rows, n_rows, m, qd, kd)
    torch.cuda.synchronize()
    off = w.token_offsets
    for r in range(3):
        ti = off[r] + per[r]
        si = off[r] + np.arange(len(per[r]))
        span = np.arange(off[r], off[r + 1])
        if r == 1:   # the empty request: its rows keep the canary / their input values
            for t in (y, y1, y2, xn, a):
                assert np.all(host(t)[span] == CANARY)
            assert np.array_equal(host(qd)[span], q[span]) and np.array_equal(host(kd)[span], k[span])
            continue
        ref = O.linear(x[ti], wt)
        mag = np.abs(x[ti]).astype(np.float64) @ np.abs(wt).astype(np.float64).T
        bound = BF16_ULP * np.abs(ref) + 1e-5 * mag + 1e-6
        assert np.all(np.abs(host(y)[ti] - ref) <= bound)
        assert np.all(np.abs(np.concatenate([host(y1)[ti], host(y2)[ti]], axis=1) - ref) <= bound)
        ref = O.rmsnorm(x[ti], gamma, 1e-5)
        assert np.all(np.abs(host(xn)[ti] - ref) <= 2 * BF16_ULP * np.abs(ref) + 1e-6)
        ref = O.silu_mul(gu[si])
        assert np.all(np.abs(host(a)[si] - ref) <= 2 * BF16_ULP * np.abs(ref) + 1e-6)
    plan.close()
