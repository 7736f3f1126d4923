"""Throughput of the sparse-KV recomputation step on one MI355X.

Default workload: the 32-layer hybrid chat stack (T = 32768 tokens, 32 query / 8 KV heads,
head_dim 128, bf16, recompute ratio 15 %).  One step is one pass of the whole path over the
stack:
    layers 0-3   KV write of every row + full causal attention
    boundary     Sparse-Q scoring + top-k selection on layer 3 (fresh keys of every token)
    layers 4-31  RoPE re-alignment + KV write of R + sparse attention of R
Inputs (per-layer Q/K/V and source pools, seeded N(0,1)) are resident in HBM before timing.

value = effective prefill tokens/s per layer = T * L / (seconds per step).

Prints one JSON line with the metric, per-kernel timings (HIP events on the launch stream),
the roofline of the dominant kernel and the CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 matrix peak
PEAK_F32_TFLOPS = 157.3       # MI355X fp32 vector peak
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
METRIC = "effective prefill tokens/s per layer at 15% recompute; MFMA util + HBM GB/s"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=3, help="named workload c1..c5")
    ap.add_argument("--ratio", type=float, default=None)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-peaks", action="store_true", help="skip the copy / GEMM measurement of achievable peaks")
    ap.add_argument("--layers", type=int, default=None, help="override the number of layers (profiling)")
    ap.add_argument("--buffer-sets", type=int, default=None,
                    help="distinct per-layer input/cache buffer sets, layer l uses set l mod N (default: one per "
                         "layer; the 400k-token batch rotates 3 sets, since 32 resident layers would not fit)")
    ap.add_argument("--score-passes", type=int, choices=(1, 2), default=1,
                    help="Sparse-Q scoring in hybrid stacks: 1 = denominators from the boundary layer's full "
                         "attention (exact-logit variant), 2 = own log-sum-exp pass")
    ap.add_argument("--kv-write", choices=("per-layer", "per-layer-rows", "all-layers", "separate"),
                    default="per-layer",
                    help="sparse layers' re-alignment + KV write of R: one pass per layer just before its "
                         "attention with R as a byte mask built once per step (default; the attention then finds "
                         "part of the cache in the Infinity Cache), the same from the row list (marks R per "
                         "layer), one pass for all sparse layers after the selection, or two passes per layer")
    ap.add_argument("--layer-body", action="store_true",
                    help="run every sparse layer as a whole layer (Algorithm 1 steps 19-22): RMSNorm, Q/K/V "
                         "projections of the rows of R, RoPE, KV write, sparse attention, output projection + "
                         "residual, RMSNorm, SwiGLU feed-forward + residual, with random weights of a Llama-3-8B "
                         "layer (hidden 4096, feed-forward 14336); the value is then whole-layer throughput")
    ap.add_argument("--ffn", type=int, default=14336, help="feed-forward size of --layer-body")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="also run a plain device copy of BYTES bytes (reference for HBM byte counters)")
    ap.add_argument("--record-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="turn two rocprofv3 --pmc counter CSVs (FETCH_SIZE, WRITE_SIZE) of a run with "
                         "--copy-calibration into profiles/traffic_<workload>.json, then exit")
    return ap.parse_args()


# kernel symbol -> (entry point, source file holding it, whether each dispatch is one call of the
# entry point; the others run inside a call beside such a kernel)
# (attention template arguments: head dim, paged, P.V product, persistent grid)
KERNELS = {
    "attn_mfma_kernel<128, true, true, true>": ("sx_sparse_attn", "k_attn.hip", True),
    "attn_mfma_kernel<128, false, true, true>": ("sx_full_attn", "k_attn.hip", True),
    "attn_mfma_kernel<128, false, true, false>": ("sx_full_attn", "k_attn.hip", True),   # (under graph capture)
    # two-pass scoring only (layers without a preceding full layer)
    "attn_mfma_kernel<128, true, false, false>": ("sx_sparseq_score", "k_attn.hip", False),
    "lse_merge_kernel": ("sx_sparseq_score", "k_attn.hip", False),
    "colsum_kernel<128, 2>": ("sx_sparseq_score", "k_attn.hip", True),
    "colsum_kernel<128, 1>": ("sx_sparseq_score", "k_attn.hip", True),
    "probe_gather_kernel<128>": ("sx_sparseq_score", "k_attn.hip", False),
    "head_reduce_kernel": ("sx_sparseq_score", "k_copy.hip", False),
    "realign_kernel": ("sx_rope_realign", "k_copy.hip", True),
    "scatter_kernel": ("sx_kv_scatter", "k_copy.hip", True),
    "realign_scatter_kernel": ("sx_realign_scatter_masked", "k_copy.hip", True),   # (also the row-list variants)
    "mark_rows_kernel": ("sx_realign_scatter", "k_copy.hip", False),   # (also sx_realign_scatter_layers)
    "fill_u8_kernel": ("sx_rows_mask", "k_copy.hip", True),
    "mask_rows_kernel": ("sx_rows_mask", "k_copy.hip", False),
    "tile_order_kernel": ("sx_rows_mask", "k_attn.hip", False),
    "topk_hist_kernel": ("sx_topk_select", "k_topk.hip", False),
    "topk_bound_kernel": ("sx_topk_select", "k_topk.hip", False),
    "topk_write_kernel": ("sx_topk_select", "k_topk.hip", True),
}


def source_code(text):
    """A kernel source with its comments and blank space removed: what the compiler sees of it."""
    import re
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def source_hash(fname):
    """Hash of a kernel source's code (comments and layout do not count): traffic counters taken on
    one version of the code stay valid while the code is unchanged."""
    import hashlib
    path = os.path.join(ROOT, "paper_2606_01751_amd", "csrc", fname)
    return hashlib.sha256(source_code(open(path).read()).encode()).hexdigest()[:16]


def record_traffic(fetch_csv, write_csv, workload):
    """HBM bytes per dispatch of each kernel from FETCH_SIZE / WRITE_SIZE (KiB per dispatch),
    scaled by the ratio of the true bytes of the largest plain device copy in the same run to
    what the counters report for it."""
    import csv
    import re

    def per_kernel(path, counter):
        acc, copy = {}, []
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            v = float(r["Counter_Value"])
            if "copyBuffer" in r["Kernel_Name"]:
                copy.append((int(r["Grid_Size"]), v))
            name = re.sub(r"\s", "", r["Kernel_Name"])
            for sym in KERNELS:
                # whole identifier only (scatter_kernel is also the tail of realign_scatter_kernel)
                if re.search(r"(?<![A-Za-z0-9_])" + re.escape(sym.replace(" ", "")), name):
                    acc.setdefault(sym, []).append(v)
        return acc, max(copy)[1] if copy else None

    fetch, cf = per_kernel(fetch_csv, "FETCH_SIZE")
    write, cw = per_kernel(write_csv, "WRITE_SIZE")
    return fetch, write, cf, cw


def load_traffic(workload):
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return {}
    d = json.load(open(path))
    total, calls, stale = {}, {}, set()
    for sym, e in d.get("kernels", {}).items():
        if sym not in KERNELS:
            continue
        entry, src, is_call = KERNELS[sym]
        if e.get("source_sha256") != source_hash(src):
            stale.add(entry)       # the kernel changed since its counters were taken
            continue
        n = e.get("dispatches", 1)
        total[entry] = total.get(entry, 0.0) + e["bytes_per_dispatch"] * n
        if is_call:
            calls[entry] = calls.get(entry, 0) + n
    # bytes per call of the entry point: the dispatch-weighted mean over its variants, plus the
    # kernels that run inside each call
    return {k: v / calls[k] for k, v in total.items() if k not in stale and calls.get(k)}


class Timers:
    """HIP events around each launch, recorded on the stream the library launches on."""

    def __init__(self, torch):
        self.torch = torch
        self.ev = {}
        self.on = False

    def run(self, name, fn):
        if not self.on:
            fn()
            return
        s = self.torch.cuda.Event(enable_timing=True)
        e = self.torch.cuda.Event(enable_timing=True)
        s.record()
        fn()
        e.record()
        self.ev.setdefault(name, []).append((s, e))

    def summary(self):
        out = {}
        for k, lst in self.ev.items():
            ms = [s.elapsed_time(e) for s, e in lst]
            p10, p50, p90 = np.percentile(ms, [10, 50, 90])
            out[k] = {"launches": len(ms), "avg_ms": float(np.mean(ms)), "total_ms": float(np.sum(ms)),
                      "p10_ms": float(p10), "median_ms": float(p50), "p90_ms": float(p90)}
        return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported (the step is not sharded).",
              file=sys.stderr)
        sys.exit(2)
    if args.record_traffic:
        import workloads as W
        w = W.config(args.config, seed=args.seed)
        fetch, write, cf, cw = record_traffic(*args.record_traffic, w.name)
        nbytes = args.copy_calibration
        assert nbytes and cf and cw, "need --copy-calibration BYTES and a copy in both counter runs"
        kf, kw = nbytes / 1024.0 / cf, nbytes / 1024.0 / cw
        rec = {"workload": w.name, "copy_bytes": nbytes, "copy_fetch_kib": cf, "copy_write_kib": cw,
               "fetch_factor": kf, "write_factor": kw, "kernels": {}}
        for sym in sorted(set(fetch) | set(write)):
            f = float(np.mean(fetch.get(sym, [0.0])))
            wr = float(np.mean(write.get(sym, [0.0])))
            rec["kernels"][sym] = {"entry_point": KERNELS[sym][0], "source_sha256": source_hash(KERNELS[sym][1]),
                                   "dispatches": max(len(fetch.get(sym, [])), len(write.get(sym, []))),
                                   "fetch_kib": f, "write_kib": wr,
                                   "bytes_per_dispatch": (f * kf + wr * kw) * 1024.0}
        out = os.path.join(ROOT, "profiles", f"traffic_{w.name}.json")
        json.dump(rec, open(out, "w"), indent=1)
        print(json.dumps(rec, indent=1))
        return
    import torch

    import paper_2606_01751_amd as sx
    import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    w = W.config(args.config, seed=args.seed)
    ratio = args.ratio if args.ratio is not None else (0.15 if 0.15 in w.ratios else w.ratios[0])
    L = args.layers if args.layers else w.n_layers
    nfull = min(w.n_full_layers, L)
    T = w.total_tokens
    Hq, Hkv, d = w.n_q_heads, w.n_kv_heads, w.head_dim
    esz = 2 if w.dtype == "bf16" else 4
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    desc = sx.make_desc(Hq, Hkv, d, w.dtype, w.rope_base, w.rope_style)
    plan = sx.Plan(desc, w.requests, w.n_dst_blocks, w.n_src_blocks)
    info = plan.info()
    k_total, max_rows = plan.budget(ratio)
    log(f"workload {w.name}: T={T} layers={L} (full {nfull}) ratio={ratio} k={k_total} max_rows={max_rows}")

    t0 = time.time()
    # per-layer buffers; with --buffer-sets N the layers rotate N sets (each far beyond the 256 MB
    # Infinity Cache, so no layer finds the previous one's data there)
    nsets = args.buffer_sets if args.buffer_sets else (3 if w.total_tokens > 200000 else L)
    nsets = max(1, min(nsets, L))
    sets = []
    pool = (w.n_dst_blocks, Hkv, w.block_size, d)
    for l in range(nsets):
        need = ("q", "k", "v") + (("k_src", "v_src") if (l >= nfull or nsets < L) else ())
        tl = W.layer_tensors_torch(w, l, args.seed, which=need)
        tl["kc"] = torch.zeros(pool, dtype=dt, device="cuda")
        tl["vc"] = torch.zeros(pool, dtype=dt, device="cuda")
        sets.append(tl)
    layers = [sets[l % nsets] for l in range(L)]
    out = torch.empty((T, Hq, d), dtype=dt, device="cuda")
    lse = torch.empty((T, Hq), dtype=torch.float32, device="cuda")   # boundary layer's denominators
    rmask = torch.zeros(T, dtype=torch.uint8, device="cuda")           # R as a byte mask
    scores = torch.zeros(T, dtype=torch.float32, device="cuda")
    rows = torch.zeros(T, dtype=torch.int32, device="cuda")
    n_rows = torch.zeros(len(w.requests), dtype=torch.int32, device="cuda")
    cu = torch.tensor(w.token_offsets, dtype=torch.int32, device="cuda")
    max_T = max(r.n_tokens for r in w.requests)
    nr_rows, nr_n, nr_max = plan.nonreused_rows()
    torch.cuda.synchronize()
    log(f"inputs resident in HBM ({torch.cuda.memory_allocated() / 2**30:.1f} GiB, {nsets} buffer sets for {L} "
        f"layers) in {time.time() - t0:.1f}s")

    H, F, eps = Hq * d, args.ffn, 1e-5
    body = None
    if args.layer_body:
        # per sparse layer: its own random weights (~N(0, 1/fan_in), bf16); one hidden-state buffer
        # carried from layer to layer; per-step scratch for the intermediates
        gen = torch.Generator(device="cuda")
        gen.manual_seed(args.seed + 12345)

        def lin(o, i):
            return (torch.randn((o, i), generator=gen, device="cuda", dtype=torch.float32) / math.sqrt(i)).to(dt)

        def norm_w():
            return (1 + 0.1 * torch.randn(H, generator=gen, device="cuda", dtype=torch.float32)).to(dt)
        body = {"w": [], "hidden": torch.randn((T, H), generator=gen, device="cuda", dtype=torch.float32).to(dt)}
        for l in range(nfull, L):
            # wqkv stacks the query, key and value projections ([(Hq + 2 Hkv) d][H])
            body["w"].append({"ln1": norm_w(), "wqkv": lin((Hq + 2 * Hkv) * d, H), "wo": lin(H, Hq * d),
                              "ln2": norm_w(), "wgu": lin(2 * F, H), "wd": lin(H, F)})
        z = lambda *shape: torch.zeros(shape, dtype=dt, device="cuda")
        body.update({"x1": z(T, H), "att": z(T, Hq, d), "h1": z(T, H), "x2": z(T, H), "gu": z(T, 2 * F),
                     "a": z(T, F)})
        torch.cuda.synchronize()
        log(f"layer body: {len(body['w'])} layers of weights ({torch.cuda.memory_allocated() / 2**30:.1f} GiB resident)")

    def sparse_layer_body(l, tl):
        """Algorithm 1 steps 19-22 for sparse layer l on the rows of R: the fresh Q/K/V of R are
        projected into the layer's token-indexed q/k/v buffers, the hidden states of R updated in
        place."""
        wl = body["w"][l - nfull]
        hid = body["hidden"]
        tm.run("sx_rmsnorm_rows", lambda: sx.rmsnorm_rows(plan, rows, n_rows, max_rows, hid, wl["ln1"], eps, body["x1"],
                                                          x_by_token=True))
        tm.run("sx_gemm_rows qkv", lambda: sx.gemm_rows_split(plan, rows, n_rows, max_rows, body["x1"], wl["wqkv"],
                                                              [tl["q"], tl["k"], tl["v"]], y_by_token=True))
        tm.run("sx_rope_rows", lambda: sx.rope_rows(plan, rows, n_rows, max_rows, tl["q"], tl["k"]))
        tm.run("sx_realign_scatter_masked",
               lambda: sx.realign_scatter_masked(plan, tl["k_src"], tl["v_src"], tl["k"], tl["v"], rmask, tl["kc"],
                                                 tl["vc"]))
        tm.run("sx_sparse_attn", lambda: sx.sparse_attn(plan, tl["q"], rows, n_rows, max_rows, tl["kc"], tl["vc"],
                                                        body["att"]))
        tm.run("sx_gemm_rows o", lambda: sx.gemm_rows(plan, rows, n_rows, max_rows, body["att"].view(T, H), wl["wo"],
                                                      body["h1"], residual=hid, y_by_token=True))
        tm.run("sx_rmsnorm_rows", lambda: sx.rmsnorm_rows(plan, rows, n_rows, max_rows, body["h1"], wl["ln2"], eps,
                                                          body["x2"], x_by_token=True))
        tm.run("sx_gemm_rows gate_up", lambda: sx.gemm_rows(plan, rows, n_rows, max_rows, body["x2"], wl["wgu"],
                                                            body["gu"]))
        tm.run("sx_silu_mul_rows", lambda: sx.silu_mul_rows(plan, n_rows, max_rows, body["gu"], body["a"]))
        tm.run("sx_gemm_rows down", lambda: sx.gemm_rows(plan, rows, n_rows, max_rows, body["a"], wl["wd"], hid,
                                                         residual=body["h1"], y_by_token=True))

    tm = Timers(torch)
    sparse_kv = [(tl["k_src"], tl["v_src"], tl["k"], tl["v"], tl["kc"], tl["vc"])
                 for l, tl in enumerate(layers) if l >= nfull and not (nfull == 0 and l == 0)]

    def step():
        for l in range(nfull):
            tl = layers[l]
            # the last full layer is the selecting (boundary) layer: with --score-passes 1 its attention
            # also writes the softmax denominators of every row and the Sparse-Q scoring makes one pass
            lse_l = lse if (l == nfull - 1 and args.score_passes == 1) else None
            tm.run("sx_kv_scatter", lambda: sx.kv_scatter(plan, tl["k"], tl["v"], tl["kc"], tl["vc"]))
            tm.run("sx_full_attn", lambda: sx.full_attn(desc, tl["q"], tl["k"], tl["v"], cu, len(w.requests), max_T,
                                                        out, lse_l))
        if nfull == 0:
            # single selecting layer: mixed keys (re-aligned cached + fresh uncached)
            tl = layers[0]
            tm.run("sx_rope_realign", lambda: sx.rope_realign(plan, tl["k_src"], tl["v_src"], tl["kc"], tl["vc"]))
            tm.run("sx_kv_scatter", lambda: sx.kv_scatter(plan, tl["k"], tl["v"], tl["kc"], tl["vc"], rows=nr_rows,
                                                          n_rows=nr_n, max_rows=nr_max))
            sel = tl
        else:
            sel = layers[nfull - 1]
        tm.run("sx_sparseq_score", lambda: sx.sparseq_score(plan, sel["q"], sel["kc"], scores,
                                                            lse_in=lse if (nfull > 0 and args.score_passes == 1)
                                                            else None))
        tm.run("sx_topk_select", lambda: sx.topk_select(plan, scores, ratio, rows, n_rows))
        if (args.kv_write == "per-layer" or args.layer_body) and L > max(nfull, 1):
            tm.run("sx_rows_mask", lambda: sx.rows_mask(plan, rows, n_rows, max_rows, rmask))
        if args.kv_write == "all-layers" and sparse_kv:
            # every sparse layer's cache in one call (two launches of at most 16 layers)
            tm.run("sx_realign_scatter_layers",
                   lambda: sx.realign_scatter_layers(plan, sparse_kv, rows, n_rows, max_rows))
        for l in range(max(nfull, 0), L):
            tl = layers[l]
            if args.layer_body and l >= nfull and not (nfull == 0 and l == 0):
                sparse_layer_body(l, tl)
                continue
            if nfull == 0 and l == 0:
                # the selecting layer's cache is already re-aligned: only R's fresh rows remain
                tm.run("sx_kv_scatter", lambda: sx.kv_scatter(plan, tl["k"], tl["v"], tl["kc"], tl["vc"], rows=rows,
                                                              n_rows=n_rows, max_rows=max_rows))
            elif args.kv_write == "all-layers":
                pass
            elif args.kv_write == "separate":
                tm.run("sx_rope_realign",
                       lambda: sx.rope_realign(plan, tl["k_src"], tl["v_src"], tl["kc"], tl["vc"]))
                tm.run("sx_kv_scatter", lambda: sx.kv_scatter(plan, tl["k"], tl["v"], tl["kc"], tl["vc"], rows=rows,
                                                              n_rows=n_rows, max_rows=max_rows))
            elif args.kv_write == "per-layer":
                # one pass: each slot gets either its fresh row (token in R) or its re-aligned cached row
                tm.run("sx_realign_scatter_masked",
                       lambda: sx.realign_scatter_masked(plan, tl["k_src"], tl["v_src"], tl["k"], tl["v"], rmask,
                                                         tl["kc"], tl["vc"]))
            else:
                tm.run("sx_realign_scatter",
                       lambda: sx.realign_scatter(plan, tl["k_src"], tl["v_src"], tl["k"], tl["v"], rows, n_rows,
                                                  max_rows, tl["kc"], tl["vc"]))
            tm.run("sx_sparse_attn", lambda: sx.sparse_attn(plan, tl["q"], rows, n_rows, max_rows, tl["kc"], tl["vc"],
                                                            out))

    if args.copy_calibration:
        src = torch.empty(args.copy_calibration // 2, dtype=torch.bfloat16, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy calibration: {src.numel() * 2} bytes read, {dst.numel() * 2} bytes written")
        del src, dst
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # the recompute set is a function of the fixed inputs: read it once for the work counts
    offs = w.token_offsets
    R = [rows[offs[r]:offs[r] + int(n_rows[r])].cpu().numpy().astype(np.int64) for r in range(len(w.requests))]

    tm.on = True
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    ms_per_step = elapsed * 1e3 / args.steps
    kern = tm.summary()

    # ---- algorithmic work per launch ----
    def probe_rows(req):
        cached = req.cached_mask()
        last = [sg for sg in req.segments if sg.seq_start <= req.n_tokens - 1 < sg.seq_start + sg.length][0]
        p = ~cached
        if last.cached:
            p[max(last.seq_start, req.n_tokens - 64):] = True
        return np.flatnonzero(p)

    pairs_R = float(sum(np.sum(Rr + 1) for Rr in R))
    pairs_P = float(sum(np.sum(probe_rows(req) + 1) for req in w.requests))
    pairs_full = float(sum(req.n_tokens * (req.n_tokens + 1) / 2 for req in w.requests))
    n_R = int(sum(len(Rr) for Rr in R))
    row_bytes = Hkv * d * esz
    work = {
        "sx_sparse_attn": ("mfma", 4.0 * Hq * d * pairs_R),
        "sx_full_attn": ("mfma", 4.0 * Hq * d * pairs_full),
        "sx_sparseq_score": ("mfma", 2.0 * Hq * d * pairs_P),
        "sx_rope_realign": ("hbm", 4.0 * info["n_reused"] * row_bytes),
        "sx_topk_select": ("latency", 5.0 * T),
    }
    # KV write: all rows in the full layers, R in the sparse layers (and I_nr in a selecting layer)
    n_sparse = L - nfull
    n_sep = n_sparse if args.kv_write == "separate" else (1 if nfull == 0 else 0)   # sparse layers with a separate write
    n_scatter_rows = nfull * T + n_sep * n_R + (info["n_nonreused"] if nfull == 0 else 0)
    n_scatter_launches = nfull + n_sep + (1 if nfull == 0 else 0)
    if n_scatter_launches:
        work["sx_kv_scatter"] = ("hbm", 4.0 * row_bytes * n_scatter_rows / n_scatter_launches)
    # one-pass re-alignment + write: every reused token's slot plus the uncached tokens of R, each
    # read once and written once (K and V)
    n_R_uncached = int(sum(np.count_nonzero(~req.cached_mask()[Rr]) for req, Rr in zip(w.requests, R)))
    work["sx_realign_scatter"] = ("hbm", 4.0 * row_bytes * (info["n_reused"] + n_R_uncached))
    work["sx_realign_scatter_masked"] = work["sx_realign_scatter"]
    work["sx_realign_scatter_layers"] = ("hbm", len(sparse_kv) * work["sx_realign_scatter"][1])
    work["sx_rows_mask"] = ("latency", T + 4.0 * n_R)
    # layer body: matrix products 2 |R| k n, per launch (the q/k/v entry times three launches)
    work["sx_gemm_rows qkv"] = ("mfma", 2.0 * n_R * H * (Hq + 2 * Hkv) * d)
    work["sx_gemm_rows o"] = ("mfma", 2.0 * n_R * Hq * d * H)
    work["sx_gemm_rows gate_up"] = ("mfma", 2.0 * n_R * H * 2 * F)
    work["sx_gemm_rows down"] = ("mfma", 2.0 * n_R * F * H)
    work["sx_rmsnorm_rows"] = ("hbm", 2.0 * n_R * H * esz + H * esz)
    work["sx_rope_rows"] = ("hbm", 4.0 * n_R * (Hq + Hkv) * d * esz)
    work["sx_silu_mul_rows"] = ("hbm", 3.0 * n_R * F * esz)
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    kernels = {}
    for name, k in kern.items():
        kind, amount = work[name]
        sec = k["avg_ms"] / 1e3
        e = {"launches_per_step": k["launches"] // args.steps, "avg_us": round(k["avg_ms"] * 1e3, 2),
             "median_us": round(k["median_ms"] * 1e3, 2), "p10_us": round(k["p10_ms"] * 1e3, 2),
             "p90_us": round(k["p90_ms"] * 1e3, 2),
             "share_of_step": round(k["total_ms"] / args.steps / ms_per_step, 4)}
        if kind == "mfma":
            e["tflops"] = round(amount / sec / 1e12, 2)
            e["frac_of_peak"] = round(amount / sec / 1e12 / peak, 4)
        elif kind == "hbm":
            e["gbps"] = round(amount / sec / 1e9, 1)
            e["frac_of_peak"] = round(amount / sec / 1e9 / PEAK_HBM_GBS, 4)
        kernels[name] = e
    dom = max(kern, key=lambda n: kern[n]["total_ms"])
    kind, amount = work[dom]
    sec = kern[dom]["avg_ms"] / 1e3
    traffic = load_traffic(w.name)
    for name, e in kernels.items():
        if name in traffic:
            e["hbm_bytes_per_launch"] = round(traffic[name])
    if kind == "hbm":
        roof = {"kernel": dom, "bound": "hbm", "achieved": round(amount / sec / 1e9, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(amount / sec / 1e9 / PEAK_HBM_GBS, 4),
                "traffic": round(traffic[dom]) if dom in traffic else None, "algorithmic_per_launch": amount}
    else:
        roof = {"kernel": dom, "bound": "mfma", "achieved": round(amount / sec / 1e12, 2), "peak": peak,
                "unit": "TFLOP/s", "frac": round(amount / sec / 1e12 / peak, 4),
                "traffic": round(traffic[dom]) if dom in traffic else None, "traffic_unit": "HBM bytes per launch",
                "algorithmic_per_launch": amount}

    value = T * L / (ms_per_step / 1e3)
    # per layer kind: a sparse layer's calls (one-pass re-alignment + KV write, sparse attention), a
    # full layer's (KV write of every row, full attention), and the once-per-step selection
    layer_rates = None
    us = {n: kern[n]["avg_ms"] * 1e3 for n in kern}
    if not args.layer_body and "sx_sparse_attn" in us and "sx_full_attn" in us:
        kv_us = us.get("sx_realign_scatter_masked", us.get("sx_realign_scatter", 0.0))
        sp = kv_us + us["sx_sparse_attn"]
        fu = us.get("sx_kv_scatter", 0.0) + us["sx_full_attn"]
        layer_rates = {"sparse_layer_us": round(sp, 1), "sparse_layer_tokens_per_s": round(T / (sp / 1e6), 1),
                       "full_layer_us": round(fu, 1), "full_layer_tokens_per_s": round(T / (fu / 1e6), 1),
                       "selection_us": round(sum(us.get(n, 0.0) for n in ("sx_sparseq_score", "sx_topk_select",
                                                                           "sx_rows_mask")), 1)}
    peaks = None if args.no_peaks else measured_peaks(torch)
    cpu = None
    if not args.no_cpu_baseline and not args.layer_body:
        cpu = cpu_baseline(w, layers, R, nfull, L, ratio, torch)
    res = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": w.dtype, "data": "synthetic (seeded N(0,1) inputs, layout rules of the workload)",
        "config": {"workload": f"{w.name}: {w.description}", "tokens": T, "layers": L, "full_layers": nfull,
                   "ratio": ratio, "recompute_rows": n_R, "k": int(k_total), "q_heads": Hq, "kv_heads": Hkv,
                   "head_dim": d, "requests": len(w.requests), "score_passes": args.score_passes,
                   "kv_write": args.kv_write, "layer_body": bool(args.layer_body), "buffer_sets": nsets,
                   **({"hidden": H, "ffn": F} if args.layer_body else {})},
        "kernels": kernels, "roofline": roof, "cpu_baseline": cpu,
        "layer_rates": layer_rates, "measured_peaks": peaks,
    }
    print(json.dumps(res), flush=True)
    plan.close()


def measured_peaks(torch):
    """Achievable rates on this GPU next to the datasheet peaks: a device copy of 2 GiB (far beyond
    the 256 MB Infinity Cache; read + write bytes) and a bf16 8192^3 matrix product (torch.matmul,
    i.e. hipBLASLt).  Outside the timed steps."""
    src = torch.empty(1 << 30, dtype=torch.bfloat16, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    a = torch.randn((8192, 8192), dtype=torch.float32, device="cuda").to(torch.bfloat16)
    b = torch.randn((8192, 8192), dtype=torch.float32, device="cuda").to(torch.bfloat16)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    dst.copy_(src)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(5):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    copy_gbs = 5 * 2 * src.numel() * 2 / (e0.elapsed_time(e1) / 1e3) / 1e9
    c = a @ b
    torch.cuda.synchronize()
    e0.record()
    for _ in range(10):
        c = a @ b
    e1.record()
    torch.cuda.synchronize()
    gemm_tf = 10 * 2 * 8192 ** 3 / (e0.elapsed_time(e1) / 1e3) / 1e12
    del src, dst, a, b, c
    torch.cuda.empty_cache()
    return {"hbm_copy_gbps": round(copy_gbs, 1), "hbm_copy_frac_of_peak": round(copy_gbs / PEAK_HBM_GBS, 4),
            "bf16_gemm_tflops": round(gemm_tf, 1), "bf16_gemm_frac_of_peak": round(gemm_tf / PEAK_BF16_TFLOPS, 4),
            "copy": "device copy of 2 GiB (read + write bytes)", "gemm": "torch.matmul 8192^3 bf16 (hipBLASLt)"}


def cpu_model() -> str:
    """The host CPU as lscpu reports it: model name, with family / model / stepping and the max clock
    when the model name alone is terse (some virtual machines report only the vendor's product line),
    and /proc/cpuinfo's model name when it says more."""
    import subprocess
    fields = {}
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if ":" in line:
                k, v = line.split(":", 1)
                fields.setdefault(k.strip(), v.strip())
    except (OSError, subprocess.SubprocessError):
        pass
    proc = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                proc = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    name = fields.get("Model name") or proc or "unknown"
    extra = [f"{k.lower()} {fields[k]}" for k in ("CPU family", "Model", "Stepping", "CPU max MHz") if fields.get(k)]
    if proc and proc != name:
        extra.append(f"/proc/cpuinfo: {proc}")
    return name + (f" ({', '.join(extra)})" if extra else "")


def cpu_baseline(w, layers, R, nfull, L, ratio, torch, n_sample=512):
    """The CPU oracle timed on a bounded sample of one step, scaled to the metric.

    Timed on the host for one layer of request 0: the full re-alignment of every reused token, the
    KV writes of R and of every row, the selection (Eq. topk, overflow, tail) over the full score
    vector; and, each on n_sample seeded rows, the sparse attention of rows of R, the Sparse-Q scores
    of probe rows and full attention of rows (the oracle's matrix form).  The sampled parts are
    scaled by the oracle's cost per row (a row's cost is proportional to the keys it sees), the
    request-0 parts by the requests' token counts."""
    import threadpoolctl

    import oracle as O

    rng = np.random.default_rng(0)
    b = w.block_size
    scale = O.softmax_scale(w.head_dim)
    req = w.requests[0]
    T = req.n_tokens
    lay = layers[min(nfull, L - 1)]
    o1 = int(w.token_offsets[1])
    h = {k: lay[k][:o1].float().cpu().numpy() for k in ("q", "k", "v") if k in lay}
    h.update({k: lay[k].float().cpu().numpy() for k in ("k_src", "v_src") if k in lay})
    info = threadpoolctl.threadpool_info()
    threads = max((x.get("num_threads", 1) for x in info), default=1)
    tot_tokens = float(sum(r.n_tokens for r in w.requests))
    share = T / tot_tokens
    kp = np.zeros((w.n_dst_blocks, w.n_kv_heads, b, w.head_dim), np.float32)
    vp = np.zeros_like(kp)
    t = {}
    s0 = time.perf_counter()
    O.realign_request(req, w, h["k_src"], h["v_src"], kp, vp)
    t["realign"] = (time.perf_counter() - s0) / share
    s0 = time.perf_counter()
    O.scatter_rows(req, w, R[0], h["k"], h["v"], kp, vp)
    t["scatter_R"] = (time.perf_counter() - s0) * sum(len(x) for x in R) / max(1, len(R[0]))
    s0 = time.perf_counter()
    O.scatter_rows(req, w, np.arange(T), h["k"], h["v"], kp, vp)
    t["scatter_all"] = (time.perf_counter() - s0) / share
    kt, vt = O.gather_tokens(req, w, kp), O.gather_tokens(req, w, vp)

    def per_key_cost(rows_all, rows_s):
        # the sampled rows' share of the keys every listed row sees
        return float(np.sum(rows_s + 1)) / float(np.sum(rows_all + 1))

    R_all = [np.asarray(x, dtype=np.int64) for x in R]
    samp = np.sort(rng.choice(R_all[0], size=min(n_sample, len(R_all[0])), replace=False))
    s0 = time.perf_counter()
    O.attention_rows(h["q"], kt, vt, samp, scale)
    pairs_R = sum(float(np.sum(x + 1)) for x in R_all)
    t["sparse_attn"] = (time.perf_counter() - s0) * pairs_R / float(np.sum(samp + 1))
    probes_all = [O.probe_positions(r.n_tokens, r.segments) for r in w.requests]
    ps = np.sort(rng.choice(probes_all[0], size=min(n_sample, len(probes_all[0])), replace=False))
    s0 = time.perf_counter()
    sc = O.sparseq_scores(h["q"], kt, ps, scale)
    # the matrix form evaluates every probe row against all T keys of its request
    t["score"] = (time.perf_counter() - s0) * sum(len(p) * r.n_tokens for p, r in zip(probes_all, w.requests)) / (
        len(ps) * T)
    full_sc = np.zeros(T)
    full_sc[:] = sc
    s0 = time.perf_counter()
    O.recompute_set(T, req.segments, full_sc, ratio, b)
    t["topk"] = (time.perf_counter() - s0) / share
    full_rows = np.sort(rng.choice(T, size=min(n_sample, T), replace=False))
    s0 = time.perf_counter()
    O.attention_rows(h["q"], h["k"], h["v"], full_rows, scale)
    pairs_full = sum(r.n_tokens * (r.n_tokens + 1) / 2 for r in w.requests)
    t["full_attn"] = (time.perf_counter() - s0) * pairs_full / float(np.sum(full_rows + 1))
    if nfull > 0:
        t_step = nfull * (t["scatter_all"] + t["full_attn"]) + t["score"] + t["topk"] + (L - nfull) * (
            t["realign"] + t["scatter_R"] + t["sparse_attn"])
    else:
        t_step = t["realign"] + 2 * t["scatter_R"] + t["score"] + t["topk"] + t["sparse_attn"]
    value = w.total_tokens * L / t_step
    return {"value": round(value, 2), "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
            "sample": (f"one layer of request 0: full re-alignment, KV writes of R and of every row, selection over "
                       f"the full score vector; attention of {len(samp)} rows of R, Sparse-Q scores of {len(ps)} "
                       f"probe rows and full attention of {len(full_rows)} rows; sampled parts scaled by the keys "
                       f"each row sees, request-0 parts by token counts, to the whole {L}-layer step"),
            "seconds_estimated_per_step": round(t_step, 2),
            "step_seconds": {k: round(v, 4) for k, v in t.items()}}


if __name__ == "__main__":
    main()
