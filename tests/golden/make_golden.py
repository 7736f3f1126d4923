"""Writes the oracle's Sparse-Q scores and recompute sets for the full-size workloads.

Calls only the CPU oracle and the seeded input generator; nothing here touches the GPU.  The
GPU tests regenerate the same inputs from the same seeds and compare against these files.

    python tests/golden/make_golden.py [c3] [c4] [c5]

c3: the boundary selection of the 32-layer chat stack (layer 3's queries and fresh keys of every
    token, Algorithm 1 steps 11-17).
c4: the selecting layer of the agent workload (mixed keys: re-aligned cached keys and fresh
    uncached keys, Section 3.1-3.2), at every recompute ratio of the workload.
c5: two requests of the serving batch -- request 4 (16592 tokens, ends uncached) and request 7
    (41392 tokens, ends cached, so the tail fallback probes) -- in both modes the batch runs:
    "mixed", the selecting layer on layer 4's inputs (re-aligned cached keys, fresh uncached keys);
    "fresh", the boundary selection of the hybrid stack on layer 3's queries and fresh keys.  Inputs
    of these requests come from workloads.request_tensors (the GPU tests overlay them on a batch
    drawn on the device).  Scores are stored as float32 (the comparisons use relative 1e-4 and 1e-5).
"""
import hashlib
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle as O  # noqa: E402
import workloads as W  # noqa: E402


def layout_hash(w) -> str:
    h = hashlib.sha256()
    for r in w.requests:
        for s in r.segments:
            h.update(np.array([s.seq_start, s.length, int(s.cached), s.old_pos, s.new_pos, s.src_block_start],
                              dtype=np.int64).tobytes())
        h.update(np.asarray(r.block_table, dtype=np.int64).tobytes())
        h.update(np.asarray(r.src_block_ids, dtype=np.int64).tobytes())
    return h.hexdigest()[:16]


def c3():
    w = W.config(3)
    req = w.requests[0]
    layer = w.n_full_layers - 1
    t0 = time.time()
    t = W.layer_tensors(w, layer)
    print(f"c3: inputs of layer {layer} in {time.time() - t0:.1f}s", flush=True)
    t0 = time.time()
    s = O.sparseq_scores(t["q"], t["k"], O.probe_positions(req.n_tokens, req.segments),
                         O.softmax_scale(w.head_dim))
    print(f"c3: scores in {time.time() - t0:.1f}s", flush=True)
    sets = O.recompute_set(req.n_tokens, req.segments, s, 0.15, w.block_size)
    np.savez_compressed(os.path.join(HERE, "c3_boundary.npz"), scores=s, R=sets["R"], k=sets["k"], layer=layer,
                        layout=layout_hash(w))


def c4():
    w = W.config(4)
    req = w.requests[0]
    t0 = time.time()
    t = W.layer_tensors(w, 0)
    print(f"c4: inputs in {time.time() - t0:.1f}s", flush=True)
    kp = np.zeros((w.n_dst_blocks, w.n_kv_heads, w.block_size, w.head_dim), np.float32)
    vp = np.zeros_like(kp)
    O.realign_request(req, w, t["k_src"], t["v_src"], kp, vp)
    O.scatter_rows(req, w, O.nonreuse_positions(req.n_tokens, req.segments), t["k"], t["v"], kp, vp)
    t0 = time.time()
    s = O.sparseq_scores(t["q"], O.gather_tokens(req, w, kp), O.probe_positions(req.n_tokens, req.segments),
                         O.softmax_scale(w.head_dim))
    print(f"c4: scores in {time.time() - t0:.1f}s", flush=True)
    out = {"scores": s, "layout": layout_hash(w)}
    for r in w.ratios:
        sets = O.recompute_set(req.n_tokens, req.segments, s, r, w.block_size)
        out[f"R_{int(round(r * 100))}"] = sets["R"]
    np.savez_compressed(os.path.join(HERE, "c4_layer.npz"), **out)


C5_REQUESTS = (4, 7)
C5_LAYERS = {"mixed": 4, "fresh": 3}


def c5():
    w = W.config(5)
    out = {"layout": layout_hash(w)}
    scale = O.softmax_scale(w.head_dim)
    for mode, layer in C5_LAYERS.items():
        for r in C5_REQUESTS:
            req = w.requests[r]
            T = req.n_tokens
            rt = W.request_tensors(w, layer, r)
            if mode == "mixed":
                ks, vs = W.request_pools(w, r, rt)
                kp = np.zeros((w.n_dst_blocks, w.n_kv_heads, w.block_size, w.head_dim), np.float32)
                vp = np.zeros_like(kp)
                O.realign_request(req, w, ks, vs, kp, vp)
                O.scatter_rows(req, w, O.nonreuse_positions(T, req.segments), rt["k"], rt["v"], kp, vp)
                keys = O.gather_tokens(req, w, kp)
                del ks, vs, kp, vp
            else:
                keys = rt["k"]
            t0 = time.time()
            s = O.sparseq_scores(rt["q"], keys, O.probe_positions(T, req.segments), scale)
            print(f"c5 {mode} request {r}: scores in {time.time() - t0:.1f}s", flush=True)
            sets = O.recompute_set(T, req.segments, s, 0.15, w.block_size)
            out[f"{mode}_{r}_scores"] = s.astype(np.float32)
            out[f"{mode}_{r}_R"] = sets["R"].astype(np.int32)
            out[f"{mode}_{r}_k"] = sets["k"]
    np.savez_compressed(os.path.join(HERE, "c5_requests.npz"), **out)


if __name__ == "__main__":
    which = sys.argv[1:] or ["c3", "c4", "c5"]
    for name in which:
        {"c3": c3, "c4": c4, "c5": c5}[name]()
