"""Helpers of the GPU parity tests: run the library's steps on a workload and bring results back.

Device tensors come from the seeded host generator (workloads.layer_tensors); nothing the
oracle consumes is produced by the library.
"""
from __future__ import annotations

import math
import sys

import numpy as np
import torch

import paper_2606_01751_amd as sx
import workloads as W

CANARY = -7.0


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def tdtype(w):
    return torch.bfloat16 if w.dtype == "bf16" else torch.float32


def desc_of(w):
    return sx.make_desc(w.n_q_heads, w.n_kv_heads, w.head_dim, w.dtype, w.rope_base, w.rope_style)


def dev(x, w):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda").to(tdtype(w)).contiguous()


def host(t):
    return t.detach().float().cpu().numpy()


def pool_shape(w, n_blocks):
    return (n_blocks, w.n_kv_heads, w.block_size, w.head_dim)


def rows_per_request(w, rows_t, n_rows_t):
    """Split a device row list into per-request numpy arrays."""
    rows = rows_t.cpu().numpy()
    n = n_rows_t.cpu().numpy()
    offs = w.token_offsets
    return [rows[offs[r]:offs[r] + n[r]].astype(np.int64) for r in range(len(w.requests))]


class GpuLayer:
    """Device state of one layer of a workload (fresh tensors, source pool, destination cache)."""

    def __init__(self, w, tensors: dict):
        self.w = w
        self.plan = sx.Plan(desc_of(w), w.requests, w.n_dst_blocks, w.n_src_blocks)
        self.t = {k: dev(v, w) for k, v in tensors.items()}
        dt = tdtype(w)
        self.k_cache = torch.full(pool_shape(w, w.n_dst_blocks), CANARY, dtype=dt, device="cuda")
        self.v_cache = torch.full(pool_shape(w, w.n_dst_blocks), CANARY, dtype=dt, device="cuda")
        tot = w.total_tokens
        self.scores = torch.zeros(tot, dtype=torch.float32, device="cuda")
        self.rows = torch.zeros(tot, dtype=torch.int32, device="cuda")
        self.n_rows = torch.zeros(len(w.requests), dtype=torch.int32, device="cuda")
        self.out = torch.zeros((tot, w.n_q_heads, w.head_dim), dtype=dt, device="cuda")

    def realign(self):
        sx.rope_realign(self.plan, self.t["k_src"], self.t["v_src"], self.k_cache, self.v_cache)

    def scatter_nonreused(self):
        rows, n, m = self.plan.nonreused_rows()
        sx.kv_scatter(self.plan, self.t["k"], self.t["v"], self.k_cache, self.v_cache, rows=rows, n_rows=n, max_rows=m)

    def score(self):
        sx.sparseq_score(self.plan, self.t["q"], self.k_cache, self.scores)

    def select(self, ratio):
        sx.topk_select(self.plan, self.scores, ratio, self.rows, self.n_rows)

    def scatter_rows(self, ratio):
        sx.kv_scatter(self.plan, self.t["k"], self.t["v"], self.k_cache, self.v_cache, rows=self.rows,
                      n_rows=self.n_rows, max_rows=self.plan.budget(ratio)[1])

    def attend(self, ratio):
        sx.sparse_attn(self.plan, self.t["q"], self.rows, self.n_rows, self.plan.budget(ratio)[1], self.k_cache,
                       self.v_cache, self.out)

    def run_sparse(self, ratio):
        self.realign()
        self.scatter_nonreused()
        self.score()
        self.select(ratio)
        self.scatter_rows(ratio)
        self.attend(ratio)
        torch.cuda.synchronize()

    def set_rows(self, per_request_rows):
        """Load a row list computed elsewhere (e.g. by the oracle) into the device row list."""
        rows = np.zeros(self.w.total_tokens, dtype=np.int32)
        offs = self.w.token_offsets
        n = np.zeros(len(self.w.requests), dtype=np.int32)
        for r, R in enumerate(per_request_rows):
            rows[offs[r]:offs[r] + len(R)] = R
            n[r] = len(R)
        self.rows.copy_(torch.from_numpy(rows))
        self.n_rows.copy_(torch.from_numpy(n))


def oracle_pool(w):
    return np.full(pool_shape(w, w.n_dst_blocks), CANARY, dtype=np.float32)


def tie_band_ok(gpu_R, ora_R, ora_scores, cand_mask, k, rel=1e-5):
    """Indices of R may differ only where the oracle's score is within rel of its k-th largest
    candidate score (the tie band).  Returns (ok, n_diff, detail)."""
    diff = np.setxor1d(gpu_R, ora_R)
    if len(diff) == 0:
        return True, 0, ""
    if k == 0:
        return False, len(diff), "k = 0 but sets differ"
    cand_scores = np.sort(ora_scores[cand_mask])[::-1]
    s_star = cand_scores[k - 1]
    bad = [int(j) for j in diff if abs(ora_scores[j] - s_star) > rel * abs(s_star)]
    return len(bad) == 0, len(diff), f"s*={s_star!r}, outside band: {bad[:10]}"
