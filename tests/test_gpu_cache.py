"""The cache manager's schedule drives the GPU re-alignment: a knowledge base prefilled into one
block pool, published and frozen; a later prompt that embeds it at another position is scheduled,
and sx_rope_realign copies the hit blocks into the fresh carrier blocks of the same pool.  The
carriers must hold exactly the oracle's re-aligned keys and the cached values (Virtual Block, Block
Retrieval and Reuse; Section 3.1 for the rotation)."""
import numpy as np
import pytest
import torch

import oracle as O
import oracle.cache as OC
import paper_2606_01751_amd as sx
import paper_2606_01751_amd.cache as N
import workloads as W
from sxgpu import log

pytestmark = pytest.mark.gpu


def test_schedule_drives_gpu_realignment():
    log("[cache -> realign] knowledge base reused at a new position, one shared pool")
    b, Hkv, d, base, nblk = 16, 2, 128, 5e5, 64
    rng = np.random.default_rng(5)
    emb = rng.standard_normal((4000, Hkv, d)).astype(np.float32)
    vals = rng.standard_normal((4000, Hkv, d)).astype(np.float32)
    pool_k = np.zeros((nblk, Hkv, b, d), np.float32)
    pool_v = np.zeros((nblk, Hkv, b, d), np.float32)
    c = N.BlockCache(nblk, b, 0.9)

    def prefill(toks, table):   # what the model's prefill would leave in the carrier blocks
        for t, tok in enumerate(toks):
            pool_k[table[t // b], :, t % b] = O.to_bf16(O.rope_rotate(emb[tok % 4000], t, base, "neox"))
            pool_v[table[t // b], :, t % b] = O.to_bf16(vals[tok % 4000])

    kb = list(range(100, 300))                       # 200 tokens: 13 blocks, the last padded
    toks, spans = c.pad([(kb, True, b"kb")], -1)
    s = c.schedule(toks, spans)
    prefill(toks, s.block_table)
    c.commit(s.req_id, publish=[(st, n, k, True) for st, n, k in spans])
    c.release(s.req_id)
    # the new prompt: 37 tokens of text, the knowledge base (from block 3 on), 50 more tokens
    toks, spans = c.pad([(list(range(3000, 3037)), False, b""), (kb, True, b"kb"),
                         (list(range(3100, 3150)), False, b"")], -1)
    s = c.schedule(toks, spans)
    assert s.n_virtual_hits == 13 and spans[0][0] == 48
    ref = OC.BlockCache(nblk, b, 0.9)   # the oracle takes the same decisions
    r0 = ref.schedule(OC.pad_pieces([(kb, True, b"kb")], b, -1)[0], [(0, 208, b"kb")])
    ref.commit(r0.req_id, publish=[(0, 208, b"kb", True)])
    ref.release(r0.req_id)
    assert N.Schedule(**ref.schedule(toks, spans).__dict__) == s

    segs = [W.Segment(st, n, bool(ca), old, new, ss) for st, n, ca, old, new, ss in s.segments]
    req = W.Request(len(toks), segs, np.array(s.block_table, np.int32), np.array(s.src_block_ids, np.int32),
                    np.zeros(0, np.int64))
    desc = sx.make_desc(8, Hkv, d, "bf16", base, "neox")
    plan = sx.Plan(desc, [req], nblk, nblk)
    dk = torch.from_numpy(pool_k).cuda().to(torch.bfloat16).contiguous()
    dv = torch.from_numpy(pool_v).cuda().to(torch.bfloat16).contiguous()
    sx.rope_realign(plan, dk, dv, dk, dv)            # sources and carriers in the same pool
    torch.cuda.synchronize()
    got_k, got_v = dk.float().cpu().numpy(), dv.float().cpu().numpy()

    class Desc:
        block_size, rope_base, rope_style, dtype = b, base, "neox", "bf16"
    want_k, want_v = pool_k.copy(), pool_v.copy()
    O.realign_request(req, Desc, pool_k, pool_v, want_k, want_v)
    assert np.array_equal(got_k, want_k) and np.array_equal(got_v, want_v)
    # and the carriers hold the keys of the new positions (up to the bf16 rounding of both sides)
    for t in range(48, 248):
        blk, slot = s.block_table[t // b], t % b
        want = O.rope_rotate(emb[toks[t] % 4000], t, base, "neox")
        assert np.abs(got_k[blk, :, slot] - want).max() <= 2e-2 * max(1.0, np.abs(want).max())
    plan.close()
    log("  carriers bit-identical to the oracle's re-alignment")
