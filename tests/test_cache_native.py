"""The native cache manager (include/sx_cache.h, libsx) against the oracle: every result of seeded
operation sequences (segment tables, block tables, source blocks, hit counts, pool statistics)
must be identical, and the hashes must equal the oracle's byte for byte.  CPU only: the cache
manager is host code."""
import hashlib

import numpy as np
import pytest

import oracle.cache as C
import paper_2606_01751_amd.cache as N
from test_cache_oracle import PAD, run_random_ops

pytestmark = pytest.mark.filterwarnings("ignore")


def test_sha256_matches_hashlib():
    assert N.sha256(b"abc").hex() == "ba7816bf8f01cfea414140de5dae2223b00361a396177a9cb410ff61f20015ad"
    assert N.sha256(b"") == hashlib.sha256(b"").digest()
    rng = np.random.default_rng(0)
    for n in (1, 55, 56, 63, 64, 65, 119, 120, 128, 1000, 4097):   # around the padding boundaries
        data = rng.integers(0, 256, n, dtype=np.uint8).tobytes()
        assert N.sha256(data) == hashlib.sha256(data).digest(), n


def test_block_hashes_match_the_oracle():
    rng = np.random.default_rng(1)
    for _ in range(50):
        toks = rng.integers(-2**31, 2**31, rng.integers(0, 40)).tolist()
        key = rng.integers(0, 256, rng.integers(0, 20), dtype=np.uint8).tobytes()
        assert N.virtual_hash(toks, key) == C.virtual_hash(toks, key)
        parent = None if rng.integers(0, 2) else rng.integers(0, 256, 32, dtype=np.uint8).tobytes()
        assert N.prefix_hash(parent, toks, key) == C.prefix_hash(parent, toks, key)


@pytest.mark.parametrize("seed", range(6))
def test_pad_matches_the_oracle(seed):
    rng = np.random.default_rng(seed)
    b = int(rng.choice([1, 4, 16]))
    pieces = [(rng.integers(0, 1000, rng.integers(0, 50)).tolist(), bool(rng.integers(0, 2)),
               rng.integers(0, 256, rng.integers(0, 6), dtype=np.uint8).tobytes()) for _ in range(10)]
    assert N.pad(pieces, b, PAD) == C.pad_pieces(pieces, b, PAD)
    assert N.pad([], b, PAD) == ([], [])


def _same_state(nat: N.BlockCache, ora: C.BlockCache):
    assert nat.stats() == ora.stats()
    assert nat.free_queue() == ora.free
    for blk in range(ora.n_blocks):
        i = nat.block_info(blk)
        assert (i["ref"], bool(i["frozen"]), i["hits"], i["last_use"], i["n_virtual"], bool(i["has_prefix"])) == \
            (ora.ref[blk], ora.frozen[blk], ora.hits[blk], ora.last_use[blk], len(ora.virt_of[blk]),
             ora.prefix_of[blk] is not None), blk


def test_hand_scenarios_match_the_oracle():
    KB = [100, 101, 102, 103, 104, 105, 106, 107]
    nat, ora = N.BlockCache(8, 4, 0.9), C.BlockCache(8, 4, 0.9)
    for c in (nat, ora):
        toks, spans = C.pad_pieces([(KB, True, b"kb")], 4, PAD)
        s = c.schedule(toks, spans)
        c.commit(s.req_id, publish=[(0, 8, b"kb", True)])
        c.release(s.req_id)
    _same_state(nat, ora)
    toks, spans = C.pad_pieces([([1, 2, 3], False, b""), (KB, True, b"kb"), ([8, 9], False, b"")], 4, PAD)
    for _ in range(3):
        a, b = nat.schedule(toks, spans), ora.schedule(toks, spans)
        assert a == N.Schedule(**b.__dict__)
        _same_state(nat, ora)
        nat.commit(a.req_id)
        ora.commit(b.req_id)
        nat.release(a.req_id)
        ora.release(b.req_id)
        _same_state(nat, ora)


class _Both:
    """Drives the oracle and the native cache with the same calls and compares every result."""

    def __init__(self, n, b, limit):
        self.nat, self.ora = N.BlockCache(n, b, limit), C.BlockCache(n, b, limit)
        self.block_size, self.n_blocks = b, n

    def pad(self, pieces, pad):
        got = self.nat.pad(pieces, pad)
        assert got == C.pad_pieces(pieces, self.block_size, pad)
        return got

    def block_info(self, blk):
        return self.nat.block_info(blk)

    def schedule(self, toks, spans):
        try:
            b = self.ora.schedule(toks, spans)
        except C.OutOfBlocks:
            with pytest.raises(N.CacheFull):
                self.nat.schedule(toks, spans)
            _same_state(self.nat, self.ora)
            raise
        a = self.nat.schedule(toks, spans)
        assert a == N.Schedule(**b.__dict__)
        return a

    def commit(self, rid, publish=()):
        self.nat.commit(rid, publish)
        self.ora.commit(rid, publish)

    def release(self, rid):
        self.nat.release(rid)
        self.ora.release(rid)

    def frozen_delete(self, blocks):
        self.nat.frozen_delete(blocks)
        self.ora.frozen_delete(blocks)

    def stats(self):
        s = self.nat.stats()
        assert s == self.ora.stats()
        return s


@pytest.mark.parametrize("seed,n,b,limit", [(0, 48, 8, 0.8), (1, 48, 8, 0.8), (2, 24, 4, 0.9), (3, 64, 16, 1.0),
                                            (4, 16, 8, 0.5), (5, 96, 8, 0.9)])
def test_random_sequences_match_the_oracle(seed, n, b, limit):
    both = _Both(n, b, limit)
    log = run_random_ops(both, seed, n_ops=150, on_step=lambda c: _same_state(c.nat, c.ora))
    assert any(e[0] == "sched" and e[6] > 0 for e in log)


def test_errors_leave_the_state_unchanged():
    c = N.BlockCache(8, 4, 0.9)
    s = c.schedule(list(range(8)), [(0, 8, b"k")])
    before = (c.stats(), c.free_queue())
    for bad in ([(2, 4, b"k")], [(0, 12, b"k")], [(4, 4, b"k"), (0, 4, b"k")], [(0, 0, b"k")]):
        with pytest.raises(N.SxError) as e:
            c.schedule(list(range(8)), bad)
        assert e.value.status == -1
    with pytest.raises(N.SxError):
        c.schedule([], [])
    with pytest.raises(N.CacheFull):
        c.schedule(list(range(40)))
    with pytest.raises(N.SxError):
        c.commit(s.req_id, publish=[(0, 6, b"k", True)])
    with pytest.raises(N.SxError):
        c.frozen_add([s.block_table[0]])          # nothing published
    with pytest.raises(N.SxError):
        c.frozen_delete([0])                      # not frozen
    with pytest.raises(N.SxError):
        c.release(12345)
    assert (c.stats(), c.free_queue()) == before
    c.commit(s.req_id, publish=[(0, 8, b"k", True)])
    with pytest.raises(N.SxError):
        c.commit(s.req_id)                        # twice
    with pytest.raises(N.SxError):
        c.frozen_delete([0, 0])                   # listed twice
    c.release(s.req_id)
    assert c.stats()["idle_frozen"] == 2
    with pytest.raises(ValueError):
        c.schedule([2**31])                        # token ids are int32
    with pytest.raises(N.SxError):
        N.BlockCache(0, 4)
    with pytest.raises(N.SxError):
        N.BlockCache(8, 4, 1.5)


def test_schedule_output_builds_a_plan():
    """The schedule is directly an sx_request: the plan validates it (block ids in range, tiling,
    cached segments block aligned in their sources)."""
    import paper_2606_01751_amd as sx
    import workloads as W
    c = N.BlockCache(32, 16, 0.9)
    kb = list(range(1000, 1100))
    toks, spans = c.pad([(kb, True, b"kb")], PAD)
    s = c.schedule(toks, spans)
    c.commit(s.req_id, publish=[(st, n, k, True) for st, n, k in spans])
    c.release(s.req_id)
    toks, spans = c.pad([(list(range(7)), False, b""), (kb, True, b"kb"), (list(range(30)), False, b"")], PAD)
    s = c.schedule(toks, spans)
    assert s.n_virtual_hits == 7 and any(g[2] for g in s.segments)
    segs = [W.Segment(st, n, bool(ca), old, new, ss) for st, n, ca, old, new, ss in s.segments]
    req = W.Request(len(toks), segs, np.array(s.block_table, np.int32), np.array(s.src_block_ids, np.int32),
                    np.zeros(0, np.int64))
    desc = sx.make_desc(8, 2, 128, "bf16", 5e5, "neox")
    import torch
    if torch.cuda.is_available():
        sx.Plan(desc, [req], 32, 32).close()      # one pool serves as source and destination
    else:
        with pytest.raises(sx.SxError) as e:      # host validation passed; only the device is missing
            sx.Plan(desc, [req], 32, 32)
        assert e.value.status in (sx.SX_ENOMEM, sx.SX_EHIP), str(e.value)
