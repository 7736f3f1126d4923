"""Pins of the cache-management oracle (Section 4: Frozen Block, Frozen Block Pool, Extra Keys,
Virtual Block, Block Retrieval and Reuse) against what the paper and the definitions fix:
hand-worked lifecycles with every block id derived by hand from the stated policy, hash
properties (namespace isolation, position and context independence, chaining), padding
properties, invariants over random operation sequences, a brute-force lookup, and an end-to-end
check that the produced segment table re-aligns cached keys to their new positions.  A last test
plants mistakes in the oracle and checks that a pin notices each."""

import numpy as np
import pytest

import oracle as O
import oracle.cache as C
import workloads as W

PAD = -1


# ---------------------------------------------------------------------------------------------
# hashes and padding
# ---------------------------------------------------------------------------------------------
def test_sha256_and_encoding_pins():
    import hashlib
    # FIPS 180-2 example: SHA-256("abc")
    assert hashlib.sha256(b"abc").hexdigest() == \
        "ba7816bf8f01cfea414140de5dae2223b00361a396177a9cb410ff61f20015ad"
    # the byte encoding, assembled by hand: tag, token count, tokens (little-endian int32), key
    msg = b"V" + bytes([2, 0, 0, 0]) + bytes([1, 0, 0, 0]) + bytes([0xFF, 0xFF, 0xFF, 0xFF]) + bytes([2, 0, 0, 0]) + b"kb"
    assert C.virtual_hash([1, -1], b"kb") == hashlib.sha256(msg).digest()
    parent = bytes(range(32))
    msg = b"P" + parent + bytes([1, 0, 0, 0]) + bytes([7, 1, 0, 0]) + bytes([0, 0, 0, 0])
    assert C.prefix_hash(parent, [263], b"") == hashlib.sha256(msg).digest()
    assert C.prefix_hash(None, [263]) == C.prefix_hash(bytes(32), [263])


def test_hash_namespaces_and_chaining():
    rng = np.random.default_rng(0)
    blk = rng.integers(0, 50000, 16)
    other = blk.copy()
    other[7] += 1
    # same tokens and key -> same hash; another key or another token -> another hash
    assert C.virtual_hash(blk, b"kb1") == C.virtual_hash(blk.copy(), b"kb1")
    assert C.virtual_hash(blk, b"kb1") != C.virtual_hash(blk, b"kb2")
    assert C.virtual_hash(blk, b"kb1") != C.virtual_hash(other, b"kb1")
    assert C.virtual_hash(blk, b"") != C.virtual_hash(blk, b"\x00")   # the key length is encoded
    # prefix and virtual namespaces never meet; a prefix hash depends on every earlier block
    assert C.prefix_hash(None, blk) != C.virtual_hash(blk, b"")
    h0 = C.prefix_hash(None, blk)
    h0b = C.prefix_hash(None, other)
    assert C.prefix_hash(h0, blk) != C.prefix_hash(h0b, blk)
    assert C.prefix_hash(h0, blk, b"salt") != C.prefix_hash(h0, blk)


def test_pad_pieces_hand_example():
    toks, spans = C.pad_pieces([([1, 2, 3], False, b""), ([5, 6], True, b"k"), ([7], False, b"")], 4, PAD)
    assert toks == [1, 2, 3, PAD, 5, 6, PAD, PAD, 7]
    assert spans == [(4, 4, b"k")]
    # aligned pieces need no padding; an empty reuse piece gives no span
    toks, spans = C.pad_pieces([([1, 2, 3, 4], False, b""), ([5, 6, 7, 8], True, b"k"), ([], True, b"k")], 4, PAD)
    assert toks == [1, 2, 3, 4, 5, 6, 7, 8] and spans == [(4, 4, b"k")]


@pytest.mark.parametrize("seed", range(5))
def test_pad_pieces_properties(seed):
    rng = np.random.default_rng(seed)
    b = 16
    pieces = [(list(rng.integers(0, 1000, rng.integers(0, 60))), bool(rng.integers(0, 2)), bytes([seed, i]))
              for i in range(12)]
    toks, spans = C.pad_pieces(pieces, b, PAD)
    # removing the pad tokens gives back the pieces in order
    assert [t for t in toks if t != PAD] == [t for p in pieces for t in p[0]]
    reuse = [p for p in pieces if p[1] and p[0]]
    assert len(spans) == len(reuse)
    for (s, n, e), p in zip(spans, reuse):
        assert s % b == 0 and n % b == 0 and n - len(p[0]) < b and e == p[2]
        assert toks[s:s + len(p[0])] == p[0] and all(t == PAD for t in toks[s + len(p[0]):s + n])
    # fewer than b pad tokens at every boundary
    assert len(toks) - sum(len(p[0]) for p in pieces) < 2 * b * len(reuse) + 1


# ---------------------------------------------------------------------------------------------
# hand-worked lifecycles (n = 8 blocks of 4 tokens; every expected id derived from the policy)
# ---------------------------------------------------------------------------------------------
KB = [100, 101, 102, 103, 104, 105, 106, 107]


def test_knowledge_base_then_two_requests():
    c = C.BlockCache(8, 4, limit=0.9)
    # knowledge-base prefill: two blocks from the head of the free queue, published and frozen
    toks, spans = C.pad_pieces([(KB, True, b"kb")], 4, PAD)
    s = c.schedule(toks, spans)
    assert s.block_table == [0, 1] and s.src_block_ids == [] and s.n_virtual_hits == 0
    assert s.segments == [(0, 8, 0, 0, 0, -1)]
    c.commit(s.req_id, publish=[(0, 8, b"kb", True)])
    c.release(s.req_id)
    assert c.free == [2, 3, 4, 5, 6, 7] and c.frozen[:2] == [True, True]
    assert c.stats()["idle_frozen"] == 2 and c.stats()["virtual_entries"] == 2 and c.stats()["prefix_entries"] == 2

    # request B: 3 question tokens, the knowledge base (padded to block 1), 2 more tokens
    toks, spans = C.pad_pieces([([1, 2, 3], False, b""), (KB, True, b"kb"), ([8, 9], False, b"")], 4, PAD)
    assert toks == [1, 2, 3, PAD] + KB + [8, 9] and spans == [(4, 8, b"kb")]
    s = c.schedule(toks, spans)
    assert s.block_table == [2, 3, 4, 5] and s.src_block_ids == [0, 1]
    assert s.segments == [(0, 4, 0, 0, 0, -1), (4, 8, 1, 0, 4, 0), (12, 2, 0, 12, 12, -1)]
    assert (s.n_prefix_hits, s.n_virtual_hits) == (0, 2)
    assert c.ref[:6] == [1, 1, 1, 1, 1, 1] and c.hits[:2] == [1, 1]
    c.commit(s.req_id)          # sources released (frozen: they stay resident); 3 full blocks indexed
    assert c.ref[:2] == [0, 0] and c.stats()["prefix_entries"] == 5
    c.release(s.req_id)         # last block first
    assert c.free == [6, 7, 5, 4, 3, 2]

    # request C = B: block 0 is a prefix hit (B's block 2), the knowledge base two virtual hits whose
    # old positions do not continue the prefix hit's (0, then 0 again), so three segments
    s = c.schedule(toks, spans)
    assert (s.n_prefix_hits, s.n_virtual_hits) == (1, 2)
    assert s.src_block_ids == [2, 0, 1]
    assert s.segments == [(0, 4, 1, 0, 0, 0), (4, 8, 1, 0, 4, 1), (12, 2, 0, 12, 12, -1)]
    assert s.block_table == [6, 7, 5, 4] and c.free == [3]
    # block 4 held B's third full block: handing it out dropped that prefix entry
    assert c.stats()["prefix_entries"] == 4
    c.release(s.req_id)         # never committed: sources and blocks go together
    assert c.free == [3, 2, 4, 5, 7, 6] and c.ref == [0] * 8


def test_frozen_pool_deletes_least_referenced_first():
    c = C.BlockCache(8, 4, limit=0.75)
    blocks = {}
    for key, toks in ((b"k1", [1, 2, 3, 4]), (b"k2", [5, 6, 7, 8]), (b"k3", [9, 10, 11, 12])):
        s = c.schedule(toks, [(0, 4, key)])
        c.commit(s.req_id, publish=[(0, 4, key, True)])
        c.release(s.req_id)
        blocks[key] = s.block_table[0]
    assert blocks == {b"k1": 0, b"k2": 1, b"k3": 2}
    # k2 is reused twice, k3 once (the reuse block is the first of a 2-block request)
    for key, toks, times in ((b"k2", [5, 6, 7, 8], 2), (b"k3", [9, 10, 11, 12], 1)):
        for _ in range(times):
            s = c.schedule(toks + [0], [(0, 4, key)])
            assert s.src_block_ids == [blocks[key]]
            c.commit(s.req_id)
            c.release(s.req_id)
    assert c.hits[:3] == [0, 2, 1]
    # 3 resident + 3 new blocks = 6 <= 0.75 * 8: nothing deleted
    s = c.schedule(list(range(20, 32)))
    assert c.stats()["frozen"] == 3
    c.release(s.req_id)
    # 3 resident + 4 new = 7 > 6: the least referenced frozen block (k1, no hit) goes first
    s = c.schedule(list(range(40, 56)))
    assert c.frozen[:3] == [False, True, True] and c.stats()["virtual_entries"] == 2
    assert s.block_table[0] == 0      # the deleted block heads the free queue
    c.release(s.req_id)
    # 2 resident + 6 new = 8 > 6: both remaining go, k3 (1 hit) before k2 (2 hits)
    s = c.schedule(list(range(60, 84)))
    assert s.block_table[:2] == [1, 2] and c.stats()["frozen"] == 0
    c.release(s.req_id)


def test_frozen_add_and_delete_and_out_of_blocks():
    c = C.BlockCache(4, 4, limit=1.0)
    s = c.schedule([1, 2, 3, 4, 5, 6, 7, 8], [(0, 8, b"u")])
    with pytest.raises(ValueError):
        c.frozen_add([s.block_table[0]])      # nothing published yet
    c.commit(s.req_id, publish=[(0, 8, b"u", False)])
    c.release(s.req_id)
    assert c.free == [2, 3, 1, 0]
    c.frozen_add([0])                          # pinned: out of the free queue
    assert c.free == [2, 3, 1] and c.frozen[0]
    with pytest.raises(C.OutOfBlocks):
        c.schedule(list(range(100, 120)))      # 5 blocks; 3 free + 1 idle frozen
    assert c.free == [2, 3, 1] and c.frozen[0]   # a refused schedule changes nothing
    # 4 blocks: the idle frozen block is deleted to make room, and is handed out first
    s = c.schedule(list(range(100, 116)))
    assert s.block_table == [0, 2, 3, 1] and not c.frozen[0]
    c.release(s.req_id)
    with pytest.raises(ValueError):
        c.frozen_delete([0])


# ---------------------------------------------------------------------------------------------
# random operation sequences: invariants and a brute-force lookup
# ---------------------------------------------------------------------------------------------
def check_invariants(c: C.BlockCache):
    n = c.n_blocks
    assert len(set(c.free)) == len(c.free)
    holders = [0] * n
    for r in c.reqs.values():
        for blk in r.block_table:
            holders[blk] += 1
        for blk in r.src_blocks:
            holders[blk] += 1
    assert holders == c.ref
    for blk in range(n):
        in_free = blk in c.free
        assert in_free == (c.ref[blk] == 0 and not c.frozen[blk])
    for h, blk in c.prefix_index.items():
        assert c.prefix_of[blk] == h
    for blk, h in enumerate(c.prefix_of):
        assert h is None or c.prefix_index[h] == blk
    for vh, (blk, pos) in c.virt_index.items():
        assert vh in c.virt_of[blk] and pos % c.block_size == 0
    assert sum(len(v) for v in c.virt_of) == len(c.virt_index)
    for blk in range(n):
        if c.frozen[blk]:
            assert c.virt_of[blk], "a frozen block carries a published entry"


def random_prompt(rng, kbs, users, b):
    pieces = []
    for _ in range(rng.integers(1, 5)):
        kind = rng.integers(0, 3)
        if kind == 0:
            pieces.append((list(rng.integers(0, 30, rng.integers(1, 3 * b))), False, b""))
        elif kind == 1 and kbs:
            key, text = kbs[rng.integers(0, len(kbs))]
            lo = rng.integers(0, len(text) // b) * b
            pieces.append((text[lo:lo + rng.integers(1, len(text) - lo + 1)], True, key))
        elif users:
            key, text = users[rng.integers(0, len(users))]
            pieces.append((text, True, key))
    return pieces


def run_random_ops(cache, seed, n_ops=120, on_step=None):
    """A seeded mix of knowledge-base builds, user requests (published under their key or not),
    frozen-pool edits and releases.  Returns the log of every result (for comparing two caches)."""
    rng = np.random.default_rng(seed)
    b = cache.block_size
    kbs = [(b"kb%d" % i, list(rng.integers(0, 40, rng.integers(b, 5 * b)))) for i in range(3)]
    users = [(b"user%d" % i, list(rng.integers(0, 40, rng.integers(1, 3 * b)))) for i in range(3)]
    live = []
    log = []
    for step in range(n_ops):
        op = rng.integers(0, 10)
        if op <= 5 or not live:
            if op == 0:
                key, text = kbs[rng.integers(0, len(kbs))]
                pieces, publish_all, freeze = [(text, True, key)], True, True
            else:
                pieces = random_prompt(rng, kbs, users, b)
                publish_all, freeze = bool(rng.integers(0, 2)), False
            toks, spans = cache_pad(cache, pieces, b)
            try:
                s = cache.schedule(toks, spans)
            except Exception as e:   # out of blocks
                log.append(("oob", type(e).__name__))
                continue
            log.append(("sched", s.req_id, s.segments, s.block_table, s.src_block_ids, s.n_prefix_hits,
                        s.n_virtual_hits))
            if rng.integers(0, 4):
                pub = [(st, n, e, freeze) for st, n, e in spans] if publish_all else []
                cache.commit(s.req_id, publish=pub)
            live.append(s.req_id)
        elif op <= 8:
            rid = live.pop(rng.integers(0, len(live)))
            cache.release(rid)
            log.append(("rel", rid))
        else:
            frozen = [x for x in range(cache.n_blocks) if cache_is_frozen(cache, x)]
            if frozen and rng.integers(0, 2):
                blk = frozen[rng.integers(0, len(frozen))]
                cache.frozen_delete([blk])
                log.append(("fdel", blk))
        log.append(("stats", cache_stats(cache)))
        if on_step:
            on_step(cache)
    return log


def cache_pad(cache, pieces, b):
    return C.pad_pieces(pieces, b, PAD) if isinstance(cache, C.BlockCache) else cache.pad(pieces, PAD)


def cache_is_frozen(cache, blk):
    return cache.frozen[blk] if isinstance(cache, C.BlockCache) else bool(cache.block_info(blk)["frozen"])


def cache_stats(cache):
    return cache.stats()


@pytest.mark.parametrize("seed", range(6))
def test_random_operations_keep_the_invariants(seed):
    c = C.BlockCache(48, 8, limit=0.8)
    log = run_random_ops(c, seed, on_step=check_invariants)
    assert any(e[0] == "sched" and e[6] > 0 for e in log), "the sequence should reuse something"


@pytest.mark.parametrize("seed", range(4))
def test_virtual_hits_match_a_brute_force_search(seed):
    """Independently of the hashes: a reuse block hits iff a resident block holds an entry for the
    same tokens under the same key, found by comparing token lists, and the hit names that block and
    its old position.  Entries are created by publication (the first block published with given
    tokens and key holds it) and end when the block is handed out again or deleted."""
    b = 8
    c = C.BlockCache(64, b, limit=0.9)
    entries = {}   # block -> [(tokens, key, old position)]

    def holder(key):
        return [(blk, pos) for blk, ents in entries.items() for t, k, pos in ents if (t, k) == key]

    class Spy:
        block_size, n_blocks = b, 64

        def pad(self, pieces, pad):
            return C.pad_pieces(pieces, b, pad)

        def block_info(self, blk):
            return {"frozen": c.frozen[blk]}

        def schedule(self, toks, spans):
            expect = {}
            for st, n, e in spans:
                for i in range(st // b, (st + n) // b):
                    expect[i] = holder((tuple(toks[i * b:(i + 1) * b]), e))
            s = c.schedule(toks, spans)
            got = {}
            for seq_start, length, cached, old, new, sstart in s.segments:
                if cached:
                    for j in range(length // b):
                        got[seq_start // b + j] = (s.src_block_ids[sstart + j], old + j * b)
            for i, cands in expect.items():
                assert len(cands) <= 1
                assert got.get(i) == (cands[0] if cands else None), (i, got.get(i), cands)
            for blk in s.block_table:
                entries.pop(blk, None)
            return s

        def commit(self, rid, publish=()):
            r = c.reqs[rid]
            for st, n, e, _ in publish:
                for i in range(st // b, (st + n) // b):
                    key = (tuple(r.tokens[i * b:(i + 1) * b]), e)
                    if not holder(key):
                        entries.setdefault(r.block_table[i], []).append(key + (i * b,))
            c.commit(rid, publish)

        def release(self, rid):
            c.release(rid)

        def frozen_delete(self, blocks):
            for blk in blocks:
                entries.pop(blk, None)
            c.frozen_delete(blocks)

        def stats(self):
            return c.stats()

    log = run_random_ops(Spy(), 100 + seed)
    assert any(e[0] == "sched" and e[6] > 0 for e in log)


# ---------------------------------------------------------------------------------------------
# end to end: the produced segment table re-aligns cached keys to their new positions
# ---------------------------------------------------------------------------------------------
def test_schedule_drives_realignment_to_new_positions():
    b, d, Hkv, base = 4, 8, 1, 1e4
    c = C.BlockCache(16, b, limit=1.0)
    rng = np.random.default_rng(7)
    emb = rng.standard_normal((200, Hkv, d)).astype(np.float32)   # a token's unrotated key
    pool = np.zeros((16, Hkv, b, d), np.float32)

    def prefill(toks, table):
        for t, tok in enumerate(toks):
            pool[table[t // b], :, t % b, :] = O.rope_rotate(emb[tok], t, base, "neox")

    kb = list(range(10, 22))
    toks, spans = C.pad_pieces([(kb, True, b"kb")], b, PAD)
    s = c.schedule(toks, spans)
    prefill([t % 200 for t in toks], s.block_table)
    c.commit(s.req_id, publish=[(0, 12, b"kb", True)])
    c.release(s.req_id)
    # the knowledge base now sits at position 8 (after 6 question tokens and 2 pads)
    toks, spans = C.pad_pieces([(list(range(50, 56)), False, b""), (kb, True, b"kb")], b, PAD)
    s = c.schedule(toks, spans)
    assert spans == [(8, 12, b"kb")] and s.n_virtual_hits == 3
    segs = [W.Segment(st, n, bool(ca), old, new, ss) for st, n, ca, old, new, ss in s.segments]
    req = W.Request(len(toks), segs, np.array(s.block_table, np.int32), np.array(s.src_block_ids, np.int32),
                    np.zeros(0, np.int64))

    class Desc:
        block_size, rope_base, rope_style, dtype = b, base, "neox", "f32"
    dst_k = np.zeros_like(pool)
    dst_v = np.zeros_like(pool)
    O.realign_request(req, Desc, pool, pool, dst_k, dst_v)
    for t in range(8, 20):
        want = O.rope_rotate(emb[toks[t] % 200], t, base, "neox")
        got = dst_k[s.block_table[t // b], :, t % b, :]
        np.testing.assert_allclose(got, want, atol=2e-5)


# ---------------------------------------------------------------------------------------------
# planted mistakes
# ---------------------------------------------------------------------------------------------
def _bad_vhash_ignores_key(tokens, extra):
    return C.hashlib.sha256(b"V" + C._enc_tokens(tokens)).digest()


def _bad_pad_no_trailing(pieces, block_size, pad_token):
    out, spans = [], []
    for toks, reuse, extra in pieces:
        toks = [int(t) for t in toks]
        if reuse and toks:
            out += [pad_token] * ((-len(out)) % block_size)
            spans.append((len(out), len(toks), bytes(extra)))
        out += toks
    return out, spans


_orig_release = C.BlockCache.release
_orig_idle = C.BlockCache._idle_frozen
_orig_schedule = C.BlockCache.schedule


def _bad_release_forward(self, req_id):
    r = self.reqs.pop(req_id)
    for blk in r.src_blocks:
        self._put(blk)
    for blk in r.block_table:
        self._put(blk)


def _bad_idle_most_referenced(self, exclude=()):
    return list(reversed(_orig_idle(self, exclude)))


def _bad_schedule_old_pos(self, tokens, spans=(), prefix_key=b""):
    s = _orig_schedule(self, tokens, spans, prefix_key)
    s.segments = [(a, n, ca, old + (self.block_size if ca else 0), new, ss) for a, n, ca, old, new, ss in s.segments]
    return s


MISTAKES = [
    ("virtual hash ignores the key", "virtual_hash", _bad_vhash_ignores_key,
     [test_sha256_and_encoding_pins, test_hash_namespaces_and_chaining]),
    ("no trailing padding", "pad_pieces", _bad_pad_no_trailing,
     [test_pad_pieces_hand_example, lambda: test_pad_pieces_properties(0)]),
    ("blocks freed first to last", ("BlockCache", "release"), _bad_release_forward,
     [test_knowledge_base_then_two_requests]),
    ("most referenced frozen block deleted first", ("BlockCache", "_idle_frozen"), _bad_idle_most_referenced,
     [test_frozen_pool_deletes_least_referenced_first]),
    ("old position off by a block", ("BlockCache", "schedule"), _bad_schedule_old_pos,
     [test_schedule_drives_realignment_to_new_positions, test_knowledge_base_then_two_requests]),
]


@pytest.mark.parametrize("name,target,bad,checks", MISTAKES, ids=[m[0] for m in MISTAKES])
def test_planted_cache_mistake_fails_a_pin(monkeypatch, name, target, bad, checks):
    if isinstance(target, tuple):
        monkeypatch.setattr(getattr(C, target[0]), target[1], bad)
    else:
        monkeypatch.setattr(C, target, bad)
    failed = False
    for fn in checks:
        try:
            fn()
        except Exception:
            failed = True
            break
    assert failed, f"no pin notices the planted mistake: {name}"
