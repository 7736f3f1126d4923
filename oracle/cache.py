"""Oracle of the segment-level cache management (Section 4: Frozen Block, Frozen Block Pool, Extra
Keys, Virtual Block, Block Retrieval and Reuse).

Test infrastructure: only tests/ may import this module.  It is a plain, slow, dictionary-and-list
implementation of the block bookkeeping that turns a prompt into the segment table and block
tables of one step; it shares no code with the library's native cache manager.

What the paper fixes, and the readings taken where it does not (each one is listed in the design
notes):
* Block identity for reuse is the virtual hash H(B, e) of the block's token ids B and the extra
  key e (Extra Keys): equal only for the same tokens under the same key, independent of position
  and of the preceding context.  The ordinary prefix portion keeps a chained prefix hash, which
  depends on every earlier block.  H is SHA-256 over a tagged byte encoding (reading): tag "V" or
  "P", then for "P" the parent hash (32 zero bytes for the first block), then the token count and
  the tokens as little-endian 32-bit integers, then the key length and the key bytes.
* Entry padding (Block Retrieval): a reuse segment starts at a block boundary (pad tokens before
  it) and ends on one (pad tokens after it), so its blocks hash the same in every prompt.
* Lookup: native prefix hits over the full blocks before the first reuse segment, stopping at the
  first miss and never covering the block of the last token; virtual hits per block of each reuse
  segment.  A hit becomes a cached segment whose source is the resident block and whose old
  position is where that block's first token was when it was cached; runs of hits whose old
  positions continue merge into one segment.
* Every token gets a fresh carrier block (Virtual Block: reused KV is copied, Key re-aligned, into
  newly allocated ordinary blocks; prefix hits are copied with shift 0 in this reading).
* Lifecycle (Frozen Block): reference counts; a block whose count drops to zero goes to the tail
  of the free queue, keeping its hashes until it is handed out again (from the head), unless it
  is frozen, in which case it stays resident.  A request's blocks are queued in reverse order, so
  its last blocks are reused first.
* Frozen-block pool: blocks published under a key can be frozen, frozen blocks can be deleted; when
  a schedule would take the pool's utilisation (blocks outside the free queue) above the limit,
  idle frozen blocks are deleted, least referenced first (fewest reuse hits, then least recently
  used, then lowest id), and go to the head of the free queue.
"""
from __future__ import annotations

import hashlib
import struct
from dataclasses import dataclass, field

ZERO_HASH = bytes(32)


def _enc_tokens(tokens) -> bytes:
    tokens = [int(t) for t in tokens]
    return struct.pack("<I", len(tokens)) + struct.pack(f"<{len(tokens)}i", *tokens)


def _enc_key(extra: bytes) -> bytes:
    return struct.pack("<I", len(extra)) + bytes(extra)


def virtual_hash(tokens, extra: bytes) -> bytes:
    """H(B, e) of one block (Extra Keys): SHA-256 of "V" | tokens | key."""
    return hashlib.sha256(b"V" + _enc_tokens(tokens) + _enc_key(extra)).digest()


def prefix_hash(parent, tokens, extra: bytes = b"") -> bytes:
    """Chained prefix hash of one block: SHA-256 of "P" | parent | tokens | key."""
    return hashlib.sha256(b"P" + (ZERO_HASH if parent is None else parent) + _enc_tokens(tokens)
                          + _enc_key(extra)).digest()


def pad_pieces(pieces, block_size: int, pad_token: int):
    """Entry padding: pieces is a list of (tokens, reuse, extra_key).  Returns the padded token list
    and the reuse spans (start, length, extra_key); empty reuse pieces give no span."""
    b = block_size
    out: list[int] = []
    spans = []
    for toks, reuse, extra in pieces:
        toks = [int(t) for t in toks]
        if reuse and toks:
            out += [pad_token] * ((-len(out)) % b)
            start = len(out)
            out += toks
            out += [pad_token] * ((-len(out)) % b)
            spans.append((start, len(out) - start, bytes(extra)))
        else:
            out += toks
    return out, spans


class OutOfBlocks(RuntimeError):
    pass


@dataclass
class _Req:
    tokens: list
    block_table: list
    src_blocks: list            # resident blocks read as sources (one reference each until commit)
    committed: bool = False


@dataclass
class Schedule:
    req_id: int
    segments: list              # (seq_start, length, cached, old_pos, new_pos, src_block_start or -1)
    block_table: list
    src_block_ids: list
    n_prefix_hits: int
    n_virtual_hits: int


@dataclass
class BlockCache:
    n_blocks: int
    block_size: int
    limit: float = 0.9
    free: list = field(default_factory=list)
    ref: list = field(default_factory=list)
    frozen: list = field(default_factory=list)
    hits: list = field(default_factory=list)
    last_use: list = field(default_factory=list)
    prefix_of: list = field(default_factory=list)      # the prefix hash a block carries (or None)
    virt_of: list = field(default_factory=list)        # the virtual hashes a block carries
    prefix_index: dict = field(default_factory=dict)   # prefix hash -> block
    virt_index: dict = field(default_factory=dict)     # virtual hash -> (block, old position)
    reqs: dict = field(default_factory=dict)
    next_req: int = 0
    tick: int = 0

    def __post_init__(self):
        n = self.n_blocks
        self.free = list(range(n))
        self.ref = [0] * n
        self.frozen = [False] * n
        self.hits = [0] * n
        self.last_use = [0] * n
        self.prefix_of = [None] * n
        self.virt_of = [[] for _ in range(n)]

    # ---- block state ----
    def _drop_entries(self, blk):
        h = self.prefix_of[blk]
        if h is not None:
            del self.prefix_index[h]
            self.prefix_of[blk] = None
        for vh in self.virt_of[blk]:
            del self.virt_index[vh]
        self.virt_of[blk] = []

    def _take(self, blk):
        """One more reference to a resident block (out of the free queue if it was there)."""
        if self.ref[blk] == 0 and not self.frozen[blk]:
            self.free.remove(blk)
        self.ref[blk] += 1

    def _put(self, blk):
        self.ref[blk] -= 1
        assert self.ref[blk] >= 0
        if self.ref[blk] == 0 and not self.frozen[blk]:
            self.free.append(blk)

    def _idle_frozen(self, exclude=()):
        c = [x for x in range(self.n_blocks) if self.frozen[x] and self.ref[x] == 0 and x not in exclude]
        return sorted(c, key=lambda x: (self.hits[x], self.last_use[x], x))

    def _delete_frozen(self, blk):
        """Removes a frozen block from the pool: its entries go, and it heads the free queue when idle."""
        self.frozen[blk] = False
        self._drop_entries(blk)
        self.hits[blk] = 0
        if self.ref[blk] == 0:
            self.free.insert(0, blk)

    # ---- requests ----
    def schedule(self, tokens, spans=(), prefix_key: bytes = b"") -> Schedule:
        b = self.block_size
        tokens = [int(t) for t in tokens]
        T = len(tokens)
        if T == 0:
            raise ValueError("empty request")
        spans = [(int(s), int(n), bytes(e)) for s, n, e in spans]
        end = 0
        for s, n, _ in spans:
            if s < end or n <= 0 or s % b or n % b or s + n > T:
                raise ValueError("reuse spans must be sorted, disjoint, block aligned and inside the request")
            end = s + n
        nb = -(-T // b)
        hit = {}   # block index in the request -> (resident block, old position)
        # native prefix hits: full blocks before the first reuse span, never the last token's block
        first = spans[0][0] if spans else T
        parent = None
        n_prefix = 0
        for i in range(min(first // b, (T - 1) // b)):
            h = prefix_hash(parent, tokens[i * b:(i + 1) * b], prefix_key)
            blk = self.prefix_index.get(h)
            if blk is None:
                break
            hit[i] = (blk, i * b)
            parent = h
            n_prefix += 1
        # virtual hits per block of each reuse span
        n_virtual = 0
        for s, n, e in spans:
            for i in range(s // b, (s + n) // b):
                ent = self.virt_index.get(virtual_hash(tokens[i * b:(i + 1) * b], e))
                if ent is not None:
                    hit[i] = ent
                    n_virtual += 1
        # feasibility before any change: fresh blocks for every token
        sources = sorted({blk for blk, _ in hit.values()})
        from_free = sum(1 for x in sources if self.ref[x] == 0 and not self.frozen[x])
        if len(self.free) - from_free + len(self._idle_frozen(exclude=sources)) < nb:
            raise OutOfBlocks(f"{nb} blocks needed")
        self.tick += 1
        src_list = []
        for i in sorted(hit):
            blk = hit[i][0]
            self._take(blk)
            src_list.append(blk)
            self.hits[blk] += 1
            self.last_use[blk] = self.tick
        # utilisation limit, then the allocation itself
        while self.n_blocks - len(self.free) + nb > self.limit * self.n_blocks or len(self.free) < nb:
            idle = self._idle_frozen()
            if not idle:
                break
            self._delete_frozen(idle[0])
        table = []
        for _ in range(nb):
            blk = self.free.pop(0)
            self._drop_entries(blk)
            self.hits[blk] = 0
            self.ref[blk] = 1
            self.last_use[blk] = self.tick
            table.append(blk)
        # segment table: runs of misses, runs of hits whose old positions continue
        segs, src_ids = [], []
        i = 0
        while i < nb:
            if i in hit:
                j = i + 1
                while j in hit and hit[j][1] == hit[j - 1][1] + b:
                    j += 1
                segs.append((i * b, (j - i) * b, 1, hit[i][1], i * b, len(src_ids)))
                src_ids += [hit[x][0] for x in range(i, j)]
            else:
                j = i + 1
                while j < nb and j not in hit:
                    j += 1
                segs.append((i * b, min(j * b, T) - i * b, 0, i * b, i * b, -1))
            i = j
        rid = self.next_req
        self.next_req += 1
        self.reqs[rid] = _Req(tokens, table, src_list)
        return Schedule(rid, segs, table, src_ids, n_prefix, n_virtual)

    def commit(self, req_id: int, publish=(), prefix_key: bytes = b"") -> None:
        """After the request's prefill: its sources are released, its full blocks enter the prefix
        index, and the blocks of each published span (start, length, key, freeze) enter the
        virtual index under that key (and the frozen pool when freeze is set).  Hashes already
        resident keep their block."""
        r = self.reqs[req_id]
        if r.committed:
            raise ValueError("request already committed")
        b = self.block_size
        publish = [(int(s), int(n), bytes(e), bool(f)) for s, n, e, f in publish]
        for s, n, _, _ in publish:
            if s < 0 or n <= 0 or s % b or n % b or s + n > len(r.tokens):
                raise ValueError("published spans must be block aligned and inside the request")
        for blk in r.src_blocks:
            self._put(blk)
        r.src_blocks = []
        r.committed = True
        parent = None
        for i in range(len(r.tokens) // b):
            h = prefix_hash(parent, r.tokens[i * b:(i + 1) * b], prefix_key)
            blk = r.block_table[i]
            if h not in self.prefix_index and self.prefix_of[blk] is None:
                self.prefix_index[h] = blk
                self.prefix_of[blk] = h
            parent = h
        for s, n, e, freeze in publish:
            for i in range(s // b, (s + n) // b):
                blk = r.block_table[i]
                vh = virtual_hash(r.tokens[i * b:(i + 1) * b], e)
                if vh not in self.virt_index:
                    self.virt_index[vh] = (blk, i * b)
                    self.virt_of[blk].append(vh)
                if freeze and self.virt_index[vh][0] == blk:
                    self.frozen[blk] = True

    def release(self, req_id: int) -> None:
        """End of the request: its references go, last block first."""
        r = self.reqs.pop(req_id)
        for blk in r.src_blocks:
            self._put(blk)
        for blk in reversed(r.block_table):
            self._put(blk)

    # ---- frozen-block pool ----
    def frozen_add(self, blocks) -> None:
        for blk in blocks:
            if not self.virt_of[blk]:
                raise ValueError(f"block {blk} carries no published entry")
        for blk in blocks:
            if not self.frozen[blk]:
                if self.ref[blk] == 0:
                    self.free.remove(blk)
                self.frozen[blk] = True

    def frozen_delete(self, blocks) -> None:
        if len(set(blocks)) != len(blocks):
            raise ValueError("a block is listed twice")
        for blk in blocks:
            if not self.frozen[blk]:
                raise ValueError(f"block {blk} is not frozen")
        for blk in blocks:
            self._delete_frozen(blk)

    def stats(self) -> dict:
        return {"free": len(self.free), "in_use": sum(1 for x in self.ref if x > 0),
                "frozen": sum(self.frozen), "idle_frozen": len(self._idle_frozen()),
                "prefix_entries": len(self.prefix_index), "virtual_entries": len(self.virt_index),
                "requests": len(self.reqs)}
