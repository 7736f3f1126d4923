/* libsx segment-level cache management: the host-side block bookkeeping that produces the
 * segment tables and block tables of include/sx.h (Section 4 of the paper: Frozen Block, Frozen
 * Block Pool, Extra Keys, Virtual Block, Block Retrieval and Reuse).
 *
 * Host code only: no call touches the GPU.  The cache keeps the state of one physical KV block
 * pool of n_blocks blocks of block_size tokens (the pool the KV tensors live in; a request's
 * re-alignment copies from blocks of this pool into fresh blocks of the same pool, so the same
 * buffer serves as sx_plan_create's source and destination pool).
 *
 *   Virtual hash of a block B with extra key e: SHA-256 of the byte string
 *     "V" | u32 len(B) | B as little-endian int32 | u32 len(e) | e
 *   Prefix hash (the ordinary prefix cache, chained over the blocks of a prompt):
 *     "P" | parent (32 bytes; zeros for the first block) | u32 len(B) | B | u32 len(e) | e
 *   where e is the request's prefix key (empty by default).
 *
 * Policy (all of it deterministic, so two runs of the same call sequence give the same ids):
 *   - sx_cache_schedule looks up the prompt: chained prefix hits over the full blocks before the
 *     first reuse span (stopping at the first miss, never covering the block of the last token),
 *     then a virtual-hash lookup of every block of every reuse span.  Each hit block gets one
 *     reference (its KV is read by the re-alignment), and every block of the prompt gets a fresh
 *     carrier block from the head of the free queue; a block handed out loses its hashes.
 *     Hits become cached segments (source = the resident block, old_pos = where its first token
 *     was cached, new_pos = seq_start); consecutive hits whose old positions continue share a
 *     segment; everything else is uncached.
 *   - Before allocating, if (blocks outside the free queue + the new blocks) would exceed
 *     limit * n_blocks, or the free queue is short, idle frozen blocks are deleted, least
 *     referenced first: fewest reuse hits, then least recently used, then lowest id.  A deleted
 *     block loses its hashes and heads the free queue.
 *   - A block whose reference count drops to zero joins the tail of the free queue and keeps its
 *     hashes (it can still be hit) until it is handed out again -- unless it is frozen: then it
 *     stays resident.  A request's blocks are released last block first.
 *
 * Ownership: the cache owns its state; pointers passed in are read during the call only.  One
 * cache must not be used by two threads at once.  Errors as in sx.h (negative status, message in
 * sx_last_error); a call that fails changes nothing.
 */
#ifndef SX_CACHE_H
#define SX_CACHE_H

#include "sx.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct sx_cache sx_cache;

/* One piece of a prompt before padding (Block Retrieval and Reuse: the entry layer aligns reuse
 * segments to the block size).  extra_key is read only for reuse pieces. */
typedef struct sx_piece {
  const int32_t* tokens;
  int32_t n_tokens;           /* >= 0 */
  int32_t reuse;              /* 1: a reuse segment under extra_key; 0: ordinary text */
  const uint8_t* extra_key;   /* may be NULL when extra_key_len == 0 */
  int32_t extra_key_len;
} sx_piece;

/* A block-aligned span of a padded prompt with its extra key (Extra Keys).  As a lookup span
 * (sx_cache_schedule) freeze is ignored; as a published span (sx_cache_commit) freeze = 1 puts its
 * blocks in the frozen-block pool. */
typedef struct sx_span {
  int32_t start;              /* multiple of block_size */
  int32_t length;             /* > 0, multiple of block_size */
  const uint8_t* extra_key;
  int32_t extra_key_len;
  int32_t freeze;
} sx_span;

/* Entry padding: concatenates the pieces, inserting pad_token before each non-empty reuse piece up
 * to a block boundary and after it up to the next one, so every reuse span starts and ends on a
 * block boundary.  Writes the padded prompt to tokens_out (capacity entries) and one span per
 * non-empty reuse piece to spans_out (span_capacity entries; extra_key points at the piece's key,
 * freeze = 0).  *n_tokens / *n_spans receive the sizes; with tokens_out == NULL only the sizes are
 * computed.  SX_EINVAL if a capacity is too small. */
sx_status sx_cache_pad(int32_t block_size, const sx_piece* pieces, int32_t n_pieces, int32_t pad_token,
                       int32_t* tokens_out, int32_t capacity, int32_t* n_tokens, sx_span* spans_out,
                       int32_t span_capacity, int32_t* n_spans);

/* The hashes above, and plain SHA-256 (FIPS 180-4), into out[32].  parent may be NULL (first
 * block). */
sx_status sx_sha256(const uint8_t* data, int64_t n, uint8_t* out);
sx_status sx_cache_virtual_hash(const int32_t* tokens, int32_t n, const uint8_t* key, int32_t key_len, uint8_t* out);
sx_status sx_cache_prefix_hash(const uint8_t* parent, const int32_t* tokens, int32_t n, const uint8_t* key,
                               int32_t key_len, uint8_t* out);

/* A cache over n_blocks >= 1 blocks of block_size >= 1 tokens, all initially free (queue order
 * 0, 1, ...); limit in (0, 1] is the utilisation above which idle frozen blocks are deleted (the
 * paper's example: 0.9). */
sx_status sx_cache_create(int32_t n_blocks, int32_t block_size, double limit, sx_cache** out);
sx_status sx_cache_destroy(sx_cache* cache);   /* NULL is allowed */

typedef struct sx_cache_schedule_info {
  int32_t request_id;         /* handle for commit / release */
  int32_t n_segments;
  int32_t n_blocks;           /* ceil(n_tokens / block_size) entries of block_table */
  int32_t n_src_blocks;       /* entries of src_block_ids */
  int32_t n_prefix_hits;      /* blocks found by the prefix hash */
  int32_t n_virtual_hits;     /* blocks found by the virtual hash */
} sx_cache_schedule_info;

/* Block Retrieval and Reuse for one padded prompt: lookup, reference taking, carrier allocation.
 * spans: the prompt's reuse spans (sorted, disjoint, block aligned, inside the prompt).
 * segments, block_table and src_block_ids each need ceil(n_tokens / block_size) entries; together
 * with n_tokens they form the sx_request of this prompt (segments tile the prompt, cached
 * segments start at slot 0 of their first source block, src_block_start = -1 when uncached).
 * SX_EFULL (nothing changed) if the pool cannot supply the carrier blocks even after deleting
 * every idle frozen block. */
sx_status sx_cache_schedule(sx_cache* cache, const int32_t* tokens, int32_t n_tokens, const sx_span* spans,
                            int32_t n_spans, const uint8_t* prefix_key, int32_t prefix_key_len,
                            sx_segment* segments, int32_t* block_table, int32_t* src_block_ids,
                            sx_cache_schedule_info* info);

/* After the request's prefill (its carrier blocks hold its KV): releases the references on its
 * source blocks, enters its full blocks into the prefix index (chained under prefix_key) and the
 * blocks of every published span into the virtual index under the span's key (Virtual Block),
 * freezing them when the span says so (Frozen Block).  A hash already present keeps its block.
 * At most once per request. */
sx_status sx_cache_commit(sx_cache* cache, int32_t request_id, const sx_span* publish, int32_t n_publish,
                          const uint8_t* prefix_key, int32_t prefix_key_len);

/* End of a request: releases its source references (if not committed) and its carrier blocks. */
sx_status sx_cache_release(sx_cache* cache, int32_t request_id);

/* Frozen-block pool edits (the paper's insert / delete APIs).  Add: blocks that carry a published
 * virtual entry become frozen (an idle one leaves the free queue).  Delete: frozen blocks lose
 * their hashes and leave the pool; an idle one heads the free queue.  Every id must be valid (and,
 * for delete, frozen and listed once) or nothing changes. */
sx_status sx_cache_frozen_add(sx_cache* cache, const int32_t* blocks, int32_t n);
sx_status sx_cache_frozen_delete(sx_cache* cache, const int32_t* blocks, int32_t n);

typedef struct sx_cache_stats {
  int32_t free;               /* blocks in the free queue */
  int32_t in_use;             /* blocks with references */
  int32_t frozen;
  int32_t idle_frozen;        /* frozen without references */
  int32_t prefix_entries;
  int32_t virtual_entries;
  int32_t requests;           /* scheduled and not released */
} sx_cache_stats;

typedef struct sx_cache_block {
  int32_t ref;
  int32_t frozen;
  int32_t in_free_queue;
  int32_t n_virtual;          /* virtual entries the block carries */
  int32_t has_prefix;
  int64_t hits;               /* reuse hits since the block was last handed out */
  int64_t last_use;           /* schedule call that last used it */
} sx_cache_block;

sx_status sx_cache_get_stats(const sx_cache* cache, sx_cache_stats* out);
sx_status sx_cache_get_block(const sx_cache* cache, int32_t block, sx_cache_block* out);
/* The free queue from head to tail into out (capacity entries); *n receives its length. */
sx_status sx_cache_free_queue(const sx_cache* cache, int32_t* out, int32_t capacity, int32_t* n);

#ifdef __cplusplus
}
#endif

#endif /* SX_CACHE_H */
