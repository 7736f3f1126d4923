// Segment-level cache management (Section 4: Frozen Block, Frozen Block Pool, Extra Keys, Virtual
// Block, Block Retrieval and Reuse): host-side block bookkeeping that turns a padded prompt into
// the segment table and block tables of include/sx.h.  The policy is stated in include/sx_cache.h.
//
// Data structures, sized for pools of up to millions of blocks:
//   free queue        intrusive doubly linked list over block ids (O(1) take / put / pop)
//   idle frozen set   ordered set of (hits, last use, id) of frozen blocks without references:
//                     its first element is the block the pool deletes next
//   prefix / virtual  hash maps from the 32-byte SHA-256 digest to the block (and, for virtual
//   indexes          entries, the position of the block's first token when it was cached); every
//                     block lists the digests it carries, so handing it out drops them
#include <algorithm>
#include <array>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <set>
#include <string>
#include <tuple>
#include <unordered_map>
#include <vector>

#include "sx_cache.h"
#include "sx_internal.h"

namespace {

sx_status cfail(sx_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  return sx::report(st, buf);
}

// ---------------------------------------------------------------------------------------------
// SHA-256 (FIPS 180-4).  The round constants are the first 32 bits of the fractional parts of the
// cube roots of the first 64 primes, the initial state those of the square roots of the first 8;
// both are computed here from that definition with exact integer roots.
// ---------------------------------------------------------------------------------------------
typedef unsigned __int128 u128;

struct ShaConst {
  uint32_t k[64];
  uint32_t h0[8];
  ShaConst() {
    int found = 0;
    for (uint32_t p = 2; found < 64; ++p) {
      bool prime = true;
      for (uint32_t q = 2; q * q <= p; ++q)
        if (p % q == 0) {
          prime = false;
          break;
        }
      if (!prime) continue;
      // floor(cbrt(p) * 2^32) = floor(cbrt(p * 2^96)); its low 32 bits are the fraction's
      const u128 n3 = (u128)p << 96;
      uint64_t lo = 0, hi = 1ull << 36;
      while (hi - lo > 1) {
        const uint64_t m = (lo + hi) / 2;
        if ((u128)m * m * m <= n3) lo = m;
        else hi = m;
      }
      k[found] = (uint32_t)lo;
      if (found < 8) {
        const u128 n2 = (u128)p << 64;
        uint64_t a = 0, b = 1ull << 36;
        while (b - a > 1) {
          const uint64_t m = (a + b) / 2;
          if ((u128)m * m <= n2) a = m;
          else b = m;
        }
        h0[found] = (uint32_t)a;
      }
      ++found;
    }
  }
};

const ShaConst& sha_const() {
  static const ShaConst c;
  return c;
}

inline uint32_t rotr(uint32_t x, int n) { return (x >> n) | (x << (32 - n)); }

struct Sha256 {
  uint32_t h[8];
  uint8_t buf[64];
  uint64_t len = 0;   // bytes absorbed
  int fill = 0;

  Sha256() { std::memcpy(h, sha_const().h0, sizeof(h)); }

  void block(const uint8_t* m) {
    const uint32_t* K = sha_const().k;
    uint32_t w[64];
    for (int t = 0; t < 16; ++t)
      w[t] = (uint32_t)m[4 * t] << 24 | (uint32_t)m[4 * t + 1] << 16 | (uint32_t)m[4 * t + 2] << 8 | m[4 * t + 3];
    for (int t = 16; t < 64; ++t) {
      const uint32_t s0 = rotr(w[t - 15], 7) ^ rotr(w[t - 15], 18) ^ (w[t - 15] >> 3);
      const uint32_t s1 = rotr(w[t - 2], 17) ^ rotr(w[t - 2], 19) ^ (w[t - 2] >> 10);
      w[t] = w[t - 16] + s0 + w[t - 7] + s1;
    }
    uint32_t a = h[0], b = h[1], c = h[2], d = h[3], e = h[4], f = h[5], g = h[6], hh = h[7];
    for (int t = 0; t < 64; ++t) {
      const uint32_t S1 = rotr(e, 6) ^ rotr(e, 11) ^ rotr(e, 25);
      const uint32_t ch = (e & f) ^ (~e & g);
      const uint32_t t1 = hh + S1 + ch + K[t] + w[t];
      const uint32_t S0 = rotr(a, 2) ^ rotr(a, 13) ^ rotr(a, 22);
      const uint32_t maj = (a & b) ^ (a & c) ^ (b & c);
      const uint32_t t2 = S0 + maj;
      hh = g;
      g = f;
      f = e;
      e = d + t1;
      d = c;
      c = b;
      b = a;
      a = t1 + t2;
    }
    h[0] += a;
    h[1] += b;
    h[2] += c;
    h[3] += d;
    h[4] += e;
    h[5] += f;
    h[6] += g;
    h[7] += hh;
  }

  void update(const void* data, size_t n) {
    const uint8_t* p = (const uint8_t*)data;
    len += n;
    if (fill == 0)
      for (; n >= 64; n -= 64, p += 64) block(p);
    while (n > 0) {
      const size_t take = std::min(n, (size_t)(64 - fill));
      std::memcpy(buf + fill, p, take);
      fill += (int)take;
      p += take;
      n -= take;
      if (fill == 64) {
        block(buf);
        fill = 0;
      }
    }
  }

  void final(uint8_t* out) {
    const uint64_t bits = len * 8;
    const uint8_t one = 0x80, zero = 0;
    update(&one, 1);
    while (fill != 56) update(&zero, 1);
    uint8_t l[8];
    for (int i = 0; i < 8; ++i) l[i] = (uint8_t)(bits >> (56 - 8 * i));
    update(l, 8);
    for (int i = 0; i < 8; ++i) {
      out[4 * i] = (uint8_t)(h[i] >> 24);
      out[4 * i + 1] = (uint8_t)(h[i] >> 16);
      out[4 * i + 2] = (uint8_t)(h[i] >> 8);
      out[4 * i + 3] = (uint8_t)h[i];
    }
  }
};

typedef std::array<uint8_t, 32> Digest;

struct DigestHash {
  size_t operator()(const Digest& d) const {
    uint64_t v;
    std::memcpy(&v, d.data(), 8);   // a SHA-256 digest is uniformly distributed already
    return (size_t)v;
  }
};

// The encoded message of a block hash: tag [| parent] | u32 n | n little-endian int32 | u32 key
// length | key, assembled in one buffer and hashed with one update.
Digest block_hash(uint8_t tag, const uint8_t* parent, const int32_t* t, int32_t n, const uint8_t* key,
                  int32_t key_len) {
  static const uint8_t zero[32] = {};
  thread_local std::vector<uint8_t> msg;
  const size_t len = 1 + (tag == 'P' ? 32 : 0) + 4 + 4 * (size_t)n + 4 + (size_t)key_len;
  if (msg.size() < len) msg.resize(len);
  uint8_t* p = msg.data();
  auto put32 = [&](uint32_t v) {
    p[0] = (uint8_t)v;
    p[1] = (uint8_t)(v >> 8);
    p[2] = (uint8_t)(v >> 16);
    p[3] = (uint8_t)(v >> 24);
    p += 4;
  };
  *p++ = tag;
  if (tag == 'P') {
    std::memcpy(p, parent ? parent : zero, 32);
    p += 32;
  }
  put32((uint32_t)n);
  for (int32_t i = 0; i < n; ++i) put32((uint32_t)t[i]);
  put32((uint32_t)key_len);
  if (key_len > 0) std::memcpy(p, key, (size_t)key_len);
  Sha256 s;
  s.update(msg.data(), len);
  Digest d;
  s.final(d.data());
  return d;
}

Digest virtual_hash(const int32_t* t, int32_t n, const uint8_t* key, int32_t key_len) {
  return block_hash('V', nullptr, t, n, key, key_len);
}

Digest prefix_hash(const uint8_t* parent, const int32_t* t, int32_t n, const uint8_t* key, int32_t key_len) {
  return block_hash('P', parent, t, n, key, key_len);
}

}  // namespace

// ---------------------------------------------------------------------------------------------
// The cache
// ---------------------------------------------------------------------------------------------
struct sx_cache {
  int32_t n = 0, b = 0;
  double limit = 0.9;
  // per block
  std::vector<int32_t> ref, prev, next;
  std::vector<uint8_t> frozen, in_free, has_prefix;
  std::vector<int64_t> hits, last_use;
  std::vector<Digest> prefix_of;
  std::vector<std::vector<Digest>> virt_of;
  // free queue
  int32_t head = -1, tail = -1, n_free = 0;
  // idle frozen blocks, deletion order
  std::set<std::tuple<int64_t, int64_t, int32_t>> idle;
  std::unordered_map<Digest, int32_t, DigestHash> prefix_index;
  struct VEnt {
    int32_t block, pos;
  };
  std::unordered_map<Digest, VEnt, DigestHash> virt_index;
  struct Req {
    std::vector<int32_t> tokens, table, src;
    bool committed = false;
  };
  std::unordered_map<int32_t, Req> reqs;
  int32_t next_req = 0;
  int64_t tick = 0;

  // ---- free queue ----
  void q_remove(int32_t x) {
    if (prev[x] >= 0) next[prev[x]] = next[x];
    else head = next[x];
    if (next[x] >= 0) prev[next[x]] = prev[x];
    else tail = prev[x];
    prev[x] = next[x] = -1;
    in_free[x] = 0;
    --n_free;
  }
  void q_push_back(int32_t x) {
    prev[x] = tail;
    next[x] = -1;
    if (tail >= 0) next[tail] = x;
    else head = x;
    tail = x;
    in_free[x] = 1;
    ++n_free;
  }
  void q_push_front(int32_t x) {
    next[x] = head;
    prev[x] = -1;
    if (head >= 0) prev[head] = x;
    else tail = x;
    head = x;
    in_free[x] = 1;
    ++n_free;
  }

  // ---- block state ----
  std::tuple<int64_t, int64_t, int32_t> idle_key(int32_t x) const { return {hits[x], last_use[x], x}; }

  void drop_entries(int32_t x) {
    if (has_prefix[x]) {
      prefix_index.erase(prefix_of[x]);
      has_prefix[x] = 0;
    }
    for (const Digest& d : virt_of[x]) virt_index.erase(d);
    virt_of[x].clear();
  }
  void take(int32_t x) {   // one more reference to a resident block
    if (ref[x] == 0) {
      if (frozen[x]) idle.erase(idle_key(x));
      else q_remove(x);
    }
    ++ref[x];
  }
  void put(int32_t x) {
    --ref[x];
    if (ref[x] == 0) {
      if (frozen[x]) idle.insert(idle_key(x));
      else q_push_back(x);
    }
  }
  void delete_frozen(int32_t x) {
    if (ref[x] == 0) idle.erase(idle_key(x));
    frozen[x] = 0;
    drop_entries(x);
    hits[x] = 0;
    if (ref[x] == 0) q_push_front(x);
  }
};

extern "C" {

sx_status sx_sha256(const uint8_t* data, int64_t n, uint8_t* out) {
  if ((!data && n > 0) || n < 0 || !out) return cfail(SX_EINVAL, "sx_sha256: bad arguments");
  Sha256 s;
  if (n > 0) s.update(data, (size_t)n);
  s.final(out);
  return SX_OK;
}

sx_status sx_cache_virtual_hash(const int32_t* tokens, int32_t n, const uint8_t* key, int32_t key_len, uint8_t* out) {
  if ((!tokens && n > 0) || n < 0 || (!key && key_len > 0) || key_len < 0 || !out)
    return cfail(SX_EINVAL, "sx_cache_virtual_hash: bad arguments");
  const Digest d = virtual_hash(tokens, n, key, key_len);
  std::memcpy(out, d.data(), 32);
  return SX_OK;
}

sx_status sx_cache_prefix_hash(const uint8_t* parent, const int32_t* tokens, int32_t n, const uint8_t* key,
                               int32_t key_len, uint8_t* out) {
  if ((!tokens && n > 0) || n < 0 || (!key && key_len > 0) || key_len < 0 || !out)
    return cfail(SX_EINVAL, "sx_cache_prefix_hash: bad arguments");
  const Digest d = prefix_hash(parent, tokens, n, key, key_len);
  std::memcpy(out, d.data(), 32);
  return SX_OK;
}

sx_status sx_cache_pad(int32_t block_size, const sx_piece* pieces, int32_t n_pieces, int32_t pad_token,
                       int32_t* tokens_out, int32_t capacity, int32_t* n_tokens, sx_span* spans_out,
                       int32_t span_capacity, int32_t* n_spans) {
  if (block_size < 1 || n_pieces < 0 || (!pieces && n_pieces > 0) || !n_tokens || !n_spans)
    return cfail(SX_EINVAL, "sx_cache_pad: bad arguments");
  const int64_t b = block_size;
  int64_t len = 0, ns = 0;
  for (int32_t i = 0; i < n_pieces; ++i) {   // sizes first: nothing is written on failure
    const sx_piece& p = pieces[i];
    if (p.n_tokens < 0 || (!p.tokens && p.n_tokens > 0) || (p.reuse && p.extra_key_len < 0) ||
        (p.reuse && !p.extra_key && p.extra_key_len > 0))
      return cfail(SX_EINVAL, "sx_cache_pad: piece %d is malformed", i);
    if (p.reuse && p.n_tokens > 0) {
      len = (len + b - 1) / b * b + (p.n_tokens + b - 1) / b * b;
      ++ns;
    } else {
      len += p.n_tokens;
    }
    if (len > INT32_MAX) return cfail(SX_EINVAL, "sx_cache_pad: padded prompt longer than 2^31 tokens");
  }
  *n_tokens = (int32_t)len;
  *n_spans = (int32_t)ns;
  if (!tokens_out) return SX_OK;
  if (capacity < len || (ns > 0 && (!spans_out || span_capacity < ns)))
    return cfail(SX_EINVAL, "sx_cache_pad: output capacity %d tokens / %d spans, need %lld / %lld", capacity,
                 span_capacity, (long long)len, (long long)ns);
  int64_t o = 0, si = 0;
  for (int32_t i = 0; i < n_pieces; ++i) {
    const sx_piece& p = pieces[i];
    const bool span = p.reuse && p.n_tokens > 0;
    if (span)
      while (o % b) tokens_out[o++] = pad_token;
    const int64_t start = o;
    if (p.n_tokens > 0) std::memcpy(tokens_out + o, p.tokens, sizeof(int32_t) * (size_t)p.n_tokens);
    o += p.n_tokens;
    if (span) {
      while (o % b) tokens_out[o++] = pad_token;
      spans_out[si++] = sx_span{(int32_t)start, (int32_t)(o - start), p.extra_key, p.extra_key_len, 0};
    }
  }
  return SX_OK;
}

sx_status sx_cache_create(int32_t n_blocks, int32_t block_size, double limit, sx_cache** out) {
  if (!out) return cfail(SX_EINVAL, "out is NULL");
  if (n_blocks < 1 || block_size < 1) return cfail(SX_EINVAL, "n_blocks and block_size must be >= 1");
  if (!(limit > 0.0 && limit <= 1.0)) return cfail(SX_EINVAL, "limit must be in (0, 1]");
  sx_cache* c = new (std::nothrow) sx_cache();
  if (!c) return cfail(SX_ENOMEM, "host allocation failed");
  try {
    c->n = n_blocks;
    c->b = block_size;
    c->limit = limit;
    const size_t n = (size_t)n_blocks;
    c->ref.assign(n, 0);
    c->prev.assign(n, -1);
    c->next.assign(n, -1);
    c->frozen.assign(n, 0);
    c->in_free.assign(n, 0);
    c->has_prefix.assign(n, 0);
    c->hits.assign(n, 0);
    c->last_use.assign(n, 0);
    c->prefix_of.resize(n);
    c->virt_of.resize(n);
  } catch (...) {
    delete c;
    return cfail(SX_ENOMEM, "host allocation failed");
  }
  for (int32_t x = 0; x < n_blocks; ++x) c->q_push_back(x);
  *out = c;
  return SX_OK;
}

sx_status sx_cache_destroy(sx_cache* cache) {
  delete cache;
  return SX_OK;
}

namespace {
sx_status check_spans(const sx_cache* c, const sx_span* spans, int32_t n_spans, int64_t T, bool sorted,
                      const char* what) {
  if (n_spans < 0 || (!spans && n_spans > 0)) return cfail(SX_EINVAL, "%s: bad span array", what);
  int64_t end = 0;
  for (int32_t i = 0; i < n_spans; ++i) {
    const sx_span& s = spans[i];
    if (s.start < 0 || s.length <= 0 || s.start % c->b || s.length % c->b || (int64_t)s.start + s.length > T ||
        (sorted && s.start < end) || s.extra_key_len < 0 || (!s.extra_key && s.extra_key_len > 0))
      return cfail(SX_EINVAL, "%s: span %d (start %d, length %d) is not %sblock aligned inside the prompt", what, i,
                   s.start, s.length, sorted ? "sorted, disjoint, " : "");
    end = (int64_t)s.start + s.length;
  }
  return SX_OK;
}
}  // namespace

sx_status sx_cache_schedule(sx_cache* c, const int32_t* tokens, int32_t n_tokens, const sx_span* spans,
                            int32_t n_spans, const uint8_t* prefix_key, int32_t prefix_key_len,
                            sx_segment* segments, int32_t* block_table, int32_t* src_block_ids,
                            sx_cache_schedule_info* info) {
  if (!c || !tokens || !segments || !block_table || !src_block_ids || !info)
    return cfail(SX_EINVAL, "sx_cache_schedule: NULL argument");
  if (n_tokens <= 0) return cfail(SX_EINVAL, "sx_cache_schedule: empty prompt");
  if (prefix_key_len < 0 || (!prefix_key && prefix_key_len > 0))
    return cfail(SX_EINVAL, "sx_cache_schedule: bad prefix key");
  sx_status st = check_spans(c, spans, n_spans, n_tokens, true, "sx_cache_schedule");
  if (st != SX_OK) return st;
  const int32_t b = c->b, T = n_tokens;
  const int32_t nb = (int32_t)(((int64_t)T + b - 1) / b);
  std::vector<int32_t> hit_blk((size_t)nb, -1), hit_pos((size_t)nb, 0);
  // native prefix hits: full blocks before the first reuse span, never the last token's block
  const int32_t first = n_spans > 0 ? spans[0].start : T;
  const int32_t n_pref = std::min(first / b, (T - 1) / b);
  int32_t n_prefix = 0, n_virtual = 0;
  Digest parent{};
  for (int32_t i = 0; i < n_pref; ++i) {
    const Digest h = prefix_hash(i ? parent.data() : nullptr, tokens + (int64_t)i * b, b, prefix_key, prefix_key_len);
    auto it = c->prefix_index.find(h);
    if (it == c->prefix_index.end()) break;
    hit_blk[i] = it->second;
    hit_pos[i] = i * b;
    parent = h;
    ++n_prefix;
  }
  // virtual hits per block of each reuse span
  for (int32_t s = 0; s < n_spans; ++s)
    for (int32_t i = spans[s].start / b; i < (spans[s].start + spans[s].length) / b; ++i) {
      auto it = c->virt_index.find(virtual_hash(tokens + (int64_t)i * b, b, spans[s].extra_key, spans[s].extra_key_len));
      if (it != c->virt_index.end()) {
        hit_blk[i] = it->second.block;
        hit_pos[i] = it->second.pos;
        ++n_virtual;
      }
    }
  // feasibility before any change
  std::vector<int32_t> sources;
  for (int32_t i = 0; i < nb; ++i)
    if (hit_blk[i] >= 0) sources.push_back(hit_blk[i]);
  std::sort(sources.begin(), sources.end());
  sources.erase(std::unique(sources.begin(), sources.end()), sources.end());
  int64_t from_free = 0, idle_sources = 0;
  for (int32_t x : sources) {
    if (c->ref[x] == 0 && !c->frozen[x]) ++from_free;
    if (c->ref[x] == 0 && c->frozen[x]) ++idle_sources;
  }
  if ((int64_t)c->n_free - from_free + ((int64_t)c->idle.size() - idle_sources) < nb)
    return cfail(SX_EFULL, "sx_cache_schedule: %d blocks needed, the pool cannot supply them", nb);
  ++c->tick;
  std::vector<int32_t> src_list;
  for (int32_t i = 0; i < nb; ++i) {
    const int32_t x = hit_blk[i];
    if (x < 0) continue;
    c->take(x);
    src_list.push_back(x);
    ++c->hits[x];
    c->last_use[x] = c->tick;
  }
  // utilisation limit and a short free queue: delete idle frozen blocks, least referenced first
  while (((double)(c->n - c->n_free + nb) > c->limit * (double)c->n || c->n_free < nb) && !c->idle.empty())
    c->delete_frozen(std::get<2>(*c->idle.begin()));
  for (int32_t i = 0; i < nb; ++i) {
    const int32_t x = c->head;
    c->q_remove(x);
    c->drop_entries(x);
    c->hits[x] = 0;
    c->ref[x] = 1;
    c->last_use[x] = c->tick;
    block_table[i] = x;
  }
  // segment table: runs of misses, and runs of hits whose old positions continue
  int32_t n_seg = 0, n_src = 0;
  for (int32_t i = 0; i < nb;) {
    int32_t j = i + 1;
    sx_segment& g = segments[n_seg++];
    g.seq_start = i * b;
    g.new_pos = i * b;
    if (hit_blk[i] >= 0) {
      while (j < nb && hit_blk[j] >= 0 && hit_pos[j] == hit_pos[j - 1] + b) ++j;
      g.length = (j - i) * b;
      g.cached = 1;
      g.old_pos = hit_pos[i];
      g.src_block_start = n_src;
      for (int32_t x = i; x < j; ++x) src_block_ids[n_src++] = hit_blk[x];
    } else {
      while (j < nb && hit_blk[j] < 0) ++j;
      g.length = std::min((int64_t)j * b, (int64_t)T) - (int64_t)i * b;
      g.cached = 0;
      g.old_pos = i * b;
      g.src_block_start = -1;
    }
    i = j;
  }
  const int32_t rid = c->next_req++;
  sx_cache::Req& r = c->reqs[rid];
  r.tokens.assign(tokens, tokens + T);
  r.table.assign(block_table, block_table + nb);
  r.src = std::move(src_list);
  info->request_id = rid;
  info->n_segments = n_seg;
  info->n_blocks = nb;
  info->n_src_blocks = n_src;
  info->n_prefix_hits = n_prefix;
  info->n_virtual_hits = n_virtual;
  return SX_OK;
}

sx_status sx_cache_commit(sx_cache* c, int32_t request_id, const sx_span* publish, int32_t n_publish,
                          const uint8_t* prefix_key, int32_t prefix_key_len) {
  if (!c) return cfail(SX_EINVAL, "cache is NULL");
  auto it = c->reqs.find(request_id);
  if (it == c->reqs.end()) return cfail(SX_EINVAL, "sx_cache_commit: no request %d", request_id);
  sx_cache::Req& r = it->second;
  if (r.committed) return cfail(SX_EINVAL, "sx_cache_commit: request %d already committed", request_id);
  if (prefix_key_len < 0 || (!prefix_key && prefix_key_len > 0))
    return cfail(SX_EINVAL, "sx_cache_commit: bad prefix key");
  sx_status st = check_spans(c, publish, n_publish, (int64_t)r.tokens.size(), false, "sx_cache_commit");
  if (st != SX_OK) return st;
  const int32_t b = c->b;
  for (int32_t x : r.src) c->put(x);
  r.src.clear();
  r.committed = true;
  Digest parent{};
  const int32_t full = (int32_t)(r.tokens.size() / (size_t)b);
  for (int32_t i = 0; i < full; ++i) {
    const Digest h = prefix_hash(i ? parent.data() : nullptr, r.tokens.data() + (int64_t)i * b, b, prefix_key,
                                 prefix_key_len);
    const int32_t x = r.table[i];
    if (!c->has_prefix[x] && c->prefix_index.find(h) == c->prefix_index.end()) {
      c->prefix_index.emplace(h, x);
      c->prefix_of[x] = h;
      c->has_prefix[x] = 1;
    }
    parent = h;
  }
  for (int32_t s = 0; s < n_publish; ++s) {
    const sx_span& p = publish[s];
    for (int32_t i = p.start / b; i < (p.start + p.length) / b; ++i) {
      const int32_t x = r.table[i];
      const Digest vh = virtual_hash(r.tokens.data() + (int64_t)i * b, b, p.extra_key, p.extra_key_len);
      auto v = c->virt_index.find(vh);
      if (v == c->virt_index.end()) {
        v = c->virt_index.emplace(vh, sx_cache::VEnt{x, i * b}).first;
        c->virt_of[x].push_back(vh);
      }
      if (p.freeze && v->second.block == x) c->frozen[x] = 1;   // held by this request: not idle
    }
  }
  return SX_OK;
}

sx_status sx_cache_release(sx_cache* c, int32_t request_id) {
  if (!c) return cfail(SX_EINVAL, "cache is NULL");
  auto it = c->reqs.find(request_id);
  if (it == c->reqs.end()) return cfail(SX_EINVAL, "sx_cache_release: no request %d", request_id);
  for (int32_t x : it->second.src) c->put(x);
  for (auto x = it->second.table.rbegin(); x != it->second.table.rend(); ++x) c->put(*x);
  c->reqs.erase(it);
  return SX_OK;
}

sx_status sx_cache_frozen_add(sx_cache* c, const int32_t* blocks, int32_t n) {
  if (!c || n < 0 || (!blocks && n > 0)) return cfail(SX_EINVAL, "sx_cache_frozen_add: bad arguments");
  for (int32_t i = 0; i < n; ++i) {
    if (blocks[i] < 0 || blocks[i] >= c->n) return cfail(SX_EINVAL, "block %d out of range", blocks[i]);
    if (c->virt_of[blocks[i]].empty()) return cfail(SX_EINVAL, "block %d carries no published entry", blocks[i]);
  }
  for (int32_t i = 0; i < n; ++i) {
    const int32_t x = blocks[i];
    if (c->frozen[x]) continue;
    c->frozen[x] = 1;
    if (c->ref[x] == 0) {
      c->q_remove(x);
      c->idle.insert(c->idle_key(x));
    }
  }
  return SX_OK;
}

sx_status sx_cache_frozen_delete(sx_cache* c, const int32_t* blocks, int32_t n) {
  if (!c || n < 0 || (!blocks && n > 0)) return cfail(SX_EINVAL, "sx_cache_frozen_delete: bad arguments");
  std::vector<int32_t> seen(blocks, blocks + n);
  std::sort(seen.begin(), seen.end());
  if (std::adjacent_find(seen.begin(), seen.end()) != seen.end()) return cfail(SX_EINVAL, "a block is listed twice");
  for (int32_t i = 0; i < n; ++i) {
    if (blocks[i] < 0 || blocks[i] >= c->n) return cfail(SX_EINVAL, "block %d out of range", blocks[i]);
    if (!c->frozen[blocks[i]]) return cfail(SX_EINVAL, "block %d is not frozen", blocks[i]);
  }
  for (int32_t i = 0; i < n; ++i) c->delete_frozen(blocks[i]);
  return SX_OK;
}

sx_status sx_cache_get_stats(const sx_cache* c, sx_cache_stats* out) {
  if (!c || !out) return cfail(SX_EINVAL, "NULL argument");
  int32_t in_use = 0, frozen = 0;
  for (int32_t x = 0; x < c->n; ++x) {
    in_use += c->ref[x] > 0;
    frozen += c->frozen[x] != 0;
  }
  out->free = c->n_free;
  out->in_use = in_use;
  out->frozen = frozen;
  out->idle_frozen = (int32_t)c->idle.size();
  out->prefix_entries = (int32_t)c->prefix_index.size();
  out->virtual_entries = (int32_t)c->virt_index.size();
  out->requests = (int32_t)c->reqs.size();
  return SX_OK;
}

sx_status sx_cache_get_block(const sx_cache* c, int32_t block, sx_cache_block* out) {
  if (!c || !out) return cfail(SX_EINVAL, "NULL argument");
  if (block < 0 || block >= c->n) return cfail(SX_EINVAL, "block %d out of range", block);
  out->ref = c->ref[block];
  out->frozen = c->frozen[block];
  out->in_free_queue = c->in_free[block];
  out->n_virtual = (int32_t)c->virt_of[block].size();
  out->has_prefix = c->has_prefix[block];
  out->hits = c->hits[block];
  out->last_use = c->last_use[block];
  return SX_OK;
}

sx_status sx_cache_free_queue(const sx_cache* c, int32_t* out, int32_t capacity, int32_t* n) {
  if (!c || !n) return cfail(SX_EINVAL, "NULL argument");
  *n = c->n_free;
  if (!out) return SX_OK;
  if (capacity < c->n_free) return cfail(SX_EINVAL, "capacity %d < %d queued blocks", capacity, c->n_free);
  int32_t i = 0;
  for (int32_t x = c->head; x >= 0; x = c->next[x]) out[i++] = x;
  return SX_OK;
}

}  // extern "C"
