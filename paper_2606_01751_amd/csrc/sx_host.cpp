// Host side of libsx: argument validation, plan construction (segment metadata, probe and base
// row sets, cos/sin tables) and dispatch of the HIP kernels.  See include/sx.h for the ABI.
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>

#include "sx_internal.h"

namespace {

thread_local std::string g_err;

sx_status fail(sx_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

sx_status ok() { return SX_OK; }

}  // namespace

// Checked library: device index arrays are validated before the kernels that read them.
#ifndef SX_DEVICE_CHECKS
#define SX_DEVICE_CHECKS 0
#endif
namespace {

const char* kCheckWhat[] = {"", "n_rows outside [0, T]", "row outside [0, T)", "rows not strictly ascending",
                            "cu_seqlens[0] is not 0", "request length negative or above max_seqlen"};

sx_status device_rows_ok(const sx_plan* p, const int32_t* rows, const int32_t* n_rows, int32_t max_rows,
                         void* stream, const char* who) {
  if (!SX_DEVICE_CHECKS || !n_rows) return SX_OK;
  int v[4] = {0, 0, 0, 0};
  const hipError_t e = sx::device_check_rows(p, rows, n_rows, max_rows, (hipStream_t)stream, v);
  if (e != hipSuccess) return fail(SX_EHIP, "%s: device check: %s", who, hipGetErrorString(e));
  if (v[0] != 0)
    return fail(SX_EDEVICE, "%s: %s (request %d, entry %d, value %d)", who, kCheckWhat[v[0] < 6 ? v[0] : 0], v[1],
                v[2], v[3]);
  return SX_OK;
}

sx_status device_cu_ok(const int32_t* cu, int32_t n_req, int32_t max_seqlen, void* stream, const char* who) {
  if (!SX_DEVICE_CHECKS) return SX_OK;
  int v[4] = {0, 0, 0, 0};
  const hipError_t e = sx::device_check_cu(cu, n_req, max_seqlen, (hipStream_t)stream, v);
  if (e != hipSuccess) return fail(SX_EHIP, "%s: device check: %s", who, hipGetErrorString(e));
  if (v[0] != 0)
    return fail(SX_EDEVICE, "%s: %s (request %d, value %d)", who, kCheckWhat[v[0] < 6 ? v[0] : 0], v[1], v[3]);
  return SX_OK;
}

}  // namespace

namespace sx {
sx_status report(sx_status st, const char* msg) {
  g_err = msg;
  return st;
}
}  // namespace sx

namespace {

sx_status hip_fail(hipError_t e, const char* what) {
  return fail(SX_EHIP, "%s: %s", what, hipGetErrorString(e));
}

// Checks a launch: the launcher's own status, then the runtime's sticky launch error.
sx_status check_launch(hipError_t e, const char* what) {
  if (e != hipSuccess) return hip_fail(e, what);
  e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, what);
  return SX_OK;
}

sx_status validate_desc(const sx_layer_desc* d) {
  if (!d) return fail(SX_EINVAL, "desc is NULL");
  if (d->n_q_heads < 1 || d->n_kv_heads < 1) return fail(SX_ESHAPE, "head counts must be >= 1");
  if (d->n_q_heads % d->n_kv_heads != 0)
    return fail(SX_ESHAPE, "n_q_heads (%d) must be a multiple of n_kv_heads (%d)", d->n_q_heads, d->n_kv_heads);
  // the scoring kernel streams at most 64 query columns (probe row x head of the group) per step
  if (d->n_q_heads / d->n_kv_heads > 64) return fail(SX_EUNSUPPORTED, "more than 64 query heads per KV head");
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(SX_EUNSUPPORTED, "head_dim %d unsupported (64 or 128)", d->head_dim);
  if (d->block_size != sx::kBlock) return fail(SX_EUNSUPPORTED, "block_size %d unsupported (16)", d->block_size);
  if (d->dtype != SX_F32 && d->dtype != SX_BF16) return fail(SX_EUNSUPPORTED, "dtype %d unsupported", d->dtype);
  if (d->rope_style != SX_ROPE_NEOX && d->rope_style != SX_ROPE_GPTJ)
    return fail(SX_EINVAL, "rope_style %d unknown", d->rope_style);
  if (!(d->rope_base > 0.0) || !std::isfinite(d->rope_base)) return fail(SX_EINVAL, "rope_base must be > 0");
  if (!(d->softmax_scale >= 0.0f) || !std::isfinite(d->softmax_scale))
    return fail(SX_EINVAL, "softmax_scale must be finite and >= 0");
  if (d->flags & ~SX_TOPK_ALL_POSITIONS) return fail(SX_EINVAL, "unknown flags 0x%x", (unsigned)d->flags);
  return SX_OK;
}

// largest thread count of a one-dimensional launch (gridDim.x * blockDim.x < 2^32, with margin)
constexpr int64_t kMaxThreads = ((int64_t)1 << 32) - ((int64_t)1 << 16);

float effective_scale(const sx_layer_desc* d) {
  return d->softmax_scale > 0.0f ? d->softmax_scale : (float)(1.0 / std::sqrt((double)d->head_dim));
}

template <typename T>
sx_status dev_alloc(sx_plan* p, T** ptr, size_t count) {
  *ptr = nullptr;
  if (count == 0) count = 1;
  hipError_t e = hipMalloc((void**)ptr, count * sizeof(T));
  if (e != hipSuccess) {
    *ptr = nullptr;
    return fail(SX_ENOMEM, "hipMalloc of %zu bytes failed: %s", count * sizeof(T), hipGetErrorString(e));
  }
  p->device_bytes += (int64_t)(count * sizeof(T));
  return SX_OK;
}

template <typename T>
sx_status dev_upload(sx_plan* p, T** ptr, const std::vector<T>& host) {
  sx_status st = dev_alloc(p, ptr, host.size());
  if (st != SX_OK) return st;
  if (!host.empty()) {
    hipError_t e = hipMemcpy(*ptr, host.data(), host.size() * sizeof(T), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy (plan upload)");
  }
  return SX_OK;
}

void free_plan(sx_plan* p) {
  if (!p) return;
  void* bufs[] = {p->d_req, p->d_bt, p->d_ra, p->d_cs, p->d_probe, p->d_nr, p->d_n_nr, p->d_n_probe,
                  p->d_flags, p->d_tok_row, p->d_rmark, p->d_lse, p->d_colsum,
                  p->d_qp, p->d_lse2p, p->d_lsep, p->d_tok_pos, p->d_theta, p->d_topk, p->d_queue,
                  p->d_order};
  for (void* b : bufs)
    if (b) (void)hipFree(b);
  delete p;
}

// The scoring scratch a plan owns (allocated and padded in sx_plan_create).
sx::ScoreScratch plan_scratch(const sx_plan* p) { return sx::ScoreScratch{p->d_colsum, p->d_qp, p->d_lse2p}; }

// k_r = min(n, floor(ratio * n + 1/2)), each float64 operation rounded on its own.
int64_t budget_of(int64_t n, double ratio) {
#pragma clang fp contract(off)
  volatile double prod = ratio * (double)n;
  double k = std::floor(prod + 0.5);
  if (k > (double)n) k = (double)n;
  if (k < 0) k = 0;
  return (int64_t)k;
}

}  // namespace

extern "C" {

const char* sx_last_error(void) { return g_err.c_str(); }

const char* sx_version(void) { return SX_DEVICE_CHECKS ? "libsx 0.2 (gfx950, device checks)" : "libsx 0.2 (gfx950)"; }

sx_status sx_plan_create(const sx_layer_desc* desc, const sx_request* requests, int32_t n_requests,
                         int64_t n_dst_blocks, int64_t n_src_blocks, sx_plan** out) {
  if (!out) return fail(SX_EINVAL, "out is NULL");
  sx_status st = validate_desc(desc);
  if (st != SX_OK) return st;
  if (!requests || n_requests < 1) return fail(SX_EINVAL, "need at least one request");
  if (n_dst_blocks < 1 || n_src_blocks < 0) return fail(SX_ESHAPE, "bad pool sizes");
  if (n_dst_blocks > (INT32_MAX / sx::kBlock) || n_src_blocks > (INT32_MAX / sx::kBlock))
    return fail(SX_EUNSUPPORTED, "pool larger than 2^31 slots");
  const int b = desc->block_size;
  const int d = desc->head_dim;

  // ---- validate every request before allocating anything ----
  int64_t total = 0;
  std::vector<uint8_t> dst_seen((size_t)n_dst_blocks, 0);
  for (int r = 0; r < n_requests; ++r) {
    const sx_request& q = requests[r];
    if (q.n_tokens < 1) return fail(SX_EINVAL, "request %d: n_tokens must be >= 1", r);
    if (q.n_segments < 1 || !q.segments) return fail(SX_EINVAL, "request %d: no segments", r);
    if (!q.block_table) return fail(SX_EINVAL, "request %d: block_table is NULL", r);
    int64_t t = 0;
    for (int m = 0; m < q.n_segments; ++m) {
      const sx_segment& s = q.segments[m];
      if (s.seq_start != t) return fail(SX_EINVAL, "request %d segment %d: starts at %d, expected %lld", r, m,
                                        s.seq_start, (long long)t);
      if (s.length < 1) return fail(SX_EINVAL, "request %d segment %d: length must be >= 1", r, m);
      if (s.cached != 0 && s.cached != 1) return fail(SX_EINVAL, "request %d segment %d: cached must be 0/1", r, m);
      if (s.new_pos < 0 || (int64_t)s.new_pos + s.length > INT32_MAX)
        return fail(SX_EINVAL, "request %d segment %d: bad new_pos", r, m);
      if (s.cached) {
        if (s.old_pos < 0 || (int64_t)s.old_pos + s.length > INT32_MAX)
          return fail(SX_EINVAL, "request %d segment %d: bad old_pos", r, m);
        const int64_t nb = (s.length + b - 1) / b;
        if (!q.src_block_ids || s.src_block_start < 0 || s.src_block_start + nb > q.n_src_block_ids)
          return fail(SX_ESHAPE, "request %d segment %d: source blocks out of range", r, m);
        for (int64_t i = 0; i < nb; ++i) {
          const int32_t id = q.src_block_ids[s.src_block_start + i];
          if (id < 0 || id >= n_src_blocks)
            return fail(SX_ESHAPE, "request %d segment %d: source block id %d out of range", r, m, id);
        }
      }
      t += s.length;
    }
    if (t != q.n_tokens) return fail(SX_EINVAL, "request %d: segments cover %lld tokens, n_tokens is %d", r,
                                     (long long)t, q.n_tokens);
    const int64_t nblk = (q.n_tokens + b - 1) / b;
    for (int64_t i = 0; i < nblk; ++i) {
      const int32_t id = q.block_table[i];
      if (id < 0 || id >= n_dst_blocks)
        return fail(SX_ESHAPE, "request %d: destination block id %d out of range", r, id);
      if (dst_seen[id]) return fail(SX_EINVAL, "destination block %d used twice", id);
      dst_seen[id] = 1;
    }
    total += q.n_tokens;
    if (total > INT32_MAX) return fail(SX_EUNSUPPORTED, "more than 2^31 tokens in one plan");
    if (q.n_tokens > (int64_t)sx::kTopkMaxChunks * sx::kTopkChunk)
      return fail(SX_EUNSUPPORTED, "request %d: %d tokens; the selection handles up to %d per request", r, q.n_tokens,
                  sx::kTopkMaxChunks * sx::kTopkChunk);
  }
  {
    // the element-wise kernels give each thread one 16-byte piece of a token row (queries have the
    // most pieces), in one-dimensional grids of fewer than 2^32 threads
    const int64_t pieces = total * desc->n_q_heads * d * (desc->dtype == SX_BF16 ? 2 : 4) / 16;
    if (pieces >= kMaxThreads)
      return fail(SX_EUNSUPPORTED, "%lld tokens x %d query heads exceed one launch", (long long)total, desc->n_q_heads);
  }

  sx_plan* p = new (std::nothrow) sx_plan();
  if (!p) return fail(SX_ENOMEM, "host allocation failed");
  p->desc = *desc;
  p->scale = effective_scale(desc);
  p->n_req = n_requests;
  p->total = total;
  p->n_dst_blocks = n_dst_blocks;
  p->n_src_blocks = n_src_blocks;
  (void)hipGetDevice(&p->device);
  if (hipDeviceGetAttribute(&p->n_cu, hipDeviceAttributeMultiprocessorCount, p->device) != hipSuccess ||
      p->n_cu < 1)
    p->n_cu = 256;

  // ---- derive the per-token sets (Sections 3.2-3.3, Algorithm 1 steps 15-16) ----
  std::vector<sx::ReqDev> rdev(n_requests);
  std::vector<int32_t> bt_all;
  std::vector<sx::RealignRow> ra;
  std::vector<float2> cs;
  // the probe list carries kProbePad zero entries past the last request: the column-sum kernel
  // reads whole chunks of probe rows without clamping
  std::vector<int32_t> probe((size_t)total + sx::kProbePad, 0), nr((size_t)total, 0);
  std::vector<int32_t> n_nr(n_requests), n_probe(n_requests);
  std::vector<uint8_t> flags((size_t)total, 0);
  std::vector<sx::RealignRow> tok_row((size_t)total, sx::RealignRow{-1, 0, 0, 0});
  std::vector<int32_t> tok_pos((size_t)total, 0);
  std::vector<double> theta(d / 2);
  for (int i = 0; i < d / 2; ++i) theta[i] = std::pow(desc->rope_base, -2.0 * i / d);
  int64_t off = 0;
  int32_t cs_rows = 0;
  for (int r = 0; r < n_requests; ++r) {
    const sx_request& q = requests[r];
    const int T = q.n_tokens;
    sx::HostReq h{};
    h.T = T;
    h.tok_off = (int32_t)off;
    h.bt_off = (int32_t)bt_all.size();
    const int nblk = (T + b - 1) / b;
    bt_all.insert(bt_all.end(), q.block_table, q.block_table + nblk);
    for (int t = 0; t < T; ++t) tok_row[off + t].dst_slot = q.block_table[t / b] * b + (t % b);
    uint8_t* fl = flags.data() + off;
    const sx_segment* last = nullptr;
    for (int m = 0; m < q.n_segments; ++m) {
      const sx_segment& s = q.segments[m];
      for (int j = 0; j < s.length; ++j) tok_pos[off + s.seq_start + j] = s.new_pos + j;
      if (s.seq_start <= T - 1 && T - 1 < s.seq_start + s.length) last = &s;
      if (!s.cached) continue;
      const double delta = (double)s.new_pos - (double)s.old_pos;
      for (int i = 0; i < d / 2; ++i) {
        const double phi = delta * theta[i];
        cs.push_back(make_float2((float)std::cos(phi), (float)std::sin(phi)));
      }
      for (int j = 0; j < s.length; ++j) {
        const int tok = s.seq_start + j;
        fl[tok] |= sx::kFlagCandidate;
        sx::RealignRow row;
        row.src_slot = q.src_block_ids[s.src_block_start + j / b] * b + (j % b);
        row.dst_slot = q.block_table[tok / b] * b + (tok % b);
        row.cs_row = cs_rows;
        row.pad = 0;
        tok_row[off + tok] = row;
        ra.push_back(row);
      }
      ++cs_rows;
    }
    // I_nr, overflow blocks around each maximal uncached run, tail fallback
    int cnt_nr = 0;
    for (int t = 0; t < T; ++t)
      if (!(fl[t] & sx::kFlagCandidate)) nr[off + cnt_nr++] = t;
    std::vector<uint8_t> base(T, 0);
    for (int t = 0; t < T;) {
      if (fl[t] & sx::kFlagCandidate) { ++t; continue; }
      const int a = t;
      while (t < T && !(fl[t] & sx::kFlagCandidate)) base[t++] = 1;
      const int e = t;
      for (int x = (a - b > 0 ? a - b : 0); x < a; ++x) base[x] = 1;
      for (int x = e; x < T && x < e + b; ++x) base[x] = 1;
    }
    int tail_lo = T;  // tail-fallback rows [tail_lo, T) when the final segment is reused
    if (last && last->cached) tail_lo = (T - sx::kTail > last->seq_start) ? T - sx::kTail : last->seq_start;
    for (int t = tail_lo; t < T; ++t) base[t] = 1;
    int cnt_probe = 0, cnt_base = 0, cnt_reuse = 0;
    for (int t = 0; t < T; ++t) {
      const bool cand = fl[t] & sx::kFlagCandidate;
      cnt_reuse += cand;
      if (!cand || t >= tail_lo) probe[off + cnt_probe++] = t;
      if (base[t]) { fl[t] |= sx::kFlagBase; ++cnt_base; }
    }
    if (p->desc.flags & SX_TOPK_ALL_POSITIONS) {   // Eq. topk over every position
      for (int t = 0; t < T; ++t) fl[t] |= sx::kFlagCandidate;
      cnt_reuse = T;
    }
    h.n_reuse = cnt_reuse;
    h.n_probe = cnt_probe;
    h.n_nr = cnt_nr;
    h.n_base = cnt_base;
    p->reqs.push_back(h);
    rdev[r] = sx::ReqDev{h.T, h.tok_off, h.bt_off, h.n_reuse, h.n_probe, h.n_nr, h.n_base, (int32_t)p->n_probe};
    n_nr[r] = cnt_nr;
    n_probe[r] = cnt_probe;
    p->n_reuse += cnt_reuse;
    p->n_nr += cnt_nr;
    p->n_probe += cnt_probe;
    p->n_base += cnt_base;
    if (cnt_nr > p->max_nr) p->max_nr = cnt_nr;
    if (cnt_probe > p->max_probe) p->max_probe = cnt_probe;
    if (T > p->max_T) p->max_T = T;
    off += T;
  }
  p->n_realign = (int64_t)ra.size();

  st = SX_OK;
  if (st == SX_OK) st = dev_upload(p, &p->d_req, rdev);
  if (st == SX_OK) st = dev_upload(p, &p->d_bt, bt_all);
  if (st == SX_OK) st = dev_upload(p, &p->d_ra, ra);
  if (st == SX_OK) st = dev_upload(p, &p->d_cs, cs);
  if (st == SX_OK) st = dev_upload(p, &p->d_probe, probe);
  if (st == SX_OK) st = dev_upload(p, &p->d_nr, nr);
  if (st == SX_OK) st = dev_upload(p, &p->d_n_nr, n_nr);
  if (st == SX_OK) st = dev_upload(p, &p->d_n_probe, n_probe);
  if (st == SX_OK) st = dev_upload(p, &p->d_flags, flags);
  if (st == SX_OK) st = dev_upload(p, &p->d_tok_row, tok_row);
  if (st == SX_OK) st = dev_upload(p, &p->d_tok_pos, tok_pos);
  if (st == SX_OK) st = dev_upload(p, &p->d_theta, theta);
  if (st == SX_OK) st = dev_upload(p, &p->d_rmark, std::vector<uint32_t>((size_t)total, 0u));
  if (st == SX_OK) st = dev_upload(p, &p->d_queue, std::vector<int32_t>((size_t)desc->n_kv_heads + 1, 0));
  if (st == SX_OK) st = dev_upload(p, &p->d_order, std::vector<int32_t>(1 + (size_t)sx::kOrderMax, -1));
  if (st == SX_OK) st = dev_alloc(p, &p->d_lse, (size_t)total * desc->n_q_heads);
  if (st == SX_OK) st = dev_alloc(p, &p->d_colsum, (size_t)total * desc->n_kv_heads);
  if (st == SX_OK) {
    // selection scratch, zeroed once: every call leaves the histograms at zero
    const int64_t chunks = (p->max_T + sx::kTopkChunk - 1) / sx::kTopkChunk;
    const size_t words = (size_t)n_requests * (sx::kTopkFine + 256 + 4 + 2 * chunks) + 2 * (size_t)total;
    st = dev_alloc(p, &p->d_topk, words);
    if (st == SX_OK) {
      hipError_t e = hipMemset(p->d_topk, 0, words * sizeof(uint32_t));
      if (e != hipSuccess) st = hip_fail(e, "hipMemset (selection scratch)");
    }
    if (st == SX_OK) {
      uint32_t* w = p->d_topk;
      p->topk.hist = w;   // 16-byte aligned rows of 65536 + 256 words
      w += (size_t)n_requests * (sx::kTopkFine + 256);
      p->topk.list = (uint2*)w;   // (8-byte aligned: the histograms fill a multiple of 16 bytes)
      w += 2 * (size_t)total;
      p->topk.state = w;
      w += (size_t)n_requests * 4;
      p->topk.cnt = (int32_t*)w;
      p->topk.max_chunks = (int32_t)chunks;
    }
  }
  if (st == SX_OK && desc->dtype == SX_BF16) {
    // gathered probe columns, kProbePad padding rows past the last probe row (per KV head for the
    // log-sum-exps) so that a chunk read past the end stays in bounds: zero queries, +inf
    // log-sum-exps
    const size_t rows = (size_t)p->n_probe + sx::kProbePad;
    uint16_t* qp = nullptr;
    st = dev_alloc(p, &qp, rows * desc->n_q_heads * d);
    p->d_qp = qp;
    if (st == SX_OK) st = dev_alloc(p, &p->d_lse2p, rows * desc->n_q_heads);
    // (max, sum) partials of the split log-sum-exp pass: every entry of a probe row is written by
    // its pieces before the merge reads it
    if (st == SX_OK && p->n_probe > 0)
      st = dev_alloc(p, &p->d_lsep, (size_t)sx::kLseSplit * p->n_probe * desc->n_q_heads);
    if (st == SX_OK) {
      hipError_t e = hipMemset(p->d_qp, 0, rows * desc->n_q_heads * d * sizeof(uint16_t));
      if (e == hipSuccess) e = hipMemset(p->d_lse2p, 0, rows * desc->n_q_heads * sizeof(float));
      const int64_t G = desc->n_q_heads / desc->n_kv_heads;
      for (int h = 0; h < desc->n_kv_heads && e == hipSuccess; ++h)
        e = hipMemsetD32((hipDeviceptr_t)(p->d_lse2p + ((int64_t)h * rows + p->n_probe) * G), (int)sx::kProbePadLse,
                         (size_t)sx::kProbePad * G);
      if (e != hipSuccess) st = hip_fail(e, "hipMemset (plan scratch)");
    }
  }
  if (st != SX_OK) {
    std::string keep = g_err;
    free_plan(p);
    g_err = keep;
    return st;
  }
  *out = p;
  return ok();
}

sx_status sx_plan_destroy(sx_plan* plan) {
  if (!plan) return SX_OK;
  hipError_t e = hipDeviceSynchronize();
  free_plan(plan);
  if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize before freeing the plan");
  return SX_OK;
}

sx_status sx_plan_get_info(const sx_plan* p, sx_plan_info* info) {
  if (!p || !info) return fail(SX_EINVAL, "NULL argument");
  info->total_tokens = p->total;
  info->n_requests = p->n_req;
  info->max_tokens = p->max_T;
  info->n_reused = p->n_reuse;
  info->n_nonreused = p->n_nr;
  info->n_probes = p->n_probe;
  info->n_base = p->n_base;
  info->max_nonreused = p->max_nr;
  info->max_probes = p->max_probe;
  info->device_bytes = p->device_bytes;
  return SX_OK;
}

sx_status sx_plan_budget(const sx_plan* p, double ratio, int64_t* k_total, int32_t* max_rows) {
  if (!p) return fail(SX_EINVAL, "plan is NULL");
  if (!(ratio >= 0.0 && ratio <= 1.0)) return fail(SX_EINVAL, "ratio must lie in [0, 1]");
  int64_t kt = 0;
  int64_t mr = 0;
  for (const auto& h : p->reqs) {
    const int64_t k = budget_of(h.n_reuse, ratio);
    kt += k;
    int64_t bound = h.n_base + k;
    if (bound > h.T) bound = h.T;
    if (bound > mr) mr = bound;
  }
  if (k_total) *k_total = kt;
  if (max_rows) *max_rows = (int32_t)mr;
  return SX_OK;
}

sx_status sx_plan_nonreused_rows(const sx_plan* p, const int32_t** rows, const int32_t** n_rows,
                                 int32_t* max_rows) {
  if (!p) return fail(SX_EINVAL, "plan is NULL");
  if (rows) *rows = p->d_nr;
  if (n_rows) *n_rows = p->d_n_nr;
  if (max_rows) *max_rows = p->max_nr;
  return SX_OK;
}

sx_status sx_rope_realign(const sx_plan* p, const void* src_k, const void* src_v, void* k_cache,
                          void* v_cache, void* stream) {
  if (!p) return fail(SX_EINVAL, "plan is NULL");
  if (p->n_realign == 0) return SX_OK;
  if (!src_k || !src_v || !k_cache || !v_cache) return fail(SX_EINVAL, "NULL tensor argument");
  return check_launch(sx::launch_realign(p, src_k, src_v, k_cache, v_cache, (hipStream_t)stream),
                      "sx_rope_realign launch");
}

sx_status sx_kv_scatter(const sx_plan* p, const void* k_new, const void* v_new, const int32_t* rows,
                        const int32_t* n_rows, int32_t max_rows, void* k_cache, void* v_cache, void* stream) {
  if (!p) return fail(SX_EINVAL, "plan is NULL");
  if (!k_new || !v_new || !k_cache || !v_cache) return fail(SX_EINVAL, "NULL tensor argument");
  if (rows) {
    if (!n_rows) return fail(SX_EINVAL, "n_rows is NULL while rows is not");
    if (max_rows < 0) return fail(SX_EINVAL, "max_rows must be >= 0");
    if (max_rows == 0) return SX_OK;
    sx_status st = device_rows_ok(p, rows, n_rows, max_rows, stream, "sx_kv_scatter");
    if (st != SX_OK) return st;
  }
  return check_launch(sx::launch_scatter(p, k_new, v_new, rows, n_rows, rows ? max_rows : p->max_T, k_cache,
                                         v_cache, (hipStream_t)stream),
                      "sx_kv_scatter launch");
}

sx_status sx_realign_scatter_layers(const sx_plan* p, int32_t n_layers, const sx_layer_kv* layers,
                                    const int32_t* rows, const int32_t* n_rows, int32_t max_rows, void* stream) {
  if (!p) return fail(SX_EINVAL, "plan is NULL");
  if (n_layers < 0) return fail(SX_EINVAL, "n_layers must be >= 0");
  if (n_layers > 0 && !layers) return fail(SX_EINVAL, "layers is NULL");
  if (!rows || !n_rows) return fail(SX_EINVAL, "NULL row list");
  if (max_rows < 0) return fail(SX_EINVAL, "max_rows must be >= 0");
  for (int32_t l = 0; l < n_layers; ++l) {
    const sx_layer_kv& x = layers[l];
    if (!x.k_new || !x.v_new || !x.k_cache || !x.v_cache) return fail(SX_EINVAL, "layer %d: NULL tensor", l);
    if (p->n_realign > 0 && (!x.src_k || !x.src_v)) return fail(SX_EINVAL, "layer %d: NULL source pool", l);
  }
  if (p->total == 0 || n_layers == 0) return SX_OK;
  {
    sx_status st = device_rows_ok(p, rows, n_rows, max_rows, stream, "sx_realign_scatter");
    if (st != SX_OK) return st;
  }
  const int64_t units = (int64_t)p->desc.n_kv_heads * p->desc.head_dim * (p->desc.dtype == SX_BF16 ? 2 : 4) / 32;
  if (p->total * units >= ((int64_t)1 << 31))
    return fail(SX_EUNSUPPORTED, "%lld tokens x %lld units exceed one launch", (long long)p->total, (long long)units);
  // a new generation for this call's row set; on wrap-around every mark is cleared first
  bool clear = false;
  if (++p->rgen == 0) {
    p->rgen = 1;
    clear = true;
  }
  return check_launch(sx::launch_realign_scatter(p, n_layers, layers, rows, n_rows, max_rows, p->rgen, clear,
                                                 nullptr, (hipStream_t)stream),
                      "sx_realign_scatter launch");
}

sx_status sx_rows_mask(const sx_plan* p, const int32_t* rows, const int32_t* n_rows, int32_t max_rows, uint8_t* mask,
                       void* stream) {
  if (!p) return fail(SX_EINVAL, "plan is NULL");
  if (!rows || !n_rows || !mask) return fail(SX_EINVAL, "NULL argument");
  if (max_rows < 0) return fail(SX_EINVAL, "max_rows must be >= 0");
  if (p->total == 0) return SX_OK;
  {
    sx_status st = device_rows_ok(p, rows, n_rows, max_rows, stream, "sx_rows_mask");
    if (st != SX_OK) return st;
  }
  sx_status st = check_launch(sx::launch_rows_mask(p, rows, n_rows, max_rows, mask, (hipStream_t)stream),
                              "sx_rows_mask launch");
  if (st != SX_OK || p->desc.dtype != SX_BF16) return st;
  // the planned row-tile order of sx_sparse_attn for this row list
  st = check_launch(sx::launch_tile_order(p, rows, n_rows, max_rows, (hipStream_t)stream), "sx_rows_mask order launch");
  if (st == SX_OK) {
    p->order_rows = rows;
    p->order_n_rows = n_rows;
    p->order_max_rows = max_rows;
  }
  return st;
}

sx_status sx_realign_scatter_masked(const sx_plan* p, const void* src_k, const void* src_v, const void* k_new,
                                    const void* v_new, const uint8_t* mask, void* k_cache, void* v_cache,
                                    void* stream) {
  if (!p) return fail(SX_EINVAL, "plan is NULL");
  if (!mask) return fail(SX_EINVAL, "mask is NULL");
  if (!k_new || !v_new || !k_cache || !v_cache) return fail(SX_EINVAL, "NULL tensor argument");
  if (p->n_realign > 0 && (!src_k || !src_v)) return fail(SX_EINVAL, "NULL source pool");
  if (p->total == 0) return SX_OK;
  const int64_t units = (int64_t)p->desc.n_kv_heads * p->desc.head_dim * (p->desc.dtype == SX_BF16 ? 2 : 4) / 32;
  if (p->total * units >= ((int64_t)1 << 31))
    return fail(SX_EUNSUPPORTED, "%lld tokens x %lld units exceed one launch", (long long)p->total, (long long)units);
  const sx_layer_kv one{src_k, src_v, k_new, v_new, k_cache, v_cache};
  return check_launch(sx::launch_realign_scatter(p, 1, &one, nullptr, nullptr, 0, 0, false, mask, (hipStream_t)stream),
                      "sx_realign_scatter_masked launch");
}

sx_status sx_realign_scatter(const sx_plan* p, const void* src_k, const void* src_v, const void* k_new,
                             const void* v_new, const int32_t* rows, const int32_t* n_rows, int32_t max_rows,
                             void* k_cache, void* v_cache, void* stream) {
  const sx_layer_kv one{src_k, src_v, k_new, v_new, k_cache, v_cache};
  return sx_realign_scatter_layers(p, 1, &one, rows, n_rows, max_rows, stream);
}

namespace {

sx_status check_rows(const sx_plan* p, const int32_t* rows, const int32_t* n_rows, int32_t max_rows, bool need_rows,
                     void* stream, const char* who) {
  if (!p) return fail(SX_EINVAL, "plan is NULL");
  if (p->desc.dtype != SX_BF16) return fail(SX_EUNSUPPORTED, "the layer body runs on bfloat16 plans");
  if (!n_rows || (need_rows && !rows)) return fail(SX_EINVAL, "NULL row list");
  if (max_rows < 0) return fail(SX_EINVAL, "max_rows must be >= 0");
  if (max_rows > p->max_T) return fail(SX_ESHAPE, "max_rows %d exceeds the longest request (%d)", max_rows, p->max_T);
  if (max_rows == 0) return SX_OK;
  return device_rows_ok(p, rows, n_rows, max_rows, stream, who);
}

}  // namespace

sx_status sx_gemm_rows(const sx_plan* p, const int32_t* rows, const int32_t* n_rows, int32_t max_rows, const void* x,
                       int32_t x_by_token, const void* w, int32_t k, int32_t n, const void* residual, void* y,
                       int32_t y_by_token, void* stream) {
  sx_status st = check_rows(p, rows, n_rows, max_rows, x_by_token || y_by_token, stream, "sx_gemm_rows");
  if (st != SX_OK) return st;
  if (!x || !w || !y) return fail(SX_EINVAL, "NULL tensor argument");
  if (k <= 0 || n <= 0 || k % 64 != 0 || n % 256 != 0)
    return fail(SX_EUNSUPPORTED, "sx_gemm_rows needs k a multiple of 64 and n a multiple of 256 (k=%d n=%d)", k, n);
  if (max_rows == 0) return SX_OK;
  const sx::RowsArg r{rows, n_rows, max_rows};
  const int part_n[1] = {n};
  void* const ys[1] = {y};
  return check_launch(sx::launch_gemm_rows(p, r, x, x_by_token != 0, w, k, 1, part_n, ys, residual, y_by_token != 0,
                                           (hipStream_t)stream),
                      "sx_gemm_rows launch");
}

sx_status sx_gemm_rows_split(const sx_plan* p, const int32_t* rows, const int32_t* n_rows, int32_t max_rows,
                             const void* x, int32_t x_by_token, const void* w, int32_t k, int32_t n_parts,
                             const int32_t* part_n, void* const* y_parts, int32_t y_by_token, void* stream) {
  sx_status st = check_rows(p, rows, n_rows, max_rows, x_by_token || y_by_token, stream, "sx_gemm_rows_split");
  if (st != SX_OK) return st;
  if (!x || !w || !part_n || !y_parts) return fail(SX_EINVAL, "NULL argument");
  if (n_parts < 1 || n_parts > 4) return fail(SX_EINVAL, "n_parts %d outside 1..4", n_parts);
  if (k <= 0 || k % 64 != 0) return fail(SX_EUNSUPPORTED, "sx_gemm_rows_split needs k a multiple of 64 (k=%d)", k);
  int64_t n = 0;
  for (int i = 0; i < n_parts; ++i) {
    if (!y_parts[i]) return fail(SX_EINVAL, "output part %d is NULL", i);
    if (part_n[i] <= 0 || part_n[i] % 256 != 0)
      return fail(SX_EUNSUPPORTED, "part %d width %d is not a positive multiple of 256", i, part_n[i]);
    n += part_n[i];
  }
  if (n > INT32_MAX) return fail(SX_EINVAL, "total width %lld too large", (long long)n);
  if (max_rows == 0) return SX_OK;
  const sx::RowsArg r{rows, n_rows, max_rows};
  return check_launch(sx::launch_gemm_rows(p, r, x, x_by_token != 0, w, k, n_parts, part_n, y_parts, nullptr,
                                           y_by_token != 0, (hipStream_t)stream),
                      "sx_gemm_rows_split launch");
}

sx_status sx_rmsnorm_rows(const sx_plan* p, const int32_t* rows, const int32_t* n_rows, int32_t max_rows,
                          const void* x, int32_t x_by_token, const void* gamma, float eps, int32_t h, void* y,
                          int32_t y_by_token, void* stream) {
  sx_status st = check_rows(p, rows, n_rows, max_rows, x_by_token || y_by_token, stream, "sx_rmsnorm_rows");
  if (st != SX_OK) return st;
  if (!x || !gamma || !y) return fail(SX_EINVAL, "NULL tensor argument");
  if (h <= 0 || h % 8 != 0) return fail(SX_EUNSUPPORTED, "hidden size %d must be a positive multiple of 8", h);
  if (!(eps > 0.0f) || !std::isfinite(eps)) return fail(SX_EINVAL, "eps must be finite and > 0");
  if (max_rows == 0) return SX_OK;
  const sx::RowsArg r{rows, n_rows, max_rows};
  return check_launch(sx::launch_rmsnorm_rows(p, r, x, x_by_token != 0, gamma, eps, h, y, y_by_token != 0,
                                              (hipStream_t)stream),
                      "sx_rmsnorm_rows launch");
}

sx_status sx_rope_rows(const sx_plan* p, const int32_t* rows, const int32_t* n_rows, int32_t max_rows, void* q,
                       void* k, void* stream) {
  sx_status st = check_rows(p, rows, n_rows, max_rows, true, stream, "sx_rope_rows");
  if (st != SX_OK) return st;
  if (!q || !k) return fail(SX_EINVAL, "NULL tensor argument");
  if (max_rows == 0) return SX_OK;
  const sx::RowsArg r{rows, n_rows, max_rows};
  return check_launch(sx::launch_rope_rows(p, r, q, k, (hipStream_t)stream), "sx_rope_rows launch");
}

sx_status sx_silu_mul_rows(const sx_plan* p, const int32_t* n_rows, int32_t max_rows, const void* gate_up, int32_t f,
                           void* y, void* stream) {
  sx_status st = check_rows(p, nullptr, n_rows, max_rows, false, stream, "sx_silu_mul_rows");
  if (st != SX_OK) return st;
  if (!gate_up || !y) return fail(SX_EINVAL, "NULL tensor argument");
  if (f <= 0 || f % 8 != 0) return fail(SX_EUNSUPPORTED, "feed-forward size %d must be a positive multiple of 8", f);
  if ((int64_t)max_rows * (f / 8) >= kMaxThreads) return fail(SX_EUNSUPPORTED, "%d rows x %d exceed one launch", max_rows, f);
  if (max_rows == 0) return SX_OK;
  const sx::RowsArg r{nullptr, n_rows, max_rows};
  return check_launch(sx::launch_silu_mul_rows(p, r, gate_up, f, y, (hipStream_t)stream), "sx_silu_mul_rows launch");
}

sx_status sx_sparseq_score(const sx_plan* p, const void* q, const void* k_cache, const float* lse_in, float* scores,
                           void* stream) {
  if (!p) return fail(SX_EINVAL, "plan is NULL");
  if (!q || !k_cache || !scores) return fail(SX_EINVAL, "NULL tensor argument");
  hipStream_t s = (hipStream_t)stream;
  if (lse_in) {
    // one pass: the denominators come from the caller (natural log, indexed by token)
    sx_status st = check_launch(sx::launch_colsum(p, plan_scratch(p), q, k_cache, lse_in, 1, s),
                                "sx_sparseq_score column-sum launch");
    if (st != SX_OK) return st;
    return check_launch(sx::launch_head_reduce(p, p->d_colsum, scores, s), "sx_sparseq_score head-sum launch");
  }
  // pass 1: log-sum-exp of every (probe row, query head)
  sx::AttnLaunch a{};
  a.Hq = p->desc.n_q_heads;
  a.Hkv = p->desc.n_kv_heads;
  a.D = p->desc.head_dim;
  a.n_req = p->n_req;
  a.grid_rows = p->max_probe;
  a.dtype = p->desc.dtype;
  a.scale = p->scale;
  a.q = q;
  a.k = k_cache;
  a.v = nullptr;
  a.out = nullptr;
  a.lse = p->d_lse;
  a.lse_base2 = 1;
  a.reqs = p->d_req;
  a.bt = p->d_bt;
  a.rows = p->d_probe;
  a.n_rows = p->d_n_probe;
  a.lse_part = p->d_lsep;
  a.n_part_rows = p->n_probe;
  sx_status st = SX_OK;
  if (p->max_probe > 0) {
    st = check_launch(sx::launch_attn_paged(a, s), "sx_sparseq_score pass 1 launch");
    if (st != SX_OK) return st;
  }
  // pass 2: per-key column sums of the probabilities, per KV head
  st = check_launch(sx::launch_colsum(p, plan_scratch(p), q, k_cache, p->d_lse, 0, s), "sx_sparseq_score pass 2 launch");
  if (st != SX_OK) return st;
  // pass 3: fixed-order sum over KV heads
  return check_launch(sx::launch_head_reduce(p, p->d_colsum, scores, s), "sx_sparseq_score pass 3 launch");
}

}  // extern "C"

namespace {

// Scratch of sx_sparseq_score_static: one array per device, in the library's code object, so the
// entry point needs no allocation.  Host code never uses the array's name as an address: the
// device address comes from hipGetSymbolAddress, once per device on its first call.
constexpr size_t kStaticScratchBytes = (size_t)32 << 20;
__device__ __align__(256) char scratch[kStaticScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

sx_status static_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(SX_EUNSUPPORTED, "device %d beyond the static scratch table", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) return hip_fail(e, "hipGetSymbolAddress of the static scratch");
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return SX_OK;
}

size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

}  // namespace

extern "C" {

sx_status sx_sparseq_score_static(const sx_plan* p, const void* q, const void* k_cache, const float* lse_in,
                                  float* scores, void* stream) {
  if (!p) return fail(SX_EINVAL, "plan is NULL");
  if (!q || !k_cache || !scores) return fail(SX_EINVAL, "NULL tensor argument");
  if (!lse_in) return fail(SX_EINVAL, "sx_sparseq_score_static needs lse_in (one-pass scoring)");
  const int64_t Hq = p->desc.n_q_heads, Hkv = p->desc.n_kv_heads, G = Hq / Hkv;
  const bool bf16 = p->desc.dtype == SX_BF16;
  const int64_t rows = p->n_probe + sx::kProbePad;
  const size_t colsum_b = align256((size_t)(Hkv * p->total) * sizeof(double));
  const size_t qp_b = bf16 ? align256((size_t)(rows * Hq * p->desc.head_dim) * sizeof(uint16_t)) : 0;
  const size_t lse_b = bf16 ? align256((size_t)(Hkv * rows * G) * sizeof(float)) : 0;
  const size_t need = colsum_b + qp_b + lse_b;
  if (need > kStaticScratchBytes)
    return fail(SX_EUNSUPPORTED, "the plan needs %zu bytes of scoring scratch; the static scratch holds %zu", need,
                kStaticScratchBytes);
  void* base = nullptr;
  sx_status st = static_scratch(&base);
  if (st != SX_OK) return st;
  char* b = (char*)base;
  const sx::ScoreScratch sc{(double*)b, bf16 ? (void*)(b + colsum_b) : nullptr,
                            bf16 ? (float*)(b + colsum_b + qp_b) : nullptr};
  hipStream_t s = (hipStream_t)stream;
  if (bf16) {
    // the gathered probe columns' padding rows (zero queries, +inf log-sum-exps): an earlier call may
    // have left anything
    st = check_launch(sx::launch_probe_pad_clear(p, sc, s), "sx_sparseq_score_static padding clear");
    if (st != SX_OK) return st;
  }
  st = check_launch(sx::launch_colsum(p, sc, q, k_cache, lse_in, 1, s), "sx_sparseq_score_static column-sum launch");
  if (st != SX_OK) return st;
  return check_launch(sx::launch_head_reduce(p, sc.colsum, scores, s), "sx_sparseq_score_static head-sum launch");
}

sx_status sx_topk_select(const sx_plan* p, const float* scores, double ratio, int32_t* rows, int32_t* n_rows,
                         void* stream) {
  if (!p) return fail(SX_EINVAL, "plan is NULL");
  if (!scores || !rows || !n_rows) return fail(SX_EINVAL, "NULL argument");
  if (!(ratio >= 0.0 && ratio <= 1.0)) return fail(SX_EINVAL, "ratio must lie in [0, 1]");
  return check_launch(sx::launch_topk(p, scores, ratio, rows, n_rows, (hipStream_t)stream),
                      "sx_topk_select launch");
}

sx_status sx_sparse_attn(const sx_plan* p, const void* q, const int32_t* rows, const int32_t* n_rows,
                         int32_t max_rows, const void* k_cache, const void* v_cache, void* out, void* stream) {
  if (!p) return fail(SX_EINVAL, "plan is NULL");
  if (!q || !rows || !n_rows || !k_cache || !v_cache || !out) return fail(SX_EINVAL, "NULL argument");
  if (max_rows < 0) return fail(SX_EINVAL, "max_rows must be >= 0");
  if (max_rows == 0) return SX_OK;
  {
    sx_status st = device_rows_ok(p, rows, n_rows, max_rows, stream, "sx_sparse_attn");
    if (st != SX_OK) return st;
  }
  sx::AttnLaunch a{};
  a.Hq = p->desc.n_q_heads;
  a.Hkv = p->desc.n_kv_heads;
  a.D = p->desc.head_dim;
  a.n_req = p->n_req;
  a.grid_rows = max_rows;
  a.dtype = p->desc.dtype;
  a.scale = p->scale;
  a.q = q;
  a.k = k_cache;
  a.v = v_cache;
  a.out = out;
  a.lse = nullptr;
  a.reqs = p->d_req;
  a.bt = p->d_bt;
  a.rows = rows;
  a.n_rows = n_rows;
  a.queue = p->d_queue;
  a.n_cu = p->n_cu;
  a.order = rows == p->order_rows && n_rows == p->order_n_rows && max_rows == p->order_max_rows ? p->d_order : nullptr;
  return check_launch(sx::launch_attn_paged(a, (hipStream_t)stream), "sx_sparse_attn launch");
}

namespace {

// Compute units of the current device (cached per device; 0 if unknown).
int current_cu_count(int dev) {
  static std::atomic<int> cache[kMaxDevices];
  if (dev < 0 || dev >= kMaxDevices) return 0;
  int n = cache[dev].load(std::memory_order_relaxed);
  if (n == 0 && hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
    cache[dev].store(n, std::memory_order_relaxed);
  return n > 0 ? n : 0;
}

// Work-queue slot of a persistent full-attention launch on device dev: the slots are handed out in
// turn, so launches that overlap in time use different slots as long as fewer than
// kDenseQueueSlots are in flight on the device.  -1 (one workgroup per item, no counters) while the
// stream is being captured, since a graph node keeps its slot for every replay.
int dense_queue_slot(int dev, hipStream_t s) {
  static std::atomic<uint32_t> next[kMaxDevices];
  if (dev < 0 || dev >= kMaxDevices) return -1;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(s, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) {
    (void)hipGetLastError();
    return -1;
  }
  return (int)(next[dev].fetch_add(1, std::memory_order_relaxed) % (uint32_t)sx::kDenseQueueSlots);
}

}  // namespace

sx_status sx_full_attn(const sx_layer_desc* desc, const void* q, const void* k, const void* v,
                       const int32_t* cu_seqlens, int32_t n_requests, int32_t max_seqlen, void* out, float* lse,
                       void* stream) {
  sx_status st = validate_desc(desc);
  if (st != SX_OK) return st;
  if (!q || !k || !v || !out || !cu_seqlens) return fail(SX_EINVAL, "NULL argument");
  if (n_requests < 1) return fail(SX_EINVAL, "n_requests must be >= 1");
  if (max_seqlen < 0) return fail(SX_EINVAL, "max_seqlen must be >= 0");
  if (max_seqlen == 0) return SX_OK;
  st = device_cu_ok(cu_seqlens, n_requests, max_seqlen, stream, "sx_full_attn");
  if (st != SX_OK) return st;
  sx::AttnLaunch a{};
  a.Hq = desc->n_q_heads;
  a.Hkv = desc->n_kv_heads;
  a.D = desc->head_dim;
  a.n_req = n_requests;
  a.grid_rows = max_seqlen;
  a.dtype = desc->dtype;
  a.scale = effective_scale(desc);
  a.q = q;
  a.k = k;
  a.v = v;
  a.out = out;
  a.lse = lse;
  a.lse_base2 = 0;
  a.cu = cu_seqlens;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  a.n_cu = current_cu_count(dev);
  a.qslot = a.n_cu > 0 && a.Hkv < sx::kDenseQueueStride ? dense_queue_slot(dev, (hipStream_t)stream) : -1;
  return check_launch(sx::launch_attn_dense(a, (hipStream_t)stream), "sx_full_attn launch");
}

}  // extern "C"
