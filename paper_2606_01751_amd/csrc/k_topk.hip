// Key selection and recompute set (Eq. topk, Section 3.3, Algorithm 1 steps 14-17).
//
// Per request, k_r = min(n_r, floor(ratio * n_r + 1/2)) over the n_r reused candidates; S_key = the
// k_r candidates with the largest float32 score, ties to the lower index; R = base rows (I_nr,
// overflow, tail fallback: precomputed plan flags) U S_key, ascending.
//
// Every request is cut into chunks of CHUNK tokens, one 256-thread workgroup per chunk, so a
// request's selection runs on many CUs:
//   passes 0-2  radix select of the k_r-th largest score among the candidates, 11 + 11 + 10 bits from
//               the most significant (scores are >= 0, so the IEEE bit pattern orders them): each
//               workgroup builds an LDS histogram of its candidates that match the digits found so
//               far and adds it to the request's histogram in plan scratch.  The workgroup that
//               finishes last (a per-request arrival counter) picks the digit, updates the
//               request's state (digits, candidates still needed) and clears the histogram and
//               the counter for the next pass, so the scratch is clean again without a fill.
//   count       per chunk: rows surely in R (base rows and candidates above the threshold), and
//               candidates equal to the threshold (ties).  The last workgroup turns the counts into
//               each chunk's output offset and tie rank (rescanning the one chunk in which the
//               tie budget runs out) and writes n_rows.
//   write       per chunk: an ordered compaction of its rows of R at the chunk's offset; a tie is in
//               R when its rank among the request's ties (index order) is below the tie budget.
// Scratch (plan-owned, zeroed once when the plan is made): the histograms and counters, the
// per-request state and the per-chunk counts and offsets.  Calls sharing a plan must be
// stream-ordered.
#include "sx_device.h"
#include "sx_internal.h"

namespace sx {
namespace {

constexpr int NT = 256;                  // threads per workgroup
constexpr int TPT = kTopkChunk / NT;     // tokens per thread (consecutive)
static_assert(TPT == 8, "a thread loads 8 consecutive scores (two 16-byte vectors) and 8 flags");
constexpr int NBINS = kTopkBins;         // 2048: 11-bit digits
constexpr int NWV = NT / 64;

__device__ __forceinline__ int64_t budget_dev(int64_t n, double ratio) {
#pragma clang fp contract(off)
  const double prod = ratio * (double)n;
  double k = floor(prod + 0.5);
  if (k > (double)n) k = (double)n;
  if (k < 0.0) k = 0.0;
  return (int64_t)k;
}

// digit layout of pass p: shift and width
__device__ __forceinline__ int pass_shift(int p) { return p == 0 ? 21 : (p == 1 ? 10 : 0); }
__device__ __forceinline__ uint32_t pass_bins(int p) { return p == 2 ? 1024u : 2048u; }

// 0: nothing selected (k = 0), 1: every candidate (k = n), 2: threshold and ties
__device__ __forceinline__ int select_mode(int64_t k, int64_t n) { return k == 0 ? 0 : (k == n ? 1 : 2); }

// this thread's 8 consecutive tokens of the chunk: score bits and flags (flags 0 past T)
__device__ __forceinline__ void load8(const uint32_t* sb, const uint8_t* fl, int t0, int T, uint32_t u[TPT],
                                      uint8_t f[TPT]) {
  // vector loads when whole and aligned (a request's tokens start anywhere in the concatenation)
  if (t0 + TPT <= T && (((uintptr_t)(sb + t0) & 15) | ((uintptr_t)(fl + t0) & 7)) == 0) {
    const uint4 a = *(const uint4*)(sb + t0);
    const uint4 b = *(const uint4*)(sb + t0 + 4);
    const uint2 fv = *(const uint2*)(fl + t0);
    u[0] = a.x; u[1] = a.y; u[2] = a.z; u[3] = a.w;
    u[4] = b.x; u[5] = b.y; u[6] = b.z; u[7] = b.w;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[i] = (uint8_t)(fv.x >> (8 * i));
      f[4 + i] = (uint8_t)(fv.y >> (8 * i));
    }
  } else {
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      const int t = t0 + i;
      u[i] = t < T ? sb[t] : 0u;
      f[i] = t < T ? fl[t] : (uint8_t)0;
    }
  }
}

// Exclusive prefix sum of v over the workgroup's threads in order, and the total.
__device__ __forceinline__ int block_excl_sum(int v, int* wsum, int& total) {
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[wv] = x;
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < NWV; ++i) {
    before += i < wv ? wsum[i] : 0;
    tot += wsum[i];
  }
  __syncthreads();
  total = tot;
  return before + x - v;
}

// Arrival of this workgroup at the request's counter; true in the last one (after the fence, it
// sees every other workgroup's scratch writes).  The last one resets the counter.
__device__ __forceinline__ bool arrive_last(uint32_t* ctr, uint32_t n_blocks, int* s_flag) {
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t old = atomicAdd(ctr, 1u);
    const bool last = old == n_blocks - 1;
    if (last) *ctr = 0u;
    *s_flag = last ? 1 : 0;
  }
  __syncthreads();
  const bool last = *s_flag != 0;
  if (last) __threadfence();
  return last;
}

struct TopkArgs {
  const ReqDev* reqs;
  const uint8_t* flags;
  const uint32_t* scores;   // float32 bit patterns
  double ratio;
  TopkScratch sc;
  int32_t* rows;
  int32_t* n_rows;
};

// Radix pass p over every chunk of every request (blockIdx.y = request, blockIdx.x = chunk).
__global__ __launch_bounds__(NT) void topk_hist_kernel(TopkArgs a, int p) {
  __shared__ uint32_t hist[NBINS];
  __shared__ int wsum[NWV];
  __shared__ int s_flag;
  __shared__ uint32_t s_digit;
  __shared__ int s_rem;
  const int r = blockIdx.y;
  const ReqDev rq = a.reqs[r];
  const int T = rq.T;
  const uint32_t nb = (uint32_t)((T + kTopkChunk - 1) / kTopkChunk);
  if (blockIdx.x >= nb) return;
  const int64_t n = rq.n_reuse;
  const int64_t k = budget_dev(n, a.ratio);
  if (select_mode(k, n) != 2) return;
  uint32_t prefix = 0, mask = 0;
  int remaining = (int)k;
  uint32_t* st = a.sc.state + 4 * r;
  if (p > 0) {
    prefix = st[0];
    mask = st[1];
    remaining = (int)st[2];
  }
  const int shift = pass_shift(p);
  const uint32_t bins = pass_bins(p);
  const int tid = threadIdx.x;
  for (int i = tid; i < NBINS; i += NT) hist[i] = 0u;
  __syncthreads();
  uint32_t u[TPT];
  uint8_t f[TPT];
  load8(a.scores + rq.tok_off, a.flags + rq.tok_off, blockIdx.x * kTopkChunk + tid * TPT, T, u, f);
#pragma unroll
  for (int i = 0; i < TPT; ++i) {
    if ((f[i] & kFlagCandidate) && (u[i] & mask) == prefix) atomicAdd(&hist[(u[i] >> shift) & (bins - 1)], 1u);
  }
  __syncthreads();
  uint32_t* gh = a.sc.hist + (size_t)r * NBINS;
  for (int i = tid; i < NBINS; i += NT) {
    const uint32_t c = hist[i];
    if (c) atomicAdd(&gh[i], c);
  }
  if (!arrive_last(a.sc.ctr + r, nb, &s_flag)) return;
  // the last workgroup: digit = the largest d with (matching candidates in bins >= d) >= remaining;
  // thread t holds bins 8t .. 8t+7 (pass 2 has 1024 bins: the upper half stays empty)
  constexpr int per = NBINS / NT;
  uint32_t c[per];
  int loc = 0;
#pragma unroll
  for (int i = 0; i < per; ++i) {
    c[i] = __hip_atomic_load(&gh[per * tid + i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    loc += (int)c[i];
  }
  int total;
  const int below = block_excl_sum(loc, wsum, total);   // bins of lower threads
  int ge = total - below - loc;                         // bins above this thread's
  int best = -1, best_gt = 0;
#pragma unroll
  for (int i = per - 1; i >= 0; --i) {
    const int gt_i = ge;
    ge += (int)c[i];
    if (best < 0 && ge >= remaining) {
      best = per * tid + i;
      best_gt = gt_i;
    }
  }
  // qualifying digits are exactly those <= the answer, so the answer is the best of the highest
  // thread that has one
  int top = best >= 0 ? tid : -1;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) top = max(top, __shfl_xor(top, o, 64));
  if ((tid & 63) == 0) wsum[tid >> 6] = top;
  __syncthreads();
  top = -1;
#pragma unroll
  for (int i = 0; i < NWV; ++i) top = max(top, wsum[i]);
  if (top < 0) {
    // fewer matching candidates than still needed: impossible when k <= n (kept defensive)
    if (tid == 0) {
      s_digit = 0u;
      s_rem = 0;
    }
  } else if (tid == top) {
    s_digit = (uint32_t)best;
    s_rem = remaining - best_gt;
  }
  __syncthreads();
  for (int i = tid; i < NBINS; i += NT) gh[i] = 0u;   // clean for the next pass or call
  if (tid == 0) {
    st[0] = prefix | (s_digit << shift);
    st[1] = mask | ((bins - 1) << shift);
    st[2] = (uint32_t)s_rem;
  }
}

// Per chunk: rows surely in R, ties and ties that are not sure rows; the last workgroup derives
// every chunk's output offset and tie rank and the request's |R|.
__global__ __launch_bounds__(NT) void topk_count_kernel(TopkArgs a) {
  __shared__ int wsum[NWV];
  __shared__ int s_flag;
  const int r = blockIdx.y;
  const ReqDev rq = a.reqs[r];
  const int T = rq.T;
  const uint32_t nb = (uint32_t)((T + kTopkChunk - 1) / kTopkChunk);
  if (blockIdx.x >= nb) return;
  const int64_t n = rq.n_reuse;
  const int64_t k = budget_dev(n, a.ratio);
  const int mode = select_mode(k, n);
  const uint32_t* st = a.sc.state + 4 * r;
  const uint32_t thr = mode == 2 ? st[0] : 0u;
  const int need_eq = mode == 2 ? (int)st[2] : 0;
  const int tid = threadIdx.x;
  const uint32_t* sb = a.scores + rq.tok_off;
  const uint8_t* fl = a.flags + rq.tok_off;
  auto classify = [&](uint32_t u, uint8_t f, bool& sure, bool& eq) {
    const bool cand = f & kFlagCandidate;
    const bool gt = mode == 2 && cand && u > thr;
    eq = mode == 2 && cand && u == thr;
    sure = (f & kFlagBase) || (mode == 1 ? cand : gt);
  };
  uint32_t u[TPT];
  uint8_t f[TPT];
  load8(sb, fl, blockIdx.x * kTopkChunk + tid * TPT, T, u, f);
  int ns = 0, ne = 0, nens = 0;
#pragma unroll
  for (int i = 0; i < TPT; ++i) {
    bool sure, eq;
    classify(u[i], f[i], sure, eq);
    ns += sure;
    ne += eq;
    nens += eq && !sure;
  }
  int ts, te, tens;
  block_excl_sum(ns, wsum, ts);
  block_excl_sum(ne, wsum, te);
  block_excl_sum(nens, wsum, tens);
  int32_t* cnt = a.sc.cnt + (size_t)r * a.sc.max_chunks * 3;
  if (tid == 0) {
    cnt[3 * blockIdx.x + 0] = ts;
    cnt[3 * blockIdx.x + 1] = te;
    cnt[3 * blockIdx.x + 2] = tens;
  }
  if (!arrive_last(a.sc.ctr + r, nb, &s_flag)) return;
  // last workgroup: walk the chunks in order (thread 0), finding the one chunk whose ties straddle
  // the tie budget; that chunk's count of selected ties that are not sure rows needs a rescan
  __shared__ int s_bchunk, s_blim;
  if (tid == 0) {
    int eb = 0, bchunk = -1, blim = 0;
    for (uint32_t b = 0; b < nb; ++b) {
      const int e = __hip_atomic_load(&cnt[3 * b + 1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const int lim = min(max(need_eq - eb, 0), e);
      if (lim > 0 && lim < e) {
        bchunk = (int)b;
        blim = lim;
      }
      eb += e;
    }
    s_bchunk = bchunk;
    s_blim = blim;
  }
  __syncthreads();
  int bsel = 0;   // ties of the boundary chunk with rank < blim that are not sure rows
  if (s_bchunk >= 0) {
    load8(sb, fl, s_bchunk * kTopkChunk + tid * TPT, T, u, f);
    int e_loc = 0;
    bool se[TPT], ee[TPT];
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      classify(u[i], f[i], se[i], ee[i]);
      e_loc += ee[i];
    }
    int e_tot;
    int rank = block_excl_sum(e_loc, wsum, e_tot);
    int mine = 0;
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      if (ee[i]) {
        mine += (!se[i] && rank < s_blim) ? 1 : 0;
        ++rank;
      }
    }
    block_excl_sum(mine, wsum, bsel);
  }
  if (tid == 0) {
    int out = 0, eb = 0;
    int32_t* pre = a.sc.pre + (size_t)r * a.sc.max_chunks * 2;
    for (uint32_t b = 0; b < nb; ++b) {
      const int s = __hip_atomic_load(&cnt[3 * b + 0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const int e = __hip_atomic_load(&cnt[3 * b + 1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const int ens = __hip_atomic_load(&cnt[3 * b + 2], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      pre[2 * b + 0] = out;
      pre[2 * b + 1] = eb;
      const int lim = min(max(need_eq - eb, 0), e);
      out += s + (lim == e ? ens : ((int)b == s_bchunk ? bsel : 0));
      eb += e;
    }
    a.n_rows[r] = out;
  }
}

// Per chunk: ordered compaction of its rows of R at the chunk's offset.
__global__ __launch_bounds__(NT) void topk_write_kernel(TopkArgs a) {
  __shared__ int wsum[NWV];
  const int r = blockIdx.y;
  const ReqDev rq = a.reqs[r];
  const int T = rq.T;
  const uint32_t nb = (uint32_t)((T + kTopkChunk - 1) / kTopkChunk);
  if (blockIdx.x >= nb) return;
  const int64_t n = rq.n_reuse;
  const int64_t k = budget_dev(n, a.ratio);
  const int mode = select_mode(k, n);
  const uint32_t* st = a.sc.state + 4 * r;
  const uint32_t thr = mode == 2 ? st[0] : 0u;
  const int need_eq = mode == 2 ? (int)st[2] : 0;
  const int32_t* pre = a.sc.pre + (size_t)r * a.sc.max_chunks * 2;
  const int out0 = pre[2 * blockIdx.x + 0];
  const int eq0 = pre[2 * blockIdx.x + 1];
  const int tid = threadIdx.x;
  const int t0 = blockIdx.x * kTopkChunk + tid * TPT;
  uint32_t u[TPT];
  uint8_t f[TPT];
  load8(a.scores + rq.tok_off, a.flags + rq.tok_off, t0, T, u, f);
  bool sure[TPT], eq[TPT];
  int ne = 0;
#pragma unroll
  for (int i = 0; i < TPT; ++i) {
    const bool cand = f[i] & kFlagCandidate;
    const bool gt = mode == 2 && cand && u[i] > thr;
    eq[i] = mode == 2 && cand && u[i] == thr;
    sure[i] = (f[i] & kFlagBase) || (mode == 1 ? cand : gt);
    ne += eq[i];
  }
  int te;
  int erank = eq0 + block_excl_sum(ne, wsum, te);
  bool in[TPT];
  int ni = 0;
#pragma unroll
  for (int i = 0; i < TPT; ++i) {
    in[i] = sure[i] || (eq[i] && erank < need_eq);
    erank += eq[i];
    ni += in[i];
  }
  int ti;
  int pos = out0 + block_excl_sum(ni, wsum, ti);
  int32_t* out = a.rows + rq.tok_off;
#pragma unroll
  for (int i = 0; i < TPT; ++i) {
    if (in[i] && pos < T) out[pos] = t0 + i;   // (pos < T always holds; it keeps a write in the request)
    pos += in[i];
  }
}

}  // namespace

hipError_t launch_topk(const sx_plan* p, const float* scores, double ratio, int32_t* rows, int32_t* n_rows,
                       hipStream_t s) {
  TopkArgs a{};
  a.reqs = p->d_req;
  a.flags = p->d_flags;
  a.scores = (const uint32_t*)scores;
  a.ratio = ratio;
  a.sc = p->topk;
  a.rows = rows;
  a.n_rows = n_rows;
  const dim3 grid((unsigned)p->topk.max_chunks, (unsigned)p->n_req);
  for (int pass = 0; pass < 3; ++pass) {
    hipLaunchKernelGGL(topk_hist_kernel, grid, dim3(NT), 0, s, a, pass);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(topk_count_kernel, grid, dim3(NT), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(topk_write_kernel, grid, dim3(NT), 0, s, a);
  return hipGetLastError();
}

}  // namespace sx
