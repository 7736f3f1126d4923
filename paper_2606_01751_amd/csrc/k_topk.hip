// Key selection and recompute set (Eq. topk, Section 3.3, Algorithm 1 steps 14-17).
//
// Per request, k_r = min(n_r, floor(ratio * n_r + 1/2)) over the n_r reused candidates; S_key = the
// k_r candidates with the largest float32 score, ties to the lower index; R = base rows (I_nr,
// overflow, tail fallback: precomputed plan flags) U S_key, ascending.
//
// Every request is cut into chunks of kTopkChunk tokens, one 256-thread workgroup per chunk, so a
// request's selection runs on many CUs, in five launches with no counters or waits between
// workgroups:
//   passes 0-2  radix select of the k_r-th largest score among the candidates, 11 + 11 + 10 bits from
//               the most significant (scores are >= 0, so the IEEE bit pattern orders them): each
//               workgroup adds the LDS histogram of its candidates that match the digits found so far
//               to the request's histogram of the pass.  Pass p first finds digit p-1 itself from
//               pass p-1's histogram (complete once the previous launch ended); its first workgroup
//               stores the digits for the later launches.
//   count       the last digit from pass 2's histogram, then per chunk the rows surely in R (base rows
//               and candidates above the threshold), the candidates equal to it (ties) and the ties
//               that are not sure rows.
//   write       per chunk: its offset in R and first tie rank from the counts of the chunks before it
//               (the chunks after the one in which the tie budget runs out rescan that chunk), then
//               an ordered compaction of its rows of R; a tie is in R when its rank among the
//               request's ties (index order) is below the tie budget.  The first chunk clears the
//               request's histograms for the next call.
// Scratch is plan-owned; calls sharing a plan must be stream-ordered.
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

struct TopkArgs {
  const ReqDev* reqs;
  const uint8_t* flags;
  const uint32_t* scores;   // float32 bit patterns
  double ratio;
  TopkScratch sc;
  int32_t* rows;
  int32_t* n_rows;
};

// Selection state after some digits: the digits found (prefix), their bit mask, and how many
// candidates matching them are still to be selected.
struct SelState {
  uint32_t prefix, mask;
  int remaining;
};

// The digit of pass p from the request's completed histogram of that pass (every workgroup computes
// the same answer): the largest d with (matching candidates in bins >= d) >= remaining.  Thread t
// holds bins 8t .. 8t+7 (pass 2 has 1024 bins: the upper half stays empty).  All threads call it.
__device__ SelState next_digit(const uint32_t* gh, SelState in, int p, int* wsum) {
  constexpr int per = NBINS / NT;
  const int tid = threadIdx.x;
  uint32_t c[per];
  int loc = 0;
  const uint4 a0 = *(const uint4*)(gh + per * tid);
  const uint4 a1 = *(const uint4*)(gh + per * tid + 4);
  c[0] = a0.x; c[1] = a0.y; c[2] = a0.z; c[3] = a0.w;
  c[4] = a1.x; c[5] = a1.y; c[6] = a1.z; c[7] = a1.w;
#pragma unroll
  for (int i = 0; i < per; ++i) loc += (int)c[i];
  int total;
  const int below = block_excl_sum(loc, wsum, total);   // bins of lower threads
  int ge = total - below - loc;                         // bins above this thread's
  int best = -1, best_gt = 0;
#pragma unroll
  for (int i = per - 1; i >= 0; --i) {
    const int gt_i = ge;
    ge += (int)c[i];
    if (best < 0 && ge >= in.remaining) {
      best = per * tid + i;
      best_gt = gt_i;
    }
  }
  // qualifying digits are exactly those <= the answer: it is the best of the highest thread that
  // has one; broadcast (digit, candidates above it) through LDS
  int top = best >= 0 ? tid : -1;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) top = max(top, __shfl_xor(top, o, 64));
  if ((tid & 63) == 0) wsum[tid >> 6] = top;
  __syncthreads();
  top = -1;
#pragma unroll
  for (int i = 0; i < NWV; ++i) top = max(top, wsum[i]);
  __syncthreads();
  if (top >= 0 && tid == top) {
    wsum[0] = best;
    wsum[1] = best_gt;
  }
  __syncthreads();
  // (no qualifying digit means fewer matching candidates than still needed: impossible when
  // k <= n; kept defensive)
  const int d = top >= 0 ? wsum[0] : 0;
  const int gt = top >= 0 ? wsum[1] : in.remaining;
  __syncthreads();
  const int shift = pass_shift(p);
  return SelState{in.prefix | ((uint32_t)d << shift), in.mask | ((pass_bins(p) - 1) << shift), in.remaining - gt};
}

__device__ __forceinline__ void store_state(uint32_t* st, SelState s) {
  st[0] = s.prefix;
  st[1] = s.mask;
  st[2] = (uint32_t)s.remaining;
}
__device__ __forceinline__ SelState load_state(const uint32_t* st) {
  return SelState{st[0], st[1], (int)st[2]};
}

// Radix pass p over every chunk of every request (blockIdx.y = request, blockIdx.x = chunk).  The
// digits of the earlier passes come from the state the previous launch's first workgroup stored
// and from pass p-1's histogram, completed by the previous launch.
__global__ __launch_bounds__(NT) void topk_hist_kernel(TopkArgs a, int p) {
  __shared__ uint32_t hist[NBINS];
  __shared__ int wsum[2 * NWV];
  const int r = blockIdx.y;
  const ReqDev rq = a.reqs[r];
  const int T = rq.T;
  const uint32_t nb = (uint32_t)((T + kTopkChunk - 1) / kTopkChunk);
  if (blockIdx.x >= nb) return;
  const int64_t n = rq.n_reuse;
  const int64_t k = budget_dev(n, a.ratio);
  if (select_mode(k, n) != 2) return;
  const int tid = threadIdx.x;
  uint32_t u[TPT];
  uint8_t f[TPT];
  load8(a.scores + rq.tok_off, a.flags + rq.tok_off, blockIdx.x * kTopkChunk + tid * TPT, T, u, f);
  for (int i = tid; i < NBINS; i += NT) hist[i] = 0u;
  SelState s{0u, 0u, (int)k};
  if (p > 0) {
    if (p == 2) s = load_state(a.sc.state + (r * 3 + 0) * 4);   // digit 0, stored by pass 1
    s = next_digit(a.sc.hist + ((size_t)r * 3 + (p - 1)) * NBINS, s, p - 1, wsum);
    if (blockIdx.x == 0 && tid == 0) store_state(a.sc.state + (r * 3 + (p - 1)) * 4, s);
  }
  __syncthreads();
  const int shift = pass_shift(p);
  const uint32_t bins = pass_bins(p);
#pragma unroll
  for (int i = 0; i < TPT; ++i) {
    if ((f[i] & kFlagCandidate) && (u[i] & s.mask) == s.prefix) atomicAdd(&hist[(u[i] >> shift) & (bins - 1)], 1u);
  }
  __syncthreads();
  uint32_t* gh = a.sc.hist + ((size_t)r * 3 + p) * NBINS;
  for (int i = tid; i < (int)bins; i += NT) {
    const uint32_t c = hist[i];
    if (c) atomicAdd(&gh[i], c);
  }
}

// Per chunk: rows surely in R (base rows, candidates above the threshold), ties (candidates equal
// to it) and ties that are not sure rows.  The threshold's last digit comes from pass 2's
// histogram; the first workgroup stores the final state.
__global__ __launch_bounds__(NT) void topk_count_kernel(TopkArgs a) {
  __shared__ int wsum[2 * NWV];
  const int r = blockIdx.y;
  const ReqDev rq = a.reqs[r];
  const int T = rq.T;
  const uint32_t nb = (uint32_t)((T + kTopkChunk - 1) / kTopkChunk);
  if (blockIdx.x >= nb) return;
  const int64_t n = rq.n_reuse;
  const int64_t k = budget_dev(n, a.ratio);
  const int mode = select_mode(k, n);
  const int tid = threadIdx.x;
  uint32_t u[TPT];
  uint8_t f[TPT];
  load8(a.scores + rq.tok_off, a.flags + rq.tok_off, blockIdx.x * kTopkChunk + tid * TPT, T, u, f);
  SelState s{0u, 0u, 0};
  if (mode == 2) {
    s = next_digit(a.sc.hist + ((size_t)r * 3 + 2) * NBINS, load_state(a.sc.state + (r * 3 + 1) * 4), 2, wsum);
    if (blockIdx.x == 0 && tid == 0) store_state(a.sc.state + (r * 3 + 2) * 4, s);
  }
  const uint32_t thr = s.prefix;
  int ns = 0, ne = 0, nens = 0;
#pragma unroll
  for (int i = 0; i < TPT; ++i) {
    const bool cand = f[i] & kFlagCandidate;
    const bool gt = mode == 2 && cand && u[i] > thr;
    const bool eq = mode == 2 && cand && u[i] == thr;
    const bool sure = (f[i] & kFlagBase) || (mode == 1 ? cand : gt);
    ns += sure;
    ne += eq;
    nens += eq && !sure;
  }
  int ts, te, tens;
  block_excl_sum(ns, wsum, ts);
  block_excl_sum(ne, wsum, te);
  block_excl_sum(nens, wsum, tens);
  if (tid == 0) {
    int32_t* cnt = a.sc.cnt + ((size_t)r * a.sc.max_chunks + blockIdx.x) * 3;
    cnt[0] = ts;
    cnt[1] = te;
    cnt[2] = tens;
  }
}

// Per chunk: the chunk's offset in R and its first tie rank from the counts of the chunks before it
// (the one chunk in which the tie budget runs out is rescanned by the chunks after it), then an
// ordered compaction of its rows of R.  The last chunk writes n_rows; the first clears the
// request's histograms for the next call.
__global__ __launch_bounds__(NT) void topk_write_kernel(TopkArgs a) {
  __shared__ int wsum[2 * NWV];
  __shared__ int s_pre[4];
  const int r = blockIdx.y;
  const ReqDev rq = a.reqs[r];
  const int T = rq.T;
  const uint32_t nb = (uint32_t)((T + kTopkChunk - 1) / kTopkChunk);
  const uint32_t b = blockIdx.x;
  if (b >= nb) return;
  const int64_t n = rq.n_reuse;
  const int64_t k = budget_dev(n, a.ratio);
  const int mode = select_mode(k, n);
  const int tid = threadIdx.x;
  const uint32_t* sb = a.scores + rq.tok_off;
  const uint8_t* fl = a.flags + rq.tok_off;
  const SelState s = mode == 2 ? load_state(a.sc.state + (r * 3 + 2) * 4) : SelState{0u, 0u, 0};
  const uint32_t thr = s.prefix;
  const int need_eq = s.remaining;
  auto classify = [&](uint32_t u, uint8_t f, bool& sure, bool& eq) {
    const bool cand = f & kFlagCandidate;
    const bool gt = mode == 2 && cand && u > thr;
    eq = mode == 2 && cand && u == thr;
    sure = (f & kFlagBase) || (mode == 1 ? cand : gt);
  };
  uint32_t u[TPT];
  uint8_t f[TPT];
  load8(sb, fl, b * kTopkChunk + tid * TPT, T, u, f);
  // counts of the chunks before this one (this chunk's own counts past the end of the loop)
  const int32_t* cnt = a.sc.cnt + (size_t)r * a.sc.max_chunks * 3;
  int sure_before = 0, eq_before = 0, ens_before = 0;
  for (uint32_t c = tid; c < nb; c += NT) {
    if (c < b) {
      sure_before += cnt[3 * c + 0];
      eq_before += cnt[3 * c + 1];
    }
  }
  int tot;
  block_excl_sum(sure_before, wsum, tot);
  sure_before = tot;
  block_excl_sum(eq_before, wsum, tot);
  eq_before = tot;
  // selected ties of earlier chunks that are not sure rows: every such tie of a chunk wholly under
  // the budget, none of a chunk wholly over it, and in the straddling chunk those of rank < budget
  // (found by rescanning it)
  if (tid == 0) {
    int eb = 0, add = 0, bchunk = -1, blim = 0;
    for (uint32_t c = 0; c < b; ++c) {
      const int e = cnt[3 * c + 1];
      const int lim = min(max(need_eq - eb, 0), e);
      if (lim == e) add += cnt[3 * c + 2];
      else if (lim > 0) {
        bchunk = (int)c;
        blim = lim;
      }
      eb += e;
    }
    s_pre[0] = add;
    s_pre[1] = bchunk;
    s_pre[2] = blim;
  }
  __syncthreads();
  ens_before = s_pre[0];
  const int bchunk = s_pre[1], blim = s_pre[2];
  if (bchunk >= 0) {   // block-uniform
    uint32_t ub[TPT];
    uint8_t fb[TPT];
    load8(sb, fl, bchunk * kTopkChunk + tid * TPT, T, ub, fb);
    bool se[TPT], ee[TPT];
    int e_loc = 0;
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      classify(ub[i], fb[i], se[i], ee[i]);
      e_loc += ee[i];
    }
    int e_tot;
    int rank = block_excl_sum(e_loc, wsum, e_tot);
    int mine = 0;
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      if (ee[i]) {
        mine += (!se[i] && rank < blim) ? 1 : 0;
        ++rank;
      }
    }
    int bsel;
    block_excl_sum(mine, wsum, bsel);
    ens_before += bsel;
  }
  const int out0 = sure_before + ens_before;
  // this chunk
  bool sure[TPT], eq[TPT];
  int ne = 0;
#pragma unroll
  for (int i = 0; i < TPT; ++i) {
    classify(u[i], f[i], sure[i], eq[i]);
    ne += eq[i];
  }
  int te;
  int erank = eq_before + block_excl_sum(ne, wsum, te);
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
  const int t0 = b * kTopkChunk + tid * TPT;
#pragma unroll
  for (int i = 0; i < TPT; ++i) {
    if (in[i] && pos < T) out[pos] = t0 + i;   // (pos < T always holds; it keeps a write in the request)
    pos += in[i];
  }
  if (b == nb - 1 && tid == 0) a.n_rows[r] = out0 + ti;
  if (b == 0 && mode == 2) {
    // every launch that reads the histograms has finished: clear them for the next call
    uint32_t* gh = a.sc.hist + (size_t)r * 3 * NBINS;
    for (int i = tid; i < 3 * NBINS; i += NT) gh[i] = 0u;
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
