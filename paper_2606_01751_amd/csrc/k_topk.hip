// Key selection and recompute set (Eq. topk, Section 3.3, Algorithm 1 steps 14-17).
//
// Per request, k_r = min(n_r, floor(ratio * n_r + 1/2)) over the n_r reused candidates; S_key = the
// k_r candidates with the largest float32 score, ties to the lower index; R = base rows (I_nr,
// overflow, tail fallback: precomputed plan flags) U S_key, ascending.
//
// Every request is cut into chunks of kTopkChunk tokens, one 256-thread workgroup per chunk, so a
// request's selection runs on many CUs, in three launches with no counters or waits between
// workgroups.  Scores are compared through an order-preserving 32-bit key of their IEEE pattern
// (sign flip: the unsigned order of the keys is the order of the values):
//   histogram  each workgroup adds the histogram of its candidates' top 16 key bits (an LDS
//              histogram of 16-bit counters, two per word) to the request's fine histogram, and
//              the sums of its 256-bin groups to the request's coarse histogram.
//   boundary   every workgroup finds the first digit d0 of the k-th largest key from the completed
//              histograms (largest d with at least k candidates in bins >= d: the group from the
//              coarse one, the bin within it from the fine one), then records for its chunk the
//              rows surely in R (base rows, candidates whose top bits exceed d0) and, in index
//              order, the boundary candidates whose top bits equal d0 (index, base flag, key).  Its
//              first workgroup stores d0 and the candidates still needed.
//   write      every workgroup finds the last 8 + 8 key bits of the threshold from LDS histograms
//              of all boundary entries of the request, derives from the boundary entries of the
//              chunks before its own their rows above the threshold and their selected ties (a tie
//              is in R when its rank among the request's ties, index order, is below the number
//              still needed), and compacts its chunk's rows of R in order at the resulting offset.
//              The last chunk writes n_rows; the first clears the histogram bins that were used.
// With 16 bits in the first digit the boundary lists hold tens to hundreds of entries on score
// distributions that span a few binades; when many candidates share the top bits (equal scores)
// they grow to the candidates themselves, which stays correct and costs time.
// Scratch is plan-owned; calls sharing a plan must be stream-ordered.
#include "sx_device.h"
#include "sx_internal.h"

namespace sx {
namespace {

constexpr int NT = 256;                  // threads per workgroup
constexpr int TPT = kTopkChunk / NT;     // tokens per thread (consecutive)
static_assert(TPT == 8, "a thread loads 8 consecutive scores (two 16-byte vectors) and 8 flags");
constexpr int NWV = NT / 64;
constexpr int FINE = kTopkFine;          // 65536: first digit, the top 16 key bits
constexpr int COARSE = FINE / NT;        // 256 groups of 256 fine bins
static_assert(COARSE == NT, "one coarse group per thread");
constexpr uint32_t kBaseBit = 0x80000000u;   // boundary entry: the token is a base row

// order-preserving key of an IEEE float32 pattern
__device__ __forceinline__ uint32_t okey(uint32_t u) { return (u & 0x80000000u) ? ~u : (u | 0x80000000u); }
constexpr int CPT = kTopkMaxChunks / NT;     // chunk slots per thread in the chunk tables
static_assert(CPT * NT == kTopkMaxChunks, "chunk tables spread evenly over the threads");

__device__ __forceinline__ int64_t budget_dev(int64_t n, double ratio) {
#pragma clang fp contract(off)
  const double prod = ratio * (double)n;
  double k = floor(prod + 0.5);
  if (k > (double)n) k = (double)n;
  if (k < 0.0) k = 0.0;
  return (int64_t)k;
}

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

__device__ __forceinline__ int block_sum(int v, int* wsum) {
  int t;
  block_excl_sum(v, wsum, t);
  return t;
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

// Digit search over 256 bins: the largest bin d with (entries in bins >= d) >= need, and the number
// of entries in bins above d.
struct Digit {
  int d, gt;
};
// Done by wave 0 alone over the 256 bins at h (global or LDS; lane l holds bins 4l .. 4l+3), the
// answer broadcast through wsum: one barrier.  All threads call it.
__device__ Digit find_digit_w0(const uint32_t* h, int need, int* wsum) {
  const int tid = threadIdx.x;
  if (tid < 64) {
    const uint4 c4 = *(const uint4*)(h + 4 * tid);
    const int c[4] = {(int)c4.x, (int)c4.y, (int)c4.z, (int)c4.w};
    const int loc = c[0] + c[1] + c[2] + c[3];
    // entries in the bins above this lane's: suffix sum over the higher lanes
    int x = loc;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_down(x, o, 64);
      if (tid + o < 64) x += y;
    }
    int ge = x - loc;
    int best = -1, best_gt = 0;
#pragma unroll
    for (int i = 3; i >= 0; --i) {
      const int gt_i = ge;
      ge += c[i];
      if (best < 0 && ge >= need) {
        best = 4 * tid + i;
        best_gt = gt_i;
      }
    }
    int top = best >= 0 ? tid : -1;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) top = max(top, __shfl_xor(top, o, 64));
    // (no qualifying bin means fewer entries than needed: impossible when k <= n; kept defensive)
    if (top < 0 && tid == 0) {
      wsum[0] = 0;
      wsum[1] = need;
    }
    if (top >= 0 && tid == top) {
      wsum[0] = best;
      wsum[1] = best_gt;
    }
  }
  __syncthreads();
  const Digit r{wsum[0], wsum[1]};
  __syncthreads();
  return r;
}

// Histogram of the candidates' top 16 key bits (blockIdx.y = request, blockIdx.x = chunk).  LDS
// counters are 16-bit (a chunk has at most 2048 candidates), two per word: bin 2w in the low half
// of word w, bin 2w + 1 in the high half.
__global__ __launch_bounds__(NT) void topk_hist_kernel(TopkArgs a) {
  __shared__ __attribute__((aligned(16))) uint32_t hist[FINE / 2];
  __shared__ uint32_t s_grp[COARSE];   // per-group sums of this chunk
  __shared__ int s_rng[2 * NWV];
  s_grp[threadIdx.x] = 0u;   // (ordered before its use by the barriers below)
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
  // only the word range [wlo, whi] between the chunk's smallest and largest digit is cleared and
  // flushed (scores spanning a few binades touch a few hundred bins)
  uint32_t d[TPT];
  int dmin = FINE, dmax = -1;
#pragma unroll
  for (int i = 0; i < TPT; ++i) {
    d[i] = okey(u[i]) >> 16;
    if (f[i] & kFlagCandidate) {
      dmin = min(dmin, (int)d[i]);
      dmax = max(dmax, (int)d[i]);
    }
  }
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    dmin = min(dmin, __shfl_xor(dmin, o, 64));
    dmax = max(dmax, __shfl_xor(dmax, o, 64));
  }
  if ((tid & 63) == 0) {
    s_rng[tid >> 6] = dmin;
    s_rng[NWV + (tid >> 6)] = dmax;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < NWV; ++i) {
    dmin = min(dmin, s_rng[i]);
    dmax = max(dmax, s_rng[NWV + i]);
  }
  if (dmax < 0) return;   // no candidate in the chunk (uniform)
  const int wlo = dmin >> 1, whi = dmax >> 1;
  for (int w = wlo + tid; w <= whi; w += NT) hist[w] = 0u;
  __syncthreads();
#pragma unroll
  for (int i = 0; i < TPT; ++i)
    if (f[i] & kFlagCandidate) atomicAdd(&hist[d[i] >> 1], 1u << ((d[i] & 1) * 16));
  __syncthreads();
  uint32_t* gf = a.sc.hist + (size_t)r * (FINE + COARSE);
  uint32_t* gc = gf + FINE;
  for (int w = wlo + tid; w <= whi; w += NT) {
    const uint32_t v = hist[w];
    if (v) {
      const uint32_t lo = v & 0xffffu, hi = v >> 16;
      if (lo) atomicAdd(&gf[2 * w], lo);
      if (hi) atomicAdd(&gf[2 * w + 1], hi);
      atomicAdd(&s_grp[w >> 7], lo + hi);
    }
  }
  __syncthreads();
  // the coarse sums of the groups the range touches
  for (int g = (wlo >> 7) + tid; g <= (whi >> 7); g += NT) {
    const uint32_t v = s_grp[g];
    if (v) atomicAdd(&gc[g], v);
  }
}

// Per chunk: rows surely in R, and the boundary candidates (top key bits equal to d0) in index order.
__global__ __launch_bounds__(NT) void topk_bound_kernel(TopkArgs a) {
  __shared__ int wsum[2 * NWV];
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
  uint32_t u[TPT];
  uint8_t f[TPT];
  const int t0 = b * kTopkChunk + tid * TPT;
  load8(a.scores + rq.tok_off, a.flags + rq.tok_off, t0, T, u, f);
  uint32_t d0 = 0;
  if (mode == 2) {
    const uint32_t* gf = a.sc.hist + (size_t)r * (FINE + COARSE);
    const Digit g = find_digit_w0(gf + FINE, (int)k, wsum);                 // group
    const Digit fb = find_digit_w0(gf + 256 * g.d, (int)k - g.gt, wsum);    // bin within it
    d0 = (uint32_t)(256 * g.d + fb.d);
    if (b == 0 && tid == 0) {
      a.sc.state[r * 4 + 0] = d0;
      a.sc.state[r * 4 + 1] = (uint32_t)((int)k - g.gt - fb.gt);   // candidates still needed
    }
  }
  int ns = 0, nbd = 0;
  bool bd[TPT];
#pragma unroll
  for (int i = 0; i < TPT; ++i) {
    const bool cand = f[i] & kFlagCandidate;
    const bool base = f[i] & kFlagBase;
    const uint32_t top = okey(u[i]) >> 16;
    ns += (base || (mode == 1 ? cand : (mode == 2 && cand && top > d0))) ? 1 : 0;
    bd[i] = mode == 2 && cand && top == d0;
    nbd += bd[i];
  }
  const int tot_s = block_sum(ns, wsum);
  int tot_b;
  int pos = block_excl_sum(nbd, wsum, tot_b);
  // the chunk's list region: one slot per token of the chunk
  uint2* lst = a.sc.list + rq.tok_off + (size_t)b * kTopkChunk;
#pragma unroll
  for (int i = 0; i < TPT; ++i) {
    if (bd[i]) {
      lst[pos] = make_uint2((uint32_t)(t0 + i) | ((f[i] & kFlagBase) ? kBaseBit : 0u), okey(u[i]));
      ++pos;
    }
  }
  if (tid == 0) {
    int32_t* cnt = a.sc.cnt + ((size_t)r * a.sc.max_chunks + b) * 2;
    cnt[0] = tot_s;
    cnt[1] = tot_b;
  }
}

// Per chunk: the threshold's last two digits from all boundary entries, the chunk's offset in R
// from the chunks before it, then an ordered compaction of its rows of R.
__global__ __launch_bounds__(NT) void topk_write_kernel(TopkArgs a) {
  constexpr int UNR = 4;      // boundary entries per thread and step (independent loads in flight)
  constexpr int STAGE = 4096;   // boundary entries staged in LDS (more are read from global memory)
  __shared__ uint2 s_ent[STAGE];
  __shared__ __attribute__((aligned(16))) uint32_t h[256];
  __shared__ int s_off[kTopkMaxChunks + 1];   // exclusive prefix of the boundary entry counts
  __shared__ int s_sure[kTopkMaxChunks];
  __shared__ int wsum[2 * NWV];
  const int r = blockIdx.y;
  const ReqDev rq = a.reqs[r];
  const int T = rq.T;
  const int nb = (T + kTopkChunk - 1) / kTopkChunk;   // <= kTopkMaxChunks (checked on the host)
  const int b = blockIdx.x;
  if (b >= nb) return;
  const int64_t n = rq.n_reuse;
  const int64_t k = budget_dev(n, a.ratio);
  const int mode = select_mode(k, n);
  const int tid = threadIdx.x;
  uint32_t u[TPT];
  uint8_t f[TPT];
  load8(a.scores + rq.tok_off, a.flags + rq.tok_off, b * kTopkChunk + tid * TPT, T, u, f);
  // loads that do not depend on each other go first: the stored state and (first chunk) the
  // coarse bins of the histogram to clear at the end
  uint32_t* const gf = a.sc.hist + (size_t)r * (FINE + COARSE);
  const uint32_t st0 = mode == 2 ? a.sc.state[r * 4 + 0] : 0u;
  const uint32_t st1 = mode == 2 ? a.sc.state[r * 4 + 1] : 0u;
  const uint32_t used = (b == 0 && mode == 2) ? gf[FINE + tid] : 0u;
  // The first slots of every chunk's boundary list are read now, before the counts arrive (tpc
  // threads per chunk, W slots each, inside the chunk's own slots); counts past the window are
  // rare and read once the offsets are known.
  const uint2* lst = a.sc.list + rq.tok_off;
  const int tpc = nb <= NT ? NT / nb : 0;   // threads per chunk (0: no early reads)
  const int W = tpc * UNR;
  const int sp_c = tpc ? tid / tpc : nb;
  const int sp_sub = tpc ? tid - sp_c * tpc : 0;
  uint2 spec[UNR];
#pragma unroll
  for (int q = 0; q < UNR; ++q) spec[q] = make_uint2(0u, 0u);
  if (mode == 2 && sp_c < nb) {
    const int len = min(kTopkChunk, T - sp_c * kTopkChunk);
#pragma unroll
    for (int q = 0; q < UNR; ++q) {
      const int i = sp_sub + tpc * q;
      if (i < len) spec[q] = lst[(size_t)sp_c * kTopkChunk + i];
    }
  }
  // chunk tables: thread t holds chunks CPT t .. CPT t + CPT - 1
  const int32_t* cnt = a.sc.cnt + (size_t)r * a.sc.max_chunks * 2;
  int ne[CPT], loc = 0;
#pragma unroll
  for (int q = 0; q < CPT; ++q) {
    const int c = CPT * tid + q;
    s_sure[c] = c < nb ? cnt[2 * c] : 0;
    ne[q] = c < nb ? cnt[2 * c + 1] : 0;
    loc += ne[q];
  }
  int E;
  int run = block_excl_sum(loc, wsum, E);
#pragma unroll
  for (int q = 0; q < CPT; ++q) {
    s_off[CPT * tid + q] = run;
    run += ne[q];
  }
  if (tid == 0) s_off[kTopkMaxChunks] = E;
  __syncthreads();
  // boundary entry j of the request (chunk order, index order within a chunk)
  auto entry = [&](int j) -> uint2 {
    int lo = 0, hi = nb - 1;   // last chunk c with s_off[c] <= j
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_off[mid] <= j) lo = mid; else hi = mid - 1;
    }
    return lst[(size_t)lo * kTopkChunk + (j - s_off[lo])];
  };
  // the entries are read once into LDS when they fit (block-uniform choice)
  const bool staged = E <= STAGE;
  if (staged) {
    if (sp_c < nb) {
      const int c0 = s_off[sp_c], nec = s_off[sp_c + 1] - c0;
#pragma unroll
      for (int q = 0; q < UNR; ++q) {
        const int i = sp_sub + tpc * q;
        if (i < nec) s_ent[c0 + i] = spec[q];
      }
    }
    int over = 0;
#pragma unroll
    for (int q = 0; q < CPT; ++q) over |= ne[q] > W ? 1 : 0;
    if (__syncthreads_or(over)) {
      // entries past the window
      for (int j0 = 0; j0 < E; j0 += NT * UNR) {
        uint2 e[UNR];
        int jj[UNR];
#pragma unroll
        for (int q = 0; q < UNR; ++q) {
          const int j = j0 + tid + NT * q;
          jj[q] = -1;
          if (j < E) {
            int lo = 0, hi = nb - 1;
            while (lo < hi) {
              const int mid = (lo + hi + 1) >> 1;
              if (s_off[mid] <= j) lo = mid; else hi = mid - 1;
            }
            const int i = j - s_off[lo];
            if (i >= W) {
              e[q] = lst[(size_t)lo * kTopkChunk + i];
              jj[q] = j;
            }
          }
        }
#pragma unroll
        for (int q = 0; q < UNR; ++q)
          if (jj[q] >= 0) s_ent[jj[q]] = e[q];
      }
    }
    __syncthreads();
  }
  // entries j = base + stride q (q < UNR), zero past `lim`
  auto keys = [&](int base, int stride, int lim, uint32_t (&v)[UNR], uint32_t (&x)[UNR]) {
#pragma unroll
    for (int q = 0; q < UNR; ++q) {
      const int j = base + stride * q;
      const uint2 e = j < lim ? (staged ? s_ent[j] : entry(j)) : make_uint2(0u, 0u);
      x[q] = e.x;
      v[q] = e.y;
    }
  };
  uint32_t thr = 0;
  int need = 0;
  if (mode == 2) {
    const uint32_t d0 = st0;
    int rem = (int)st1;
    // key bits 8..15 over every boundary entry, then bits 0..7 over the entries matching them
    h[tid] = 0u;
    __syncthreads();
    for (int j0 = 0; j0 < E; j0 += NT * UNR) {
      uint32_t v[UNR], x[UNR];
      keys(j0 + tid, NT, E, v, x);
#pragma unroll
      for (int q = 0; q < UNR; ++q)
        if (j0 + tid + NT * q < E) atomicAdd(&h[(v[q] >> 8) & 255], 1u);
    }
    __syncthreads();
    const Digit d1 = find_digit_w0(h, rem, wsum);
    rem -= d1.gt;
    h[tid] = 0u;
    __syncthreads();
    for (int j0 = 0; j0 < E; j0 += NT * UNR) {
      uint32_t v[UNR], x[UNR];
      keys(j0 + tid, NT, E, v, x);
#pragma unroll
      for (int q = 0; q < UNR; ++q)
        if (j0 + tid + NT * q < E && ((v[q] >> 8) & 255) == (uint32_t)d1.d) atomicAdd(&h[v[q] & 255], 1u);
    }
    __syncthreads();
    const Digit d2 = find_digit_w0(h, rem, wsum);
    rem -= d2.gt;
    thr = (d0 << 16) | ((uint32_t)d1.d << 8) | (uint32_t)d2.d;
    need = rem;   // ties (candidates equal to thr) still to select, lowest indices first
  }
  // rows of R before this chunk: sure rows of the earlier chunks, boundary entries above the
  // threshold that are not base rows (base rows are counted as sure), and the selected ties that
  // are not base rows; ties of the earlier chunks, in order, for this chunk's tie ranks
  int sure_b = 0;
#pragma unroll
  for (int q = 0; q < CPT; ++q) {
    const int c = CPT * tid + q;
    sure_b += c < b ? s_sure[c] : 0;
  }
  int out0 = block_sum(sure_b, wsum);
  int ties_before = 0;
  if (mode == 2) {
    const int jb = s_off[b];
    int gt_sel = 0;
    for (int j0 = 0; j0 < jb; j0 += NT * UNR) {   // block-uniform trip count
      // this thread: UNR consecutive entries (index order within the thread, threads in order)
      uint32_t v[UNR], x[UNR];
      keys(j0 + UNR * tid, 1, jb, v, x);
      int nt_loc = 0;
#pragma unroll
      for (int q = 0; q < UNR; ++q) nt_loc += (j0 + UNR * tid + q < jb && v[q] == thr) ? 1 : 0;
      int nt;
      int rank = ties_before + block_excl_sum(nt_loc, wsum, nt);
#pragma unroll
      for (int q = 0; q < UNR; ++q) {
        const bool valid = j0 + UNR * tid + q < jb;
        const bool nb_row = !(x[q] & kBaseBit);
        const bool tie = valid && v[q] == thr;
        gt_sel += (valid && nb_row && v[q] > thr) ? 1 : 0;
        gt_sel += (tie && nb_row && rank < need) ? 1 : 0;
        rank += tie ? 1 : 0;
      }
      ties_before += nt;
    }
    out0 += block_sum(gt_sel, wsum);
  }
  // this chunk
  bool in[TPT];
  int ne_loc = 0;
  bool tie[TPT];
#pragma unroll
  for (int i = 0; i < TPT; ++i) {
    const bool cand = f[i] & kFlagCandidate;
    const bool base = f[i] & kFlagBase;
    const uint32_t key = okey(u[i]);
    tie[i] = mode == 2 && cand && key == thr;
    in[i] = base || (mode == 1 ? cand : (mode == 2 && cand && key > thr));
    ne_loc += tie[i];
  }
  int te;
  int erank = ties_before + block_excl_sum(ne_loc, wsum, te);
  int ni = 0;
#pragma unroll
  for (int i = 0; i < TPT; ++i) {
    in[i] = in[i] || (tie[i] && erank < need);
    erank += tie[i];
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
    // the histogram pass and every boundary workgroup have finished (this launch reads the stored
    // state, not the histograms): clear the used fine groups and the coarse bins for the next call
    if (used) {
      for (int i = 0; i < 64; ++i) ((uint4*)(gf + 256 * tid))[i] = make_uint4(0, 0, 0, 0);
      gf[FINE + tid] = 0u;
    }
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
  hipLaunchKernelGGL(topk_hist_kernel, grid, dim3(NT), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(topk_bound_kernel, grid, dim3(NT), 0, s, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(topk_write_kernel, grid, dim3(NT), 0, s, a);
  return hipGetLastError();
}

}  // namespace sx
