// Key selection and recompute set (Eq. topk, Section 3.3, Algorithm 1 steps 14-17).
//
// One 1024-thread workgroup per request:
//   1. k_r = min(n_r, floor(ratio * n_r + 1/2)) over the n_r reused candidates.
//   2. Radix select of the k_r-th largest float32 score among the candidates, 8 bits per pass
//      from the most significant byte (scores are >= 0, so the IEEE bit pattern orders them).
//      Histogram counts are integer LDS atomics, aggregated per distinct bin within a wave.
//      Each thread loads the scores and flags of UNR rounds before using them, so the passes
//      pay one load latency per UNR rounds of 1024 tokens.
//   3. One ordered pass over the tokens: a candidate is selected when its score is above the
//      threshold, or equal to it and among the first (lowest-index) equal candidates still
//      needed.  R = base rows (I_nr, overflow, tail fallback, precomputed in the plan) U
//      selected, compacted in ascending order with wave ballots and a block prefix sum.
#include "sx_device.h"
#include "sx_internal.h"

namespace sx {
namespace {

constexpr int NT = 1024;
constexpr int NWV = NT / 64;
constexpr int UNR = 8;    // rounds of NT tokens whose loads are issued together

__device__ __forceinline__ int64_t budget_dev(int64_t n, double ratio) {
#pragma clang fp contract(off)
  const double prod = ratio * (double)n;
  double k = floor(prod + 0.5);
  if (k > (double)n) k = (double)n;
  if (k < 0.0) k = 0.0;
  return (int64_t)k;
}

// Exclusive prefix count of `pred` over the workgroup in thread order, plus the total.
__device__ __forceinline__ int block_excl_count(bool pred, int* wtot, int& total) {
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  const uint64_t b = __ballot(pred);
  const int in_wave = __popcll(b & ((lane == 0) ? 0ull : (~0ull >> (64 - lane))));
  if (lane == 0) wtot[wv] = __popcll(b);
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < NWV; ++i) {
    const int c = wtot[i];
    before += i < wv ? c : 0;
    tot += c;
  }
  __syncthreads();
  total = tot;
  return before + in_wave;
}

// The same for two predicates with one pair of barriers: returns the exclusive prefix count of
// p1 (total in total1) and gives that of p2 in before2 / total2.
__device__ __forceinline__ int block_excl_count2(bool p1, bool p2, int* wtot, int& total1, int& before2,
                                                 int& total2) {
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const uint64_t b1 = __ballot(p1), b2 = __ballot(p2);
  if (lane == 0) {
    wtot[wv] = __popcll(b1);
    wtot[NWV + wv] = __popcll(b2);
  }
  __syncthreads();
  int bef1 = 0, tot1 = 0, bef2 = 0, tot2 = 0;
#pragma unroll
  for (int i = 0; i < NWV; ++i) {
    const int c1 = wtot[i], c2 = wtot[NWV + i];
    bef1 += i < wv ? c1 : 0;
    bef2 += i < wv ? c2 : 0;
    tot1 += c1;
    tot2 += c2;
  }
  __syncthreads();
  total1 = tot1;
  total2 = tot2;
  before2 = bef2 + __popcll(b2 & below);
  return bef1 + __popcll(b1 & below);
}

__global__ __launch_bounds__(NT) void topk_kernel(const ReqDev* __restrict__ reqs, const uint8_t* __restrict__ flags,
                                                  const float* __restrict__ scores, double ratio,
                                                  int32_t* __restrict__ rows, int32_t* __restrict__ n_rows) {
  __shared__ uint32_t hist[256];
  __shared__ int wtot[2 * NWV];
  __shared__ uint32_t s_digit;
  __shared__ int s_rem;
  const ReqDev rq = reqs[blockIdx.x];
  const int T = rq.T;
  const int off = rq.tok_off;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int64_t n = rq.n_reuse;
  const int64_t k = budget_dev(n, ratio);
  const uint8_t* fl = flags + off;
  const uint32_t* sb = (const uint32_t*)(scores + off);

  // mode: 0 none selected, 1 all candidates, 2 threshold + ties
  int mode = k == 0 ? 0 : (k == n ? 1 : 2);
  uint32_t prefix = 0, mask = 0;
  int remaining = (int)k;
  if (mode == 2) {
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int i = tid; i < 256; i += NT) hist[i] = 0;
      __syncthreads();
      for (int base = 0; base < T; base += NT * UNR) {
        // the loads of UNR rounds first, so their latencies overlap
        uint8_t fv[UNR];
        uint32_t uv[UNR];
#pragma unroll
        for (int i = 0; i < UNR; ++i) {
          const int t = base + i * NT + tid;
          fv[i] = t < T ? fl[t] : 0;
          uv[i] = t < T ? sb[t] : 0u;
        }
#pragma unroll
        for (int i = 0; i < UNR; ++i) {
          bool act = (fv[i] & kFlagCandidate) && (uv[i] & mask) == prefix;
          const uint32_t bin = (uv[i] >> shift) & 255u;
          // one LDS atomic for the wave when every active lane has the same bin (the common
          // case for the high digits, where a per-lane atomic would serialise on one address);
          // otherwise one atomic per lane
          const uint64_t pending = __ballot(act);
          if (!pending) continue;
          const int first = __ffsll((unsigned long long)pending) - 1;
          const uint32_t b0 = __shfl(bin, first, 64);
          const uint64_t same0 = __ballot(act && bin == b0);
          if (same0 == pending) {
            if (lane == first) atomicAdd(&hist[b0], (uint32_t)__popcll(same0));
          } else if (act) {
            atomicAdd(&hist[bin], 1u);
          }
        }
      }
      __syncthreads();
      if (tid < 64) {
        // digit = the largest d with (count of bins >= d) >= remaining (0 if none); lane l holds
        // bins 4l .. 4l + 3, a suffix scan over the lanes gives the counts above each lane
        int c[4], loc = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          c[i] = (int)hist[4 * lane + i];
          loc += c[i];
        }
        int suf = loc;   // bins >= 4 lane
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int v = __shfl_down(suf, o, 64);
          if (lane + o < 64) suf += v;
        }
        int ge = suf - loc;   // bins > 4 lane + 3
        int best = -1, best_gt = 0;
#pragma unroll
        for (int i = 3; i >= 0; --i) {
          const int gt_i = ge;   // bins > 4 lane + i
          ge += c[i];
          if (best < 0 && ge >= remaining) {
            best = 4 * lane + i;
            best_gt = gt_i;
          }
        }
        const int d = wave_max_i(best);
        if (d < 0) {
          if (lane == 0) {   // fewer matching candidates than needed: keep digit 0
            s_digit = 0u;
            s_rem = remaining - (suf - c[0]);
          }
        } else if (best == d) {
          s_digit = (uint32_t)d;
          s_rem = remaining - best_gt;
        }
      }
      __syncthreads();
      prefix |= s_digit << shift;
      mask |= 255u << shift;
      remaining = s_rem;
      __syncthreads();
    }
  }
  const uint32_t thr = prefix;
  const int need_eq = remaining;   // equal-to-threshold candidates to take, lowest index first

  int out_count = 0;
  int eq_seen = 0;
  int32_t* out = rows + off;
  for (int base0 = 0; base0 < T; base0 += NT * UNR) {
    uint8_t fv[UNR];
    uint32_t uv[UNR];
#pragma unroll
    for (int i = 0; i < UNR; ++i) {
      const int t = base0 + i * NT + tid;
      fv[i] = t < T ? fl[t] : 0;
      uv[i] = t < T ? sb[t] : 0u;
    }
#pragma unroll
    for (int i = 0; i < UNR; ++i) {
      const int base = base0 + i * NT;
      if (base >= T) break;
      const int t = base + tid;
      const bool in = t < T;
      const uint8_t f = fv[i];
      const bool cand = f & kFlagCandidate;
      bool gt = false, eq = false;
      if (cand && mode == 2) {
        gt = uv[i] > thr;
        eq = uv[i] == thr;
      }
      // rows in R whatever the tie decision: base rows, and candidates above the threshold (all
      // candidates when every one is selected)
      const bool sure = in && ((f & kFlagBase) || (mode == 1 ? cand : gt));
      int eq_total, sure_before, sure_total;
      const int eq_before = block_excl_count2(eq, sure, wtot, eq_total, sure_before, sure_total);
      if (eq_total == 0) {   // no tied candidate in this round (block-uniform): one scan suffices
        if (sure) out[out_count + sure_before] = t;
        out_count += sure_total;
        continue;
      }
      const int eq_rank = eq_seen + eq_before;
      const bool inR = sure || (eq && eq_rank < need_eq);
      int r_total;
      const int rpos = out_count + block_excl_count(inR, wtot, r_total);
      if (inR) out[rpos] = t;
      eq_seen += eq_total;
      out_count += r_total;
    }
  }
  if (tid == 0) n_rows[blockIdx.x] = out_count;
}

}  // namespace

hipError_t launch_topk(const sx_plan* p, const float* scores, double ratio, int32_t* rows, int32_t* n_rows,
                       hipStream_t s) {
  hipLaunchKernelGGL(topk_kernel, dim3((unsigned)p->n_req), dim3(NT), 0, s, p->d_req, p->d_flags, scores, ratio,
                     rows, n_rows);
  return hipGetLastError();
}

}  // namespace sx
