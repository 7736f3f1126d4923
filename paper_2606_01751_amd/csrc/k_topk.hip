// Key selection and recompute set (Eq. topk, Section 3.3, Algorithm 1 steps 14-17).
//
// One 1024-thread workgroup per request:
//   1. k_r = min(n_r, floor(ratio * n_r + 1/2)) over the n_r reused candidates.
//   2. Radix select of the k_r-th largest float32 score among the candidates, 8 bits per pass
//      from the most significant byte (scores are >= 0, so the IEEE bit pattern orders them).
//      Histogram counts are integer LDS atomics, aggregated per distinct bin within a wave.
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

__global__ __launch_bounds__(NT) void topk_kernel(const ReqDev* __restrict__ reqs, const uint8_t* __restrict__ flags,
                                                  const float* __restrict__ scores, double ratio,
                                                  int32_t* __restrict__ rows, int32_t* __restrict__ n_rows) {
  __shared__ uint32_t hist[256];
  __shared__ int wtot[NWV];
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
      for (int base = 0; base < T; base += NT) {
        const int t = base + tid;
        bool act = false;
        uint32_t bin = 0;
        if (t < T && (fl[t] & kFlagCandidate)) {
          const uint32_t u = sb[t];
          if ((u & mask) == prefix) {
            act = true;
            bin = (u >> shift) & 255u;
          }
        }
        // aggregate equal bins inside the wave: one LDS atomic per distinct bin
        uint64_t pending = __ballot(act);
        while (pending) {
          const int leader = __ffsll((unsigned long long)pending) - 1;
          const uint32_t lb = __shfl(bin, leader, 64);
          const uint64_t same = __ballot(act && bin == lb);
          if (lane == leader) atomicAdd(&hist[lb], (uint32_t)__popcll(same));
          if (act && bin == lb) act = false;
          pending &= ~same;
        }
      }
      __syncthreads();
      if (tid == 0) {
        int cum = 0;
        int dgt = 255;
        for (; dgt > 0; --dgt) {
          if (cum + (int)hist[dgt] >= remaining) break;
          cum += (int)hist[dgt];
        }
        s_digit = (uint32_t)dgt;
        s_rem = remaining - cum;
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
  for (int base = 0; base < T; base += NT) {
    const int t = base + tid;
    const bool in = t < T;
    const uint8_t f = in ? fl[t] : 0;
    const bool cand = f & kFlagCandidate;
    bool gt = false, eq = false;
    if (cand && mode == 2) {
      const uint32_t u = sb[t];
      gt = u > thr;
      eq = u == thr;
    }
    int eq_total;
    const int eq_rank = eq_seen + block_excl_count(eq, wtot, eq_total);
    const bool sel = mode == 1 ? cand : (gt || (eq && eq_rank < need_eq));
    const bool inR = in && ((f & kFlagBase) || sel);
    int r_total;
    const int rpos = out_count + block_excl_count(inR, wtot, r_total);
    if (inR) out[rpos] = t;
    eq_seen += eq_total;
    out_count += r_total;
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
