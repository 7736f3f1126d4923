// bfloat16 matrix-core kernels of the step:
//   * attention of a set of query rows over a paged or dense K/V (sparse attention of R,
//     Algorithm 1 step 21; full causal attention of the hybrid layers; and, without the PV
//     product, the log-sum-exp pass of Sparse-Q scoring, Eq. sparseq-attn);
//   * the per-key column sums of the Sparse-Q probabilities (Eq. sparseq-score).
//
// CDNA4 design (gfx950, wave64, v_mfma_f32_32x32x16_bf16):
//   * One workgroup = 4 waves = 128 query columns of one KV head; a column is a (query row,
//     query head) pair, so the G = Hq/Hkv heads that share a KV head share every K/V tile.
//   * Scores are formed transposed, S^T = K Q^T: each lane then owns one query column, so the
//     running max / sum of the online softmax stay in the lane (one cross-half exchange per tile).
//   * The output is accumulated transposed, O^T += V^T P^T: the B operand P^T is exactly the
//     lane's own S^T accumulator registers (converted to bf16), no data movement.
//   * K tiles sit in LDS row-major (padded rows, conflict-free 16-byte reads).  V tiles sit in
//     LDS as [key run of 4][d][4 keys], so the V^T A operand of a lane is two contiguous 8-byte
//     reads and each loader thread writes 64 contiguous bytes.
//   * K/V tiles are double-buffered in LDS (one barrier per tile); global loads of tile j+2 are
//     in flight while tile j is computed.
//   * The 1-D grid is decoded KV head fastest, then request, then query-row tile from the latest
//     rows (most keys) to the earliest: the heaviest tiles of every head start first, and with 8 KV
//     heads the round-robin dispatch keeps all tiles of one head on one XCD (one L2).
//   * Softmax: the running max is only raised when it grows by more than 8 (log2 units), so the
//     O^T rescale is rare; probabilities then stay below 2^8, safe in float32 and bfloat16.
#include "sx_device.h"
#include "sx_internal.h"

namespace sx {
namespace {

constexpr int KT = 64;     // keys per tile
constexpr int COLS = 128;  // query columns per workgroup (32 per wave)

struct AttnK {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* out;
  float* lse;
  const ReqDev* reqs;
  const int32_t* bt;
  const int32_t* rows;
  const int32_t* n_rows;
  const int32_t* cu;
  int Hq, Hkv, G, rpw, n_req;
  float scale_log2;
  int lse_base2;
};

__device__ __forceinline__ uint32_t lo16(uint32_t w) { return w & 0xffffu; }
__device__ __forceinline__ uint32_t hi16(uint32_t w) { return w >> 16; }

// Element c (0..7) of a 16-byte bf16 vector.
__device__ __forceinline__ uint32_t elem8(const uint4& v, int c) {
  const uint32_t w = c < 2 ? v.x : c < 4 ? v.y : c < 6 ? v.z : v.w;
  return (c & 1) ? hi16(w) : lo16(w);
}

template <int D, bool PAGED, bool PV>
__global__ __launch_bounds__(256, 2) void attn_mfma_kernel(AttnK a) {
  constexpr int KSTRIDE = D + 8;                 // padded K row (elements)
  constexpr int KVEC = KT * D / 8 / 256;         // 16-byte K vectors per loader thread
  constexpr int DV = D / 16;                     // V dims per loader thread (4 keys each)
  constexpr int KBUF = KT * KSTRIDE;
  constexpr int VBUF = PV ? KT * D : 8;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2 * KBUF];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[2 * VBUF];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int l32 = lane & 31;
  const int hg = lane >> 5;
  const int kvh = (int)(blockIdx.x % (unsigned)a.Hkv);
  const int rest = (int)(blockIdx.x / (unsigned)a.Hkv);
  const int r = rest % a.n_req;
  const int rank = rest / a.n_req;

  int T, tok_off, bt_off = 0, nrows;
  if constexpr (PAGED) {
    const ReqDev rq = a.reqs[r];
    T = rq.T;
    tok_off = rq.tok_off;
    bt_off = rq.bt_off;
    nrows = a.n_rows[r];
  } else {
    tok_off = a.cu[r];
    T = a.cu[r + 1] - tok_off;
    nrows = T;
  }
  const int rpw = a.rpw;
  const int ntiles = (nrows + rpw - 1) / rpw;
  if (rank >= ntiles) return;
  const int tile = ntiles - 1 - rank;
  const int row0 = tile * rpw;
  const int col = w * 32 + l32;
  const int lrow = col / a.G;
  const int hh = col - lrow * a.G;
  const int ridx = row0 + lrow;
  const bool valid = lrow < rpw && ridx < nrows;
  int pos = -1;
  if (valid) pos = PAGED ? a.rows[tok_off + ridx] : ridx;
  const int last = min(row0 + rpw, nrows) - 1;
  const int wg_max = PAGED ? a.rows[tok_off + last] : last;
  const int wave_max = wave_max_i(pos);
  const int wave_min = wave_min_i(valid ? pos : 0x7fffffff);
  const int nkt = wg_max / KT + 1;
  const int qh = kvh * a.G + hh;

  // Q^T as the B operand: lane owns column l32, d-slots 16s + 8hg .. +7.
  bf16x8_t qb[D / 16];
  {
    const uint16_t* qp = a.q + ((int64_t)(tok_off + (pos < 0 ? 0 : pos)) * a.Hq + (valid ? qh : 0)) * D + hg * 8;
#pragma unroll
    for (int s = 0; s < D / 16; ++s) {
      uint4 v = valid ? *(const uint4*)(qp + 16 * s) : make_uint4(0, 0, 0, 0);
      qb[s] = __builtin_bit_cast(bf16x8_t, v);
    }
  }

  f32x16_t o[PV ? D / 32 : 1];
#pragma unroll
  for (int i = 0; i < (PV ? D / 32 : 1); ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[i][e] = 0.f;
  float m_run = -INFINITY;
  float l_run = 0.f;

  // ---- tile loaders ----
  uint4 kreg[KVEC];
  uint4 vreg[4];      // 4 keys x DV dims (DV*2 bytes each, low part used when DV == 4)
  auto key_row = [&](const uint16_t* base, int key) -> const uint16_t* {
    if constexpr (PAGED) {
      const int32_t blk = a.bt[bt_off + (key >> 4)];
      return base + (((int64_t)blk * a.Hkv + kvh) * 16 + (key & 15)) * D;
    } else {
      return base + ((int64_t)(tok_off + key) * a.Hkv + kvh) * D;
    }
  };
  auto gload = [&](int kt) {
    const int kbase = kt * KT;
#pragma unroll
    for (int e = 0; e < KVEC; ++e) {
      const int vid = tid + 256 * e;
      const int key = vid / (D / 8);
      const int dc = vid - key * (D / 8);
      const int j = kbase + key;
      const uint4 t = *(const uint4*)(key_row(a.k, min(j, T - 1)) + dc * 8);   // clamped, branch-free
      kreg[e] = j < T ? t : make_uint4(0, 0, 0, 0);
    }
    if constexpr (PV) {
      const int run = tid >> 4;
      const int dc = tid & 15;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = kbase + run * 4 + i;
        const uint16_t* vp = key_row(a.v, min(j, T - 1));
        if constexpr (DV == 8) {
          const uint4 t = *(const uint4*)(vp + dc * 8);
          vreg[i] = j < T ? t : make_uint4(0, 0, 0, 0);
        } else {
          const uint2 t2 = *(const uint2*)(vp + dc * 4);
          vreg[i] = j < T ? make_uint4(t2.x, t2.y, 0, 0) : make_uint4(0, 0, 0, 0);
        }
      }
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int e = 0; e < KVEC; ++e) {
      const int vid = tid + 256 * e;
      const int key = vid / (D / 8);
      const int dc = vid - key * (D / 8);
      *(uint4*)(&Ks[buf * KBUF + key * KSTRIDE + dc * 8]) = kreg[e];
    }
    if constexpr (PV) {
      const int run = tid >> 4;
      const int dc = tid & 15;
      uint16_t* dst = &Vs[buf * VBUF + (run * D + dc * DV) * 4];
#pragma unroll
      for (int c = 0; c < DV; c += 2) {
        uint4 t;
        t.x = elem8(vreg[0], c) | (elem8(vreg[1], c) << 16);
        t.y = elem8(vreg[2], c) | (elem8(vreg[3], c) << 16);
        t.z = elem8(vreg[0], c + 1) | (elem8(vreg[1], c + 1) << 16);
        t.w = elem8(vreg[2], c + 1) | (elem8(vreg[3], c + 1) << 16);
        *(uint4*)(dst + c * 4) = t;
      }
    }
  };

  gload(0);
  lstore(0);
  if (nkt > 1) gload(1);
  __syncthreads();
  const float c2 = a.scale_log2;
  for (int kt = 0; kt < nkt; ++kt) {
    const int buf = kt & 1;
    const int kbase = kt * KT;
    if (kbase <= wave_max) {   // otherwise every column of this wave is before the tile
      const uint16_t* Kb = Ks + buf * KBUF;
      // S^T = K Q^T for the 64 keys of the tile: two 32-key M tiles
      f32x16_t sacc[2];
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
        for (int e = 0; e < 16; ++e) sacc[mt][e] = 0.f;
#pragma unroll
        for (int s = 0; s < D / 16; ++s) {
          const bf16x8_t ka = *(const bf16x8_t*)(&Kb[(mt * 32 + l32) * KSTRIDE + s * 16 + hg * 8]);
          sacc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qb[s], sacc[mt], 0, 0, 0);
        }
      }
      // lane value e of M tile mt is key kbase + 32 mt + 8 (e / 4) + 4 hg + e % 4 of the lane's column
      float x[32];
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int e = 0; e < 16; ++e) x[mt * 16 + e] = sacc[mt][e];
      if (kbase + KT - 1 > wave_min) {
        const int lim = pos - kbase - hg * 4;   // mask keys with offset > lim
#pragma unroll
        for (int i = 0; i < 32; ++i) {
          const int koff = (i >> 4) * 32 + ((i & 15) >> 2) * 8 + (i & 3);
          if (koff > lim) x[i] = -INFINITY;
        }
      }
      float mx = x[0];
#pragma unroll
      for (int i = 1; i < 32; ++i) mx = fmaxf(mx, x[i]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_tile = mx * c2;             // scaled, log2 domain (c2 > 0)
      // raise the running max only when it grows by more than 8
      const bool grow = m_tile > m_run + 8.f;
      if (__ballot(grow)) {
        const float m_new = grow ? m_tile : m_run;
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);   // m_run = -inf -> 0
        l_run *= alpha;
        if constexpr (PV) {
#pragma unroll
          for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
            for (int e = 0; e < 16; ++e) o[dt][e] *= alpha;
        }
        m_run = m_new;
      }
      const float m_use = m_run == -INFINITY ? 0.f : m_run;
      float psum = 0.f;
#pragma unroll
      for (int i = 0; i < 32; ++i) {
        x[i] = __builtin_amdgcn_exp2f(__builtin_fmaf(x[i], c2, -m_use));
        psum += x[i];
      }
      l_run += psum;
      if constexpr (PV) {
        const uint16_t* Vb = Vs + buf * VBUF;
        // P^T operand of k-step kk (16 keys) = lane values x[8kk .. 8kk+7]
        bf16x8_t pb[4];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          uint4 t;
          t.x = pack_bf16x2(x[8 * kk + 0], x[8 * kk + 1]);
          t.y = pack_bf16x2(x[8 * kk + 2], x[8 * kk + 3]);
          t.z = pack_bf16x2(x[8 * kk + 4], x[8 * kk + 5]);
          t.w = pack_bf16x2(x[8 * kk + 6], x[8 * kk + 7]);
          pb[kk] = __builtin_bit_cast(bf16x8_t, t);
        }
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) {
          const int d = dt * 32 + l32;
#pragma unroll
          for (int kk = 0; kk < 4; ++kk) {
            const uint2 lo = *(const uint2*)(&Vb[((4 * kk + hg) * D + d) * 4]);
            const uint2 hi = *(const uint2*)(&Vb[((4 * kk + 2 + hg) * D + d) * 4]);
            const bf16x8_t va = __builtin_bit_cast(bf16x8_t, make_uint4(lo.x, lo.y, hi.x, hi.y));
            o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[kk], o[dt], 0, 0, 0);
          }
        }
      }
    }
    // stage tile kt+1 (its loads were issued one iteration ago) and start loading tile kt+2;
    // the buffer written here was last read in iteration kt-1, which every wave has left
    if (kt + 1 < nkt) {
      lstore(buf ^ 1);
      if (kt + 2 < nkt) gload(kt + 2);
    }
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if constexpr (PV) {
    if (valid) {
      const float inv = 1.f / l_tot;
      uint16_t* op = a.out + ((int64_t)(tok_off + ridx) * a.Hq + qh) * D;
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int d = dt * 32 + j * 8 + hg * 4;
          uint2 t;
          t.x = pack_bf16x2(o[dt][4 * j + 0] * inv, o[dt][4 * j + 1] * inv);
          t.y = pack_bf16x2(o[dt][4 * j + 2] * inv, o[dt][4 * j + 3] * inv);
          *(uint2*)(op + d) = t;
        }
    }
  }
  if (a.lse && valid && hg == 0) {
    const float lse2 = m_run + __log2f(l_tot);
    a.lse[(int64_t)(tok_off + ridx) * a.Hq + qh] = a.lse_base2 ? lse2 : lse2 * 0.69314718055994531f;
  }
}

// Sparse-Q column sums, key-stationary: each wave owns 32 keys of one KV head (K^T held in
// registers as the A operand) and streams the probe columns (probe row, query head) 32 at a time:
// S^T = K Q^T, p = 2^(scale*log2e*s - lse2) masked causally, summed per key.  Per-lane partial
// sums are float32 over 8 column chunks and float64 beyond; the cross-lane sum at the end has a
// fixed order, so the result is deterministic.
struct ColsumK {
  const uint16_t* q;
  const uint16_t* k;
  const float* lse;
  const ReqDev* reqs;
  const int32_t* bt;
  const int32_t* probe;
  double* colsum;
  int64_t total;
  int Hq, Hkv, G, n_req;
  float scale_log2;
};

template <int D>
__global__ __launch_bounds__(256, 2) void colsum_mfma_kernel(ColsumK a) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int l32 = lane & 31;
  const int hg = lane >> 5;
  // 1-D grid: KV head fastest, then request, then key tile from the first keys (most probe rows)
  const int kvh = (int)(blockIdx.x % (unsigned)a.Hkv);
  const int rest = (int)(blockIdx.x / (unsigned)a.Hkv);
  const ReqDev rq = a.reqs[rest % a.n_req];
  const int T = rq.T;
  const int j0 = (rest / a.n_req) * 128;
  if (j0 >= T) return;
  const int jw = j0 + w * 32;
  // K rows of the wave's 32 keys as the A operand
  bf16x8_t ka[D / 16];
  {
    const int key = jw + l32;
    const uint16_t* kp = nullptr;
    if (key < T) {
      const int32_t blk = a.bt[rq.bt_off + (key >> 4)];
      kp = a.k + (((int64_t)blk * a.Hkv + kvh) * 16 + (key & 15)) * D + hg * 8;
    }
#pragma unroll
    for (int s = 0; s < D / 16; ++s) {
      uint4 v = kp ? *(const uint4*)(kp + 16 * s) : make_uint4(0, 0, 0, 0);
      ka[s] = __builtin_bit_cast(bf16x8_t, v);
    }
  }
  // first probe row that can see the workgroup's first key
  const int32_t* probe = a.probe + rq.tok_off;
  const int np = rq.n_probe;
  int lo = 0, hi = np;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (probe[mid] < jw) lo = mid + 1; else hi = mid;
  }
  const int ncols = np * a.G;
  double acc64[16];
  float acc32[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    acc64[e] = 0.0;
    acc32[e] = 0.f;
  }
  int pending = 0;
  for (int c0 = lo * a.G; c0 < ncols; c0 += 32) {
    const int c = c0 + l32;
    const bool valid = c < ncols;
    const int pidx = valid ? c / a.G : 0;
    const int h = valid ? c - pidx * a.G : 0;
    const int pos = valid ? probe[pidx] : -1;
    const float lse2 = valid ? a.lse[(int64_t)(rq.tok_off + pidx) * a.Hq + kvh * a.G + h] : INFINITY;
    const uint16_t* qp = a.q + ((int64_t)(rq.tok_off + (valid ? pos : 0)) * a.Hq + kvh * a.G + h) * D + hg * 8;
    f32x16_t s = {};
#pragma unroll
    for (int st = 0; st < D / 16; ++st) {
      uint4 v = valid ? *(const uint4*)(qp + 16 * st) : make_uint4(0, 0, 0, 0);
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[st], __builtin_bit_cast(bf16x8_t, v), s, 0, 0, 0);
    }
    // the chunk's first column has the smallest row; no mask when it sees all 32 keys
    const int first_pos = probe[c0 / a.G];
    const bool need_mask = first_pos < jw + 31;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      float p = __builtin_amdgcn_exp2f(s[e] * a.scale_log2 - lse2);
      if (need_mask) {
        const int key = jw + (e >> 2) * 8 + hg * 4 + (e & 3);
        p = key <= pos ? p : 0.f;
      }
      acc32[e] += p;
    }
    if (++pending == 8) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        acc64[e] += (double)acc32[e];
        acc32[e] = 0.f;
      }
      pending = 0;
    }
  }
#pragma unroll
  for (int e = 0; e < 16; ++e) acc64[e] += (double)acc32[e];
  // sum over the 32 columns (lanes with the same hg), fixed butterfly order
#pragma unroll
  for (int e = 0; e < 16; ++e)
#pragma unroll
    for (int o = 1; o < 32; o <<= 1) acc64[e] += __shfl_xor(acc64[e], o, 64);
  if (l32 == 0) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int key = jw + (e >> 2) * 8 + hg * 4 + (e & 3);
      if (key < T) a.colsum[(int64_t)kvh * a.total + rq.tok_off + key] = acc64[e];
    }
  }
}

template <int D, bool PAGED, bool PV>
hipError_t launch_mfma(const AttnLaunch& L, hipStream_t s) {
  AttnK a{};
  a.q = (const uint16_t*)L.q;
  a.k = (const uint16_t*)L.k;
  a.v = (const uint16_t*)L.v;
  a.out = (uint16_t*)L.out;
  a.lse = L.lse;
  a.reqs = L.reqs;
  a.bt = L.bt;
  a.rows = L.rows;
  a.n_rows = L.n_rows;
  a.cu = L.cu;
  a.Hq = L.Hq;
  a.Hkv = L.Hkv;
  a.G = L.Hq / L.Hkv;
  a.rpw = COLS / a.G;
  a.scale_log2 = L.scale * 1.4426950408889634f;
  a.lse_base2 = L.lse_base2;
  a.n_req = L.n_req;
  const int64_t ntiles = (L.grid_rows + a.rpw - 1) / a.rpw;
  const dim3 grid((unsigned)(ntiles * L.Hkv * L.n_req));
  hipLaunchKernelGGL((attn_mfma_kernel<D, PAGED, PV>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace

// float32 variants (vector ALU), defined in k_attn_f32.hip
hipError_t launch_attn_f32(const AttnLaunch& a, bool paged, hipStream_t s);
hipError_t launch_colsum_f32(const sx_plan* p, const void* q, const void* kc, hipStream_t s);

hipError_t launch_attn_paged(const AttnLaunch& a, hipStream_t s) {
  if (a.dtype == SX_F32) return launch_attn_f32(a, true, s);
  const bool pv = a.out != nullptr;
  if (a.D == 128) return pv ? launch_mfma<128, true, true>(a, s) : launch_mfma<128, true, false>(a, s);
  return pv ? launch_mfma<64, true, true>(a, s) : launch_mfma<64, true, false>(a, s);
}

hipError_t launch_attn_dense(const AttnLaunch& a, hipStream_t s) {
  if (a.dtype == SX_F32) return launch_attn_f32(a, false, s);
  if (a.D == 128) return launch_mfma<128, false, true>(a, s);
  return launch_mfma<64, false, true>(a, s);
}

hipError_t launch_colsum(const sx_plan* p, const void* q, const void* kc, hipStream_t s) {
  if (p->desc.dtype == SX_F32) return launch_colsum_f32(p, q, kc, s);
  ColsumK a{};
  a.q = (const uint16_t*)q;
  a.k = (const uint16_t*)kc;
  a.lse = p->d_lse;
  a.reqs = p->d_req;
  a.bt = p->d_bt;
  a.probe = p->d_probe;
  a.colsum = p->d_colsum;
  a.total = p->total;
  a.Hq = p->desc.n_q_heads;
  a.Hkv = p->desc.n_kv_heads;
  a.G = a.Hq / a.Hkv;
  a.scale_log2 = p->scale * 1.4426950408889634f;
  a.n_req = p->n_req;
  const dim3 grid((unsigned)(((p->max_T + 127) / 128) * a.Hkv * p->n_req));
  if (p->desc.head_dim == 128)
    hipLaunchKernelGGL(colsum_mfma_kernel<128>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(colsum_mfma_kernel<64>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace sx
