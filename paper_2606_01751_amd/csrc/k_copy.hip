// Bandwidth-bound passes: RoPE re-alignment of cached segments (Section 3.1, Algorithm 1 step 6),
// KV write of fresh rows (Algorithm 1 step 19) and the cross-head sum of the Sparse-Q scores.
//
// Every thread moves 16-byte vectors; consecutive threads cover consecutive 16-byte pieces of one
// (block, head) row of the pool, so each wavefront touches whole 128-256 byte runs.
#include <type_traits>

#include "sx_device.h"
#include "sx_internal.h"

namespace sx {
namespace {

// One RoPE pair, float32, no contraction: x1' = x1*c - x2*s, x2' = x2*c + x1*s.
__device__ __forceinline__ void rot(float x1, float x2, float c, float s, float& y1, float& y2) {
#pragma clang fp contract(off)
  y1 = x1 * c - x2 * s;
  y2 = x2 * c + x1 * s;
}

// Unpack a 16-byte vector into float32 lanes.
template <bool BF16>
__device__ __forceinline__ void unpack(const uint4& v, float* f) {
  if constexpr (BF16) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = bf16_lo(w[i]);
      f[2 * i + 1] = bf16_hi(w[i]);
    }
  } else {
    f[0] = __uint_as_float(v.x);
    f[1] = __uint_as_float(v.y);
    f[2] = __uint_as_float(v.z);
    f[3] = __uint_as_float(v.w);
  }
}

template <bool BF16>
__device__ __forceinline__ uint4 pack(const float* f) {
  uint4 v;
  if constexpr (BF16) {
    v.x = pack_bf16x2(f[0], f[1]);
    v.y = pack_bf16x2(f[2], f[3]);
    v.z = pack_bf16x2(f[4], f[5]);
    v.w = pack_bf16x2(f[6], f[7]);
  } else {
    v.x = __float_as_uint(f[0]);
    v.y = __float_as_uint(f[1]);
    v.z = __float_as_uint(f[2]);
    v.w = __float_as_uint(f[3]);
  }
  return v;
}

// Thread work unit: VEC RoPE pairs of one head of one reused token (two 16-byte K vectors) plus
// the same 32 bytes of its V row.
template <int D, bool BF16, bool NEOX>
__global__ __launch_bounds__(256) void realign_kernel(const RealignRow* __restrict__ rows, int64_t n_rows,
                                                      const float2* __restrict__ cs,
                                                      const void* __restrict__ src_k_, const void* __restrict__ src_v_,
                                                      void* __restrict__ kc_, void* __restrict__ vc_, int Hkv) {
  constexpr int ESZ = BF16 ? 2 : 4;
  constexpr int VEC = 16 / ESZ;         // elements per 16-byte vector
  constexpr int UPH = D / (2 * VEC);    // units per head
  const char* src_k = (const char*)src_k_;
  const char* src_v = (const char*)src_v_;
  char* kc = (char*)kc_;
  char* vc = (char*)vc_;
  const int units = Hkv * UPH;
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t row = g / units;
  if (row >= n_rows) return;
  const int u = (int)(g - row * units);
  const int head = u / UPH;
  const int ui = u - head * UPH;
  const RealignRow rr = rows[row];
  const int64_t so = pool_off(rr.src_slot, head, Hkv, D) * ESZ;
  const int64_t dof = pool_off(rr.dst_slot, head, Hkv, D) * ESZ;
  // element ranges of the two K vectors and of the V piece
  int64_t e0, e1;
  if constexpr (NEOX) {
    e0 = (int64_t)ui * VEC;             // x1 = element i, x2 = element i + D/2
    e1 = e0 + D / 2;
  } else {
    e0 = (int64_t)ui * 2 * VEC;         // adjacent pairs (2i, 2i+1) inside 2*VEC elements
    e1 = e0 + VEC;
  }
  const int64_t v0 = (int64_t)ui * 2 * VEC;
  const uint4 ka = *(const uint4*)(src_k + so + e0 * ESZ);
  const uint4 kb = *(const uint4*)(src_k + so + e1 * ESZ);
  const uint4 va = *(const uint4*)(src_v + so + v0 * ESZ);
  const uint4 vb = *(const uint4*)(src_v + so + (v0 + VEC) * ESZ);
  const float2* csr = cs + (int64_t)rr.cs_row * (D / 2) + (int64_t)ui * VEC;
  float2 c[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) c[e] = csr[e];
  float fa[VEC], fb[VEC], ya[VEC], yb[VEC];
  unpack<BF16>(ka, fa);
  unpack<BF16>(kb, fb);
  if constexpr (NEOX) {
#pragma unroll
    for (int e = 0; e < VEC; ++e) rot(fa[e], fb[e], c[e].x, c[e].y, ya[e], yb[e]);
  } else {
    // pair p = ui*VEC + e lives at (2p, 2p+1): inside fa for e < VEC/2, inside fb otherwise
#pragma unroll
    for (int e = 0; e < VEC / 2; ++e) {
      rot(fa[2 * e], fa[2 * e + 1], c[e].x, c[e].y, ya[2 * e], ya[2 * e + 1]);
      rot(fb[2 * e], fb[2 * e + 1], c[VEC / 2 + e].x, c[VEC / 2 + e].y, yb[2 * e], yb[2 * e + 1]);
    }
  }
  *(uint4*)(kc + dof + e0 * ESZ) = pack<BF16>(ya);
  *(uint4*)(kc + dof + e1 * ESZ) = pack<BF16>(yb);
  *(uint4*)(vc + dof + v0 * ESZ) = va;
  *(uint4*)(vc + dof + (v0 + VEC) * ESZ) = vb;
}

// Copies 16-byte pieces of fresh K and V rows into their cache slots: the first
// min(n_rows, max_rows) listed rows of each request (rows == NULL: every token).
__global__ __launch_bounds__(256) void scatter_kernel(const ReqDev* __restrict__ reqs, const int32_t* __restrict__ bt,
                                                      const int32_t* __restrict__ rows,
                                                      const int32_t* __restrict__ n_rows, int max_rows,
                                                      const uint4* __restrict__ k_new, const uint4* __restrict__ v_new,
                                                      uint4* __restrict__ kc, uint4* __restrict__ vc, int Hkv,
                                                      int upr /*16-byte units per token row*/, int uph /*per head*/) {
  const ReqDev rq = reqs[blockIdx.y];
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t idx = g / upr;
  const int n = rows ? n_rows[blockIdx.y] : rq.T;
  if (idx >= n || idx >= max_rows) return;
  const int u = (int)(g - idx * upr);
  const int t = rows ? rows[rq.tok_off + idx] : (int)idx;
  const int head = u / uph;
  const int hu = u - head * uph;
  const int64_t src = ((int64_t)rq.tok_off + t) * upr + u;
  const int32_t blk = bt[rq.bt_off + (t >> 4)];
  const int64_t dst = ((((int64_t)blk * Hkv + head) * 16) + (t & 15)) * uph + hu;
  kc[dst] = k_new[src];
  vc[dst] = v_new[src];
}

// Marks the listed rows of every request with the call's generation number (no clearing pass:
// a token belongs to the current row set iff its mark equals the generation).
__global__ __launch_bounds__(256) void mark_rows_kernel(const ReqDev* __restrict__ reqs, const int32_t* __restrict__ rows,
                                                        const int32_t* __restrict__ n_rows, int max_rows,
                                                        uint32_t* __restrict__ mark, uint32_t gen) {
  const ReqDev rq = reqs[blockIdx.y];
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= max_rows || idx >= n_rows[blockIdx.y]) return;
  const int t = rows[rq.tok_off + idx];
  if (t >= 0 && t < rq.T) mark[rq.tok_off + t] = gen;
}

__global__ __launch_bounds__(256) void fill_u32_kernel(uint32_t* __restrict__ p, int64_t n, uint32_t v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ __launch_bounds__(256) void fill_u8_kernel(uint8_t* __restrict__ p, int64_t n, uint8_t v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// Sets mask[off_r + t] = 1 for every listed row t of every request (the mask was cleared first).
__global__ __launch_bounds__(256) void mask_rows_kernel(const ReqDev* __restrict__ reqs, const int32_t* __restrict__ rows,
                                                        const int32_t* __restrict__ n_rows, int max_rows,
                                                        uint8_t* __restrict__ mask) {
  const ReqDev rq = reqs[blockIdx.y];
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= max_rows || idx >= n_rows[blockIdx.y]) return;
  const int t = rows[rq.tok_off + idx];
  if (t >= 0 && t < rq.T) mask[rq.tok_off + t] = 1;
}

// Per-layer pointers of one launch of the one-pass re-alignment + KV write, passed by value.
constexpr int kLayersPerLaunch = 16;
struct LayerTable {
  sx_layer_kv l[kLayersPerLaunch];
};

// Re-alignment and KV write in one pass (Algorithm 1 steps 6 and 19-20 for sparse layers whose row
// set R is known): every token's cache slot is written once -- the fresh K/V row if the token is
// in R, else the re-aligned cached row if the token is reused; other tokens are not touched.
// blockIdx.y selects the layer.  Thread work unit: VEC RoPE pairs (two 16-byte K vectors) plus
// the same 32 bytes of V, for HPT heads of one token; the unit's cos/sin values are loaded once
// for its heads.  Threads are ordered unit fastest, then token, then head group, so for each head
// a wavefront covers 64 / UPH consecutive tokens: consecutive slots of a (block, head) run of
// the pool, i.e. contiguous runs of the source and destination caches.
// Membership of a token in R: MASK = a caller's byte mask (nonzero = in R), else the plan's
// generation marks (mark == gen).  The token's record (destination slot, source slot, cos/sin row)
// and its membership are independent loads, so every row transfer waits for one load level.
template <int D, bool BF16, bool NEOX, bool MASK, int HPT>
__global__ __launch_bounds__(256) void realign_scatter_kernel(
    const RealignRow* __restrict__ tok_row, const float2* __restrict__ cs, const uint32_t* __restrict__ mark,
    const uint8_t* __restrict__ sel, uint32_t gen, int64_t total, const LayerTable tab, int Hkv) {
  constexpr int ESZ = BF16 ? 2 : 4;
  constexpr int VEC = 16 / ESZ;
  constexpr int UPH = D / (2 * VEC);
  const sx_layer_kv& lay = tab.l[blockIdx.y];
  char* kc = (char*)lay.k_cache;
  char* vc = (char*)lay.v_cache;
  // 32-bit indexing: the host guarantees total * UPH * (Hkv / HPT) < 2^31
  const uint32_t g = blockIdx.x * blockDim.x + threadIdx.x;
  const uint32_t rest = g / UPH;
  const int ui = (int)(g - rest * UPH);
  const uint32_t tok32 = rest % (uint32_t)total;
  const int h0 = (int)(rest / (uint32_t)total) * HPT;
  if (h0 >= Hkv) return;
  const int64_t tok = tok32;
  int64_t e0, e1;
  if constexpr (NEOX) {
    e0 = (int64_t)ui * VEC;
    e1 = e0 + D / 2;
  } else {
    e0 = (int64_t)ui * 2 * VEC;
    e1 = e0 + VEC;
  }
  const int64_t v0 = (int64_t)ui * 2 * VEC;
  const RealignRow rr = tok_row[tok];
  const bool in_r = MASK ? sel[tok] != 0 : mark[tok] == gen;
  if (in_r) {
    // fresh rows of a token in R (bit-exact copies)
#pragma unroll
    for (int hh = 0; hh < HPT; ++hh) {
      const int head = h0 + hh;
      const int64_t dof = pool_off(rr.dst_slot, head, Hkv, D) * ESZ;
      const char* kn = (const char*)lay.k_new + (tok * Hkv + head) * D * ESZ;
      const char* vn = (const char*)lay.v_new + (tok * Hkv + head) * D * ESZ;
      const uint4 ka = *(const uint4*)(kn + e0 * ESZ);
      const uint4 kb = *(const uint4*)(kn + e1 * ESZ);
      const uint4 va = *(const uint4*)(vn + v0 * ESZ);
      const uint4 vb = *(const uint4*)(vn + (v0 + VEC) * ESZ);
      *(uint4*)(kc + dof + e0 * ESZ) = ka;
      *(uint4*)(kc + dof + e1 * ESZ) = kb;
      *(uint4*)(vc + dof + v0 * ESZ) = va;
      *(uint4*)(vc + dof + (v0 + VEC) * ESZ) = vb;
    }
    return;
  }
  if (rr.src_slot < 0) return;   // uncached and not listed: left as it is
  const char* src_k = (const char*)lay.src_k;
  const char* src_v = (const char*)lay.src_v;
  const float2* csr = cs + (int64_t)rr.cs_row * (D / 2) + (int64_t)ui * VEC;
  float2 c[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) c[e] = csr[e];
#pragma unroll
  for (int hh = 0; hh < HPT; ++hh) {
    const int head = h0 + hh;
    const int64_t so = pool_off(rr.src_slot, head, Hkv, D) * ESZ;
    const int64_t dof = pool_off(rr.dst_slot, head, Hkv, D) * ESZ;
    const uint4 ka = *(const uint4*)(src_k + so + e0 * ESZ);
    const uint4 kb = *(const uint4*)(src_k + so + e1 * ESZ);
    const uint4 va = *(const uint4*)(src_v + so + v0 * ESZ);
    const uint4 vb = *(const uint4*)(src_v + so + (v0 + VEC) * ESZ);
    float fa[VEC], fb[VEC], ya[VEC], yb[VEC];
    unpack<BF16>(ka, fa);
    unpack<BF16>(kb, fb);
    if constexpr (NEOX) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) rot(fa[e], fb[e], c[e].x, c[e].y, ya[e], yb[e]);
    } else {
#pragma unroll
      for (int e = 0; e < VEC / 2; ++e) {
        rot(fa[2 * e], fa[2 * e + 1], c[e].x, c[e].y, ya[2 * e], ya[2 * e + 1]);
        rot(fb[2 * e], fb[2 * e + 1], c[VEC / 2 + e].x, c[VEC / 2 + e].y, yb[2 * e], yb[2 * e + 1]);
      }
    }
    *(uint4*)(kc + dof + e0 * ESZ) = pack<BF16>(ya);
    *(uint4*)(kc + dof + e1 * ESZ) = pack<BF16>(yb);
    *(uint4*)(vc + dof + v0 * ESZ) = va;
    *(uint4*)(vc + dof + (v0 + VEC) * ESZ) = vb;
  }
}

// scores[i] = sum over KV heads h (in order) of colsum[h][i], rounded once to float32.
__global__ __launch_bounds__(256) void head_reduce_kernel(const double* __restrict__ colsum, int64_t total, int Hkv,
                                                          float* __restrict__ scores) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  double s = 0.0;
  for (int h = 0; h < Hkv; ++h) s += colsum[(int64_t)h * total + i];
  scores[i] = (float)s;
}

template <int D, bool BF16>
hipError_t realign_dispatch_style(const sx_plan* p, const void* sk, const void* sv, void* kc, void* vc,
                                  hipStream_t s) {
  constexpr int VEC = BF16 ? 8 : 4;
  const int units = p->desc.n_kv_heads * (D / (2 * VEC));
  const int64_t threads = p->n_realign * units;
  const dim3 grid((unsigned)((threads + 255) / 256));
  if (p->desc.rope_style == SX_ROPE_NEOX)
    hipLaunchKernelGGL((realign_kernel<D, BF16, true>), grid, dim3(256), 0, s, p->d_ra, p->n_realign, p->d_cs, sk,
                       sv, kc, vc, p->desc.n_kv_heads);
  else
    hipLaunchKernelGGL((realign_kernel<D, BF16, false>), grid, dim3(256), 0, s, p->d_ra, p->n_realign, p->d_cs, sk,
                       sv, kc, vc, p->desc.n_kv_heads);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_realign(const sx_plan* p, const void* sk, const void* sv, void* kc, void* vc, hipStream_t s) {
  const bool bf16 = p->desc.dtype == SX_BF16;
  if (p->desc.head_dim == 128)
    return bf16 ? realign_dispatch_style<128, true>(p, sk, sv, kc, vc, s)
                : realign_dispatch_style<128, false>(p, sk, sv, kc, vc, s);
  return bf16 ? realign_dispatch_style<64, true>(p, sk, sv, kc, vc, s)
              : realign_dispatch_style<64, false>(p, sk, sv, kc, vc, s);
}

hipError_t launch_scatter(const sx_plan* p, const void* k_new, const void* v_new, const int32_t* rows,
                          const int32_t* n_rows, int32_t max_rows, void* kc, void* vc, hipStream_t s) {
  const int esz = p->desc.dtype == SX_BF16 ? 2 : 4;
  const int uph = p->desc.head_dim * esz / 16;
  const int upr = p->desc.n_kv_heads * uph;
  const int64_t threads = (int64_t)max_rows * upr;
  const dim3 grid((unsigned)((threads + 255) / 256), (unsigned)p->n_req);
  hipLaunchKernelGGL(scatter_kernel, grid, dim3(256), 0, s, p->d_req, p->d_bt, rows, n_rows, max_rows, (const uint4*)k_new,
                     (const uint4*)v_new, (uint4*)kc, (uint4*)vc, p->desc.n_kv_heads, upr, uph);
  return hipGetLastError();
}

// heads per thread of realign_scatter_kernel (measured at d = 128, 8 KV heads: 1, 2, 4, 8 heads
// per thread ran 49.2, 48.4, 48.2, 48.5 us against 49.5 us for one head of one token)
constexpr int kRsHeads = 4;

template <int D, bool BF16, bool NEOX>
hipError_t realign_scatter_dispatch(const sx_plan* p, int32_t n_layers, const sx_layer_kv* layers, uint32_t gen,
                                   const uint8_t* sel, hipStream_t s) {
  constexpr int VEC = BF16 ? 8 : 4;
  // heads per thread: the largest of kRsHeads, 2, 1 that divides the KV head count
  constexpr int HPT = kRsHeads;
  const int hkv = p->desc.n_kv_heads;
  const int hpt = hkv % HPT == 0 ? HPT : (hkv % 2 == 0 ? 2 : 1);
  const int64_t threads = p->total * (D / (2 * VEC)) * (hkv / hpt);
  for (int32_t l0 = 0; l0 < n_layers; l0 += kLayersPerLaunch) {
    const int nl = n_layers - l0 < kLayersPerLaunch ? n_layers - l0 : kLayersPerLaunch;
    LayerTable tab{};
    for (int i = 0; i < nl; ++i) tab.l[i] = layers[l0 + i];
    const dim3 grid((unsigned)((threads + 255) / 256), (unsigned)nl);
    auto go = [&](auto mask, auto hpt_c) {
      hipLaunchKernelGGL((realign_scatter_kernel<D, BF16, NEOX, decltype(mask)::value, decltype(hpt_c)::value>), grid,
                         dim3(256), 0, s, p->d_tok_row, p->d_cs, p->d_rmark, sel, gen, p->total, tab, hkv);
    };
    auto by_hpt = [&](auto mask) {
      if (hpt == HPT) go(mask, std::integral_constant<int, HPT>{});
      else if (hpt == 2) go(mask, std::integral_constant<int, 2>{});
      else go(mask, std::integral_constant<int, 1>{});
    };
    if (sel) by_hpt(std::true_type{});
    else by_hpt(std::false_type{});
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_rows_mask(const sx_plan* p, const int32_t* rows, const int32_t* n_rows, int32_t max_rows,
                            uint8_t* mask, hipStream_t s) {
  hipLaunchKernelGGL(fill_u8_kernel, dim3((unsigned)((p->total + 255) / 256)), dim3(256), 0, s, mask, p->total,
                     (uint8_t)0);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || max_rows <= 0) return e;
  hipLaunchKernelGGL(mask_rows_kernel, dim3((unsigned)((max_rows + 255) / 256), (unsigned)p->n_req), dim3(256), 0, s,
                     p->d_req, rows, n_rows, max_rows, mask);
  return hipGetLastError();
}

hipError_t launch_realign_scatter(const sx_plan* p, int32_t n_layers, const sx_layer_kv* layers, const int32_t* rows,
                                  const int32_t* n_rows, int32_t max_rows, uint32_t gen, bool clear_marks,
                                  const uint8_t* sel, hipStream_t s) {
  if (sel) {
    rows = nullptr;   // membership comes from the caller's mask
    max_rows = 0;
    clear_marks = false;
  }
  if (clear_marks) {
    hipLaunchKernelGGL(fill_u32_kernel, dim3((unsigned)((p->total + 255) / 256)), dim3(256), 0, s, p->d_rmark,
                       p->total, 0u);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (max_rows > 0) {
    hipLaunchKernelGGL(mark_rows_kernel, dim3((unsigned)((max_rows + 255) / 256), (unsigned)p->n_req), dim3(256), 0,
                       s, p->d_req, rows, n_rows, max_rows, p->d_rmark, gen);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const bool bf16 = p->desc.dtype == SX_BF16;
  const bool neox = p->desc.rope_style == SX_ROPE_NEOX;
#define SX_RS(D_, B_, N_) return realign_scatter_dispatch<D_, B_, N_>(p, n_layers, layers, gen, sel, s)
  if (p->desc.head_dim == 128) {
    if (bf16) { if (neox) SX_RS(128, true, true); else SX_RS(128, true, false); }
    else { if (neox) SX_RS(128, false, true); else SX_RS(128, false, false); }
  } else {
    if (bf16) { if (neox) SX_RS(64, true, true); else SX_RS(64, true, false); }
    else { if (neox) SX_RS(64, false, true); else SX_RS(64, false, false); }
  }
#undef SX_RS
}

hipError_t launch_head_reduce(const sx_plan* p, const double* colsum, float* scores, hipStream_t s) {
  const dim3 grid((unsigned)((p->total + 255) / 256));
  hipLaunchKernelGGL(head_reduce_kernel, grid, dim3(256), 0, s, colsum, p->total, p->desc.n_kv_heads, scores);
  return hipGetLastError();
}

hipError_t launch_probe_pad_clear(const sx_plan* p, const ScoreScratch& sc, hipStream_t s) {
  const int64_t G = p->desc.n_q_heads / p->desc.n_kv_heads;
  // queries: the kProbePad rows after the last probe row of every KV head (bf16 zero = 0)
  const int64_t qrow = G * p->desc.head_dim * 2;   // bytes of one probe row of one KV head
  const int64_t qwords = kProbePad * qrow / 4;
  hipError_t e = hipSuccess;
  for (int h = 0; h < p->desc.n_kv_heads; ++h) {
    char* base = (char*)sc.qp + ((int64_t)h * (p->n_probe + kProbePad) + p->n_probe) * qrow;
    hipLaunchKernelGGL(fill_u32_kernel, dim3((unsigned)((qwords + 255) / 256)), dim3(256), 0, s, (uint32_t*)base,
                       qwords, 0u);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  // log-sum-exps: the kProbePad rows after the last probe row of every KV head (+inf)
  for (int h = 0; h < p->desc.n_kv_heads; ++h) {
    float* base = sc.lse2p + ((int64_t)h * (p->n_probe + kProbePad) + p->n_probe) * G;
    hipLaunchKernelGGL(fill_u32_kernel, dim3((unsigned)((kProbePad * G + 255) / 256)), dim3(256), 0, s,
                       (uint32_t*)base, (int64_t)kProbePad * G, kProbePadLse);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace sx
