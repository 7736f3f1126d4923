// float32 attention and Sparse-Q column sums on the vector ALUs.  Used when the layer stores
// float32 (small, accuracy-first configurations); the bfloat16 path runs on matrix cores.
//
// Attention: one wavefront per (query row, query head).  Each lane walks keys j = lane,
// lane + 64, ... keeping its own online-softmax state (max, sum, d-vector); the 64 partial
// states are merged through LDS at the end.
#include "sx_device.h"
#include "sx_internal.h"

namespace sx {
namespace {

struct AttnF {
  const float* q;
  const float* k;
  const float* v;
  float* out;
  float* lse;
  const ReqDev* reqs;
  const int32_t* bt;
  const int32_t* rows;
  const int32_t* n_rows;
  const int32_t* cu;
  int Hq, Hkv, G;
  float scale;
  int lse_base2;
};

template <int D, bool PAGED>
__device__ __forceinline__ const float* f_row(const AttnF& a, const float* base, int tok_off, int bt_off, int kvh,
                                              int key) {
  if constexpr (PAGED) {
    const int32_t blk = a.bt[bt_off + (key >> 4)];
    return base + (((int64_t)blk * a.Hkv + kvh) * 16 + (key & 15)) * D;
  } else {
    return base + ((int64_t)(tok_off + key) * a.Hkv + kvh) * D;
  }
}

template <int D, bool PAGED, bool PV>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnF a) {
  __shared__ float qs[D];
  __shared__ float red[PV ? 64 * (D + 1) : 1];
  __shared__ float ms[64], ls[64];
  const int lane = threadIdx.x;
  const int ridx = blockIdx.x;
  const int h = blockIdx.y;
  const int r = blockIdx.z;
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
  (void)T;
  if (ridx >= nrows) return;
  const int pos = PAGED ? a.rows[tok_off + ridx] : ridx;
  const int kvh = h / a.G;
  const float* qp = a.q + ((int64_t)(tok_off + pos) * a.Hq + h) * D;
  for (int x = lane; x < D; x += 64) qs[x] = qp[x];
  __syncthreads();
  float m = -INFINITY, l = 0.f;
  float o[PV ? D : 1];
#pragma unroll
  for (int x = 0; x < (PV ? D : 1); ++x) o[x] = 0.f;
  for (int j = lane; j <= pos; j += 64) {
    const float* kp = f_row<D, PAGED>(a, a.k, tok_off, bt_off, kvh, j);
    float z = 0.f;
#pragma unroll 8
    for (int x = 0; x < D; ++x) z = fmaf(qs[x], kp[x], z);
    z *= a.scale;
    if (z > m) {
      const float f = expf(m - z);
      l *= f;
      if constexpr (PV) {
#pragma unroll
        for (int x = 0; x < D; ++x) o[x] *= f;
      }
      m = z;
    }
    const float p = expf(z - m);
    l += p;
    if constexpr (PV) {
      const float* vp = f_row<D, PAGED>(a, a.v, tok_off, bt_off, kvh, j);
#pragma unroll
      for (int x = 0; x < D; ++x) o[x] = fmaf(p, vp[x], o[x]);
    }
  }
  ms[lane] = m;
  __syncthreads();
  float M = -INFINITY;
  for (int i = 0; i < 64; ++i) M = fmaxf(M, ms[i]);
  const float f = m == -INFINITY ? 0.f : expf(m - M);
  ls[lane] = l * f;
  if constexpr (PV) {
#pragma unroll
    for (int x = 0; x < D; ++x) red[lane * (D + 1) + x] = o[x] * f;
  }
  __syncthreads();
  float L = 0.f;
  for (int i = 0; i < 64; ++i) L += ls[i];
  if constexpr (PV) {
    float* op = a.out + ((int64_t)(tok_off + ridx) * a.Hq + h) * D;
    for (int x = lane; x < D; x += 64) {
      float s = 0.f;
      for (int i = 0; i < 64; ++i) s += red[i * (D + 1) + x];
      op[x] = s / L;
    }
  }
  if (a.lse && lane == 0) {
    const float lse = M + logf(L);
    a.lse[(int64_t)(tok_off + ridx) * a.Hq + h] = lse;   // natural log of sum exp(scale q.k)
  }
}

// One thread per key (and KV head): sum over probe rows i >= j and the heads of the group of
// exp(scale q_{i,h}.k_j - lse_{i,h}), float64 accumulation in fixed (row, head) order.
struct ColsumF {
  const float* q;
  const float* k;
  const float* lse;
  const ReqDev* reqs;
  const int32_t* bt;
  const int32_t* probe;
  double* colsum;
  int64_t total;
  int Hq, Hkv, G;
  float scale;
  int lse_tok;   // 0: lse indexed by probe; 1: indexed by token position
};

template <int D>
__global__ __launch_bounds__(256) void colsum_f32_kernel(ColsumF a) {
  const ReqDev rq = a.reqs[blockIdx.z];
  const int kvh = blockIdx.y;
  const int j0 = blockIdx.x * 256;
  if (j0 >= rq.T) return;
  const int j = j0 + threadIdx.x;
  const bool valid = j < rq.T;
  float kr[D];
  {
    const int jj = valid ? j : 0;
    const int32_t blk = a.bt[rq.bt_off + (jj >> 4)];
    const float* kp = a.k + (((int64_t)blk * a.Hkv + kvh) * 16 + (jj & 15)) * D;
#pragma unroll
    for (int x = 0; x < D; ++x) kr[x] = kp[x];
  }
  const int32_t* probe = a.probe + rq.tok_off;
  int lo = 0, hi = rq.n_probe;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (probe[mid] < j0) lo = mid + 1; else hi = mid;
  }
  double acc = 0.0;
  for (int p = lo; p < rq.n_probe; ++p) {
    const int pos = probe[p];
    for (int h = 0; h < a.G; ++h) {
      const int qh = kvh * a.G + h;
      const float* qp = a.q + ((int64_t)(rq.tok_off + pos) * a.Hq + qh) * D;
      float z = 0.f;
#pragma unroll 8
      for (int x = 0; x < D; ++x) z = fmaf(qp[x], kr[x], z);
      z *= a.scale;
      const float pr = expf(z - a.lse[(int64_t)(rq.tok_off + (a.lse_tok ? pos : p)) * a.Hq + qh]);
      if (valid && j <= pos) acc += (double)pr;
    }
  }
  if (valid) a.colsum[(int64_t)kvh * a.total + rq.tok_off + j] = acc;
}

}  // namespace

hipError_t launch_attn_f32(const AttnLaunch& L, bool paged, hipStream_t s) {
  AttnF a{};
  a.q = (const float*)L.q;
  a.k = (const float*)L.k;
  a.v = (const float*)L.v;
  a.out = (float*)L.out;
  a.lse = L.lse;
  a.reqs = L.reqs;
  a.bt = L.bt;
  a.rows = L.rows;
  a.n_rows = L.n_rows;
  a.cu = L.cu;
  a.Hq = L.Hq;
  a.Hkv = L.Hkv;
  a.G = L.Hq / L.Hkv;
  a.scale = L.scale;
  a.lse_base2 = L.lse_base2;
  const dim3 grid((unsigned)L.grid_rows, (unsigned)L.Hq, (unsigned)L.n_req);
  const bool pv = L.out != nullptr;
#define SX_F32_LAUNCH(D_, P_, V_) hipLaunchKernelGGL((attn_f32_kernel<D_, P_, V_>), grid, dim3(64), 0, s, a)
  if (L.D == 128) {
    if (paged) { if (pv) SX_F32_LAUNCH(128, true, true); else SX_F32_LAUNCH(128, true, false); }
    else SX_F32_LAUNCH(128, false, true);
  } else {
    if (paged) { if (pv) SX_F32_LAUNCH(64, true, true); else SX_F32_LAUNCH(64, true, false); }
    else SX_F32_LAUNCH(64, false, true);
  }
#undef SX_F32_LAUNCH
  return hipGetLastError();
}

hipError_t launch_colsum_f32(const sx_plan* p, double* colsum, const void* q, const void* kc, const float* lse,
                             int lse_tok, hipStream_t s) {
  ColsumF a{};
  a.q = (const float*)q;
  a.k = (const float*)kc;
  a.lse = lse;
  a.lse_tok = lse_tok;
  a.reqs = p->d_req;
  a.bt = p->d_bt;
  a.probe = p->d_probe;
  a.colsum = colsum;
  a.total = p->total;
  a.Hq = p->desc.n_q_heads;
  a.Hkv = p->desc.n_kv_heads;
  a.G = a.Hq / a.Hkv;
  a.scale = p->scale;
  const dim3 grid((unsigned)((p->max_T + 255) / 256), (unsigned)a.Hkv, (unsigned)p->n_req);
  if (p->desc.head_dim == 128)
    hipLaunchKernelGGL(colsum_f32_kernel<128>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(colsum_f32_kernel<64>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace sx
