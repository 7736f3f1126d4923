// Row-sparse layer body (Algorithm 1 steps 19 and 22): the projections, normalisations and the
// feed-forward module evaluated on the rows of the recompute set R only.
//
//   gemm_rows_kernel     Y[row] = X[row] W^T (+ residual[row]): bfloat16 operands, float32
//                        accumulation on v_mfma_f32_16x16x32_bf16, W stored [n][k] (k contiguous,
//                        the layout of a linear layer's weight)
//   rmsnorm_rows_kernel  Y[row] = X[row] / sqrt(mean(X[row]^2) + eps) * gamma
//   rope_rows_kernel     RoPE of fresh query / key rows at their positions in the new sequence
//   silu_mul_rows_kernel Y[row] = silu(G[row]) * U[row] for a gate|up product [row][2f]
//
// Rows: for request r, the listed rows n < n_rows[r] of the row-list layout.  An operand row is
// addressed by slot (off_r + n: compact per request, like the sparse attention output) or by
// token (off_r + rows[off_r + n]: the request's token rows, like fresh Q/K/V and hidden states).
#include "sx_device.h"
#include "sx_internal.h"

namespace sx {
namespace {

typedef float f32x2_t __attribute__((ext_vector_type(2)));

// s_waitcnt with vmcnt <= n (n < 16), expcnt and lgkmcnt left unconstrained (gfx9 encoding).
#define SX_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt(((n) & 0xF) | (0x7 << 4) | (0xF << 8))
// the same for n < 64 (the counter's two high bits sit at 15:14)
#define SX_WAIT_VMCNT6(n) \
  __builtin_amdgcn_s_waitcnt(((n) & 0xF) | ((((n) >> 4) & 3) << 14) | (0x7 << 4) | (0xF << 8))

__device__ __forceinline__ int64_t row_index(const ReqDev& rq, const int32_t* rows, int n, bool by_token) {
  return by_token ? (int64_t)rq.tok_off + rows[rq.tok_off + n] : (int64_t)rq.tok_off + n;
}

// ---------------------------------------------------------------------------------------------
// GEMM on listed rows.  Computed transposed, Y^T = W X^T: the MFMA A operand is a slice of W (MF
// output features), the B operand a slice of X^T (MF rows), so each lane owns one row of the
// result and writes 4 consecutive features per store.
// Workgroup tile: 256 features x 256 rows; 8 waves as 4 (features) x 2 (rows), a wave owns 64
// features x 128 rows.  The default MFMA is v_mfma_f32_16x16x32_bf16 (4 x 8 accumulators of
// 16 x 16): measured 1-12 % faster than v_mfma_f32_32x32x16_bf16 (MF = 32, 2 x 4 accumulators)
// on the same tiles, most on the narrow products.  The k dimension moves in stages of BK
// through NST LDS buffers: both operand tiles go global -> LDS directly (16 bytes per lane);
// stage t + NST is issued once every wave has read stage t, so a stage has about NST - 1 stages
// of compute to land.  A tile row (BK bf16) holds BK / 8 chunks of 16 bytes, XOR-swizzled per row
// (chunk_swz) so that the rows a read instruction touches at one logical chunk hit distinct banks.
// ---------------------------------------------------------------------------------------------
constexpr int GBN = 256, GBM = 256;
constexpr int kGemmMaxParts = 4;
constexpr unsigned kGemmXcds = 8;   // XCDs of the chip, which deals workgroups round-robin
constexpr int kSgMfma = 0x8, kSgDsRead = 0x100;   // sched_group_barrier instruction classes

struct GemmRowsK {
  const ReqDev* reqs;
  const int32_t* rows;
  const int32_t* n_rows;
  const uint16_t* x;
  const uint16_t* w;
  const uint16_t* res;
  uint16_t* y[kGemmMaxParts];   // output part p: columns pn[p] .. pn[p + 1] - 1, row stride pn[p + 1] - pn[p]
  int pn[kGemmMaxParts + 1];
  int n_parts, K, N, n_req, m_tiles, max_rows, x_tok, y_tok;
};

// physical chunk of logical chunk c in tile row `row` (CH chunks per row): 16 consecutive rows
// read at one logical chunk cover the 16 four-bank groups of a 256-byte LDS line
template <int CH>
__device__ __forceinline__ int chunk_swz(int c, int row) {
  if constexpr (CH == 8) return c ^ ((row >> 1) & 7);   // 128-byte rows: two per line
  else return c ^ ((row >> 2) & 3);                     // 64-byte rows: four per line
}

template <int BK, int NST, int GM, int NW, int MF>
__global__ __launch_bounds__(NW * 64, 1) void gemm_rows_kernel(GemmRowsK a) {
  // NW = 8: a wave owns 64 features x 128 rows (two waves per SIMD); NW = 4: 128 x 128 (one wave
  // per SIMD, the accumulators in the AGPR half of the register file; measured about 10 % slower)
  // MF = 32: v_mfma_f32_32x32x16_bf16 (32 x 32 blocks, k 16); MF = 16: v_mfma_f32_16x16x32_bf16
  constexpr int WCOL = NW / 2;                 // waves across the features
  constexpr int FI = 256 / WCOL / MF;          // MF-feature fragments per wave
  constexpr int RJ = 128 / MF;                 // MF-row fragments per wave
  constexpr int KM = MF == 32 ? 16 : 32;       // k per MFMA
  typedef float accv_t __attribute__((ext_vector_type(MF == 32 ? 16 : 4)));
  constexpr int ROWB = BK * 2;                 // bytes of one tile row
  constexpr int CH = ROWB / 16;                // 16-byte chunks per row
  constexpr int TILE = 256 * ROWB;             // bytes of one operand tile
  constexpr int RPP = 1024 / ROWB;             // rows per 1 KB transfer
  constexpr int PPW = 256 / RPP / NW;          // transfers per wave per operand tile
  constexpr int NS = BK / KM;                  // k slices (one MFMA deep) per stage
  __shared__ __attribute__((aligned(1024))) char smem[NST * 2 * TILE];   // [stage][W | X]
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wu = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31;
  const int hg = lane >> 5;
  // tile order: groups of GM row tiles, the feature tile slowest within a group, so that a run of
  // consecutive tile indices covers a few feature tiles x GM row tiles.  The hardware deals block b
  // to XCD b mod 8; each XCD takes a contiguous run of tile indices, so the workgroups running
  // together on one XCD read the same W and X k-slices through that XCD's L2.
  const int n_mt = a.n_req * a.m_tiles;
  const int n_nt = a.N / GBN;
  const unsigned per_xcd = gridDim.x / kGemmXcds;   // the grid is a multiple of kGemmXcds
  const int L = (int)((blockIdx.x % kGemmXcds) * per_xcd + blockIdx.x / kGemmXcds);
  if (L >= n_mt * n_nt) return;
  const int grp = L / (GM * n_nt);
  const int in_g = L - grp * GM * n_nt;
  const int gm = min(GM, n_mt - grp * GM);
  const int mt_all = grp * GM + in_g % gm;
  const int nt = in_g / gm;
  const int r = mt_all / a.m_tiles;
  const int m0 = (mt_all - r * a.m_tiles) * GBM;
  const ReqDev rq = a.reqs[r];
  const int nr = min(a.n_rows[r], a.max_rows);
  if (m0 >= nr) return;
  const int n0 = nt * GBN;
  const int K = a.K;

  // ---- transfers: piece q (1 KB) of a tile holds rows RPP q .. RPP q + RPP - 1; lane l fills row
  // RPP q + l / CH, physical chunk l % CH with the logical chunk that chunk_swz maps there.  A wave
  // moves pieces wu + 8 i (i < PPW) of both tiles. ----
  const uint16_t* w_src[PPW];
  const uint16_t* x_src[PPW];
#pragma unroll
  for (int i = 0; i < PPW; ++i) {
    const int row = RPP * (wu + NW * i) + lane / CH;
    const int lc = chunk_swz<CH>(lane % CH, row);   // (the swizzle is an involution)
    w_src[i] = a.w + (int64_t)(n0 + row) * K + lc * 8;
    const int m = min(m0 + row, nr - 1);   // rows past the request's last read a valid row
    x_src[i] = a.x + row_index(rq, a.rows, m, a.x_tok) * K + lc * 8;
  }
  const uint32_t smem_lds = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)smem;
  auto dma16 = [&](const void* src, uint32_t lds) {
    const uint32_t m0r = __builtin_amdgcn_readfirstlane(lds);
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(m0r) : "m0", "memory");
  };
  const int nk = K / BK;
  auto issue = [&](int t) {   // stage t into buffer t mod NST
    if (t >= nk) return;
    const uint32_t base = smem_lds + (uint32_t)((t % NST) * 2 * TILE);
    const int k0 = t * BK;
#pragma unroll
    for (int i = 0; i < PPW; ++i) {
      dma16(w_src[i] + k0, base + (uint32_t)((wu + NW * i) * 1024));
      dma16(x_src[i] + k0, base + (uint32_t)(TILE + (wu + NW * i) * 1024));
    }
  };
  // wait until this wave's transfers of every stage before the n youngest have landed
  auto wait_stages = [&](int n) {
    switch (n * 2 * PPW) {
      case 0: SX_WAIT_VMCNT6(0); break;
      case 4: SX_WAIT_VMCNT6(4); break;
      case 8: SX_WAIT_VMCNT6(8); break;
      case 12: SX_WAIT_VMCNT6(12); break;
      case 16: SX_WAIT_VMCNT6(16); break;
      case 24: SX_WAIT_VMCNT6(24); break;
      default: SX_WAIT_VMCNT6(32); break;
    }
  };
  static_assert((NST - 1) * 2 * PPW <= 32 && (2 * PPW) % 4 == 0, "wait table");
  static_assert(NS % 2 == 0, "a stage holds an even number of slices");

  // ---- operand reads: row 32 j + l32 of a tile, logical chunk 2 s + hg: the lane part depends on
  // s only, the row block adds a constant (an immediate offset) ----
  const int wn = wu % WCOL, wm = wu / WCOL;
  // a lane reads row lr of each MF-row fragment, 16 bytes of k starting at chunk (KM / 8) s + cg
  const int lr = lane % MF, cg = lane / MF;
  uint32_t lane_off[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s)
    lane_off[s] = (uint32_t)(lr * ROWB + (chunk_swz<CH>((KM / 8) * s + cg, lr) << 4));
  accv_t acc[FI][RJ];
#pragma unroll
  for (int i = 0; i < FI; ++i)
#pragma unroll
    for (int j = 0; j < RJ; ++j)
#pragma unroll
      for (int e = 0; e < (MF == 32 ? 16 : 4); ++e) acc[i][j][e] = 0.f;

  // fragments of one 16-wide k slice, read from stage buffer `buf`: one base register per matrix
  // (the empty asm keeps the sums from being re-associated into one register per read), the row
  // blocks as immediate offsets
  auto read_slice = [&](int buf, int s, bf16x8_t (&fw)[FI], bf16x8_t (&fx)[RJ]) {
    const uint32_t sb = smem_lds + (uint32_t)(buf * 2 * TILE);
    uint32_t wb = sb + lane_off[s] + (uint32_t)(wn * FI * MF * ROWB);
    uint32_t xb = sb + (uint32_t)TILE + lane_off[s] + (uint32_t)(wm * 128 * ROWB);
    asm volatile("" : "+v"(wb), "+v"(xb));
#pragma unroll
    for (int i = 0; i < FI; ++i)
      fw[i] = *(const __attribute__((address_space(3))) bf16x8_t*)(uintptr_t)(wb + (uint32_t)(i * MF * ROWB));
#pragma unroll
    for (int j = 0; j < RJ; ++j)
      fx[j] = *(const __attribute__((address_space(3))) bf16x8_t*)(uintptr_t)(xb + (uint32_t)(j * MF * ROWB));
  };

  // Software pipeline: the fragments of slice s + 1 are read while the MFMAs of slice s run (two
  // register sets).  The stage barrier sits before the MFMAs of a stage's last slice: past it every
  // wave has finished reading the stage (its buffer takes stage t + NST) and stage t + 1 has landed
  // (its first slice is read during those MFMAs).
  // the row indices above are compiler-visible loads: complete before the first transfer wait
  SX_WAIT_VMCNT(0);
#pragma unroll
  for (int t = 0; t < NST; ++t) issue(t);
  wait_stages(min(NST - 1, nk - 1));   // stage 0 has landed
  __syncthreads();
  bf16x8_t fw[2][FI], fx[2][RJ];
  auto mfma_slice = [&](int c) {
#pragma unroll
    for (int i = 0; i < FI; ++i)
#pragma unroll
      for (int j = 0; j < RJ; ++j) {
        if constexpr (MF == 32)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[c][i], fx[c][j], acc[i][j], 0, 0, 0);
        else
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw[c][i], fx[c][j], acc[i][j], 0, 0, 0);
      }
  };
  // the scheduler would sink the reads below the MFMAs (to reuse their registers): pin one read
  // after each of the first FI + RJ MFMAs
  auto interleave = [&]() {
#pragma unroll
    for (int q = 0; q < FI + RJ; ++q) {
      __builtin_amdgcn_sched_group_barrier(kSgMfma, 1, 0);
      __builtin_amdgcn_sched_group_barrier(kSgDsRead, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(kSgMfma, FI * RJ - FI - RJ, 0);
  };
  read_slice(0, 0, fw[0], fx[0]);
  for (int t = 0; t + 1 < nk; ++t) {
#pragma unroll
    for (int s = 0; s + 1 < NS; ++s) {   // NS is even: a stage starts on set 0
      read_slice(t % NST, s + 1, fw[(s + 1) & 1], fx[(s + 1) & 1]);
      mfma_slice(s & 1);
      interleave();
    }
    // this wave's reads of stage t are done (the barrier alone does not wait for them) and its
    // transfers of stage t + 1 have landed (the younger ones may be in flight)
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    wait_stages(max(0, min(NST - 2, nk - 2 - t)));
    __syncthreads();
    issue(t + NST);   // into the buffer of stage t
    read_slice((t + 1) % NST, 0, fw[0], fx[0]);
    mfma_slice(1);
    interleave();
  }
  // last stage
#pragma unroll
  for (int s = 0; s + 1 < NS; ++s) {
    read_slice((nk - 1) % NST, s + 1, fw[(s + 1) & 1], fx[(s + 1) & 1]);
    mfma_slice(s & 1);
    interleave();
  }
  mfma_slice(1);

  // ---- epilogue: lane owns row 32 j + l32 of the wave's rows; value e of accumulator (i, j) is
  // feature 32 i + 8 (e / 4) + 4 hg + e % 4 of the wave's features.  Part boundaries are multiples
  // of the tile width, so the output part is the tile's. ----
  // MF = 16: lane owns row 16 j + lr, value e of accumulator (i, j) is feature 16 i + 4 cg + e
  static_assert(RJ * MF == 128, "two waves of rows cover the 256-row tile");
  int part = 0;
  while (part + 1 < a.n_parts && n0 >= a.pn[part + 1]) ++part;
  uint16_t* const yp = a.y[part];
  const int ld = a.pn[part + 1] - a.pn[part];
  const int c0 = n0 - a.pn[part] + wn * FI * MF + 4 * cg;
#pragma unroll
  for (int j = 0; j < RJ; ++j) {
    const int m = m0 + wm * 128 + MF * j + lr;
    if (m >= nr) continue;
    const int64_t yr = row_index(rq, a.rows, m, a.y_tok) * ld;
#pragma unroll
    for (int i = 0; i < FI; ++i)
#pragma unroll
      for (int g = 0; g < (MF == 32 ? 4 : 1); ++g) {
        const int c = c0 + MF * i + 8 * g;
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * g + e];
        if (a.res) {
          const uint2 rv = *(const uint2*)(a.res + yr + c);
          v[0] += bf16_lo(rv.x);
          v[1] += bf16_hi(rv.x);
          v[2] += bf16_lo(rv.y);
          v[3] += bf16_hi(rv.y);
        }
        uint2 o;
        o.x = pack_bf16x2(v[0], v[1]);
        o.y = pack_bf16x2(v[2], v[3]);
        *(uint2*)(yp + yr + c) = o;
      }
  }
}

#ifndef SX_GEMM_BK
#define SX_GEMM_BK 64
#define SX_GEMM_NST 2
#endif
#ifndef SX_GEMM_GM
#define SX_GEMM_GM 8
#endif
#ifndef SX_GEMM_NW
#define SX_GEMM_NW 8
#endif
#ifndef SX_GEMM_MF
#define SX_GEMM_MF 16
#endif

// ---------------------------------------------------------------------------------------------
// RMSNorm of listed rows: one wave per row, float32 sum of squares in a fixed order.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void rmsnorm_rows_kernel(const ReqDev* __restrict__ reqs, const int32_t* __restrict__ rows,
                                                           const int32_t* __restrict__ n_rows, int max_rows,
                                                           const uint16_t* __restrict__ x, int x_tok,
                                                           const uint16_t* __restrict__ gamma, float eps, int H,
                                                           uint16_t* __restrict__ y, int y_tok) {
  const ReqDev rq = reqs[blockIdx.y];
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (n >= n_rows[blockIdx.y] || n >= max_rows) return;
  const uint16_t* xr = x + row_index(rq, rows, n, x_tok) * H;
  uint16_t* yr = y + row_index(rq, rows, n, y_tok) * H;
  float ss = 0.f;
  for (int c = lane * 8; c < H; c += 64 * 8) {
    const uint4 v = *(const uint4*)(xr + c);
    const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float lo = bf16_lo(u[i]), hi = bf16_hi(u[i]);
      ss = __builtin_fmaf(lo, lo, ss);
      ss = __builtin_fmaf(hi, hi, ss);
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o, 64);
  const float inv = 1.0f / sqrtf(ss / (float)H + eps);
  for (int c = lane * 8; c < H; c += 64 * 8) {
    const uint4 v = *(const uint4*)(xr + c);
    const uint4 gv = *(const uint4*)(gamma + c);
    const uint32_t u[4] = {v.x, v.y, v.z, v.w}, gw[4] = {gv.x, gv.y, gv.z, gv.w};
    uint32_t o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      o[i] = pack_bf16x2(bf16_lo(u[i]) * inv * bf16_lo(gw[i]), bf16_hi(u[i]) * inv * bf16_hi(gw[i]));
    *(uint4*)(yr + c) = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

// ---------------------------------------------------------------------------------------------
// RoPE of the fresh query and key rows of listed tokens, in place.  A thread owns 8 rotation
// pairs of one token: it forms their cos / sin once (angle and cos / sin in float64, rounded to
// float32) and rotates those pairs in every query and key head (float32, no contraction, bf16
// store with round to nearest even).
// ---------------------------------------------------------------------------------------------
template <int D, bool NEOX>
__global__ __launch_bounds__(256) void rope_rows_kernel(const ReqDev* __restrict__ reqs, const int32_t* __restrict__ rows,
                                                        const int32_t* __restrict__ n_rows, int max_rows,
                                                        const int32_t* __restrict__ tok_pos,
                                                        const double* __restrict__ theta, uint16_t* __restrict__ q,
                                                        uint16_t* __restrict__ k, int Hq, int Hkv) {
  constexpr int UPR = D / 16;   // threads per token: 8 pairs each
  const ReqDev rq = reqs[blockIdx.y];
  const int g = blockIdx.x * blockDim.x + threadIdx.x;
  const int n = g / UPR;
  const int u = g - n * UPR;
  if (n >= n_rows[blockIdx.y] || n >= max_rows) return;
  const int64_t t = row_index(rq, rows, n, true);
  const double pos = (double)tok_pos[t];
  float c[8], s[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const double phi = pos * theta[u * 8 + e];
    c[e] = (float)cos(phi);
    s[e] = (float)sin(phi);
  }
  // pair p = 8u + e: NEOX (p, p + D/2); GPT-J (2p, 2p + 1)
  auto rotate_head = [&](uint16_t* h) {
#pragma clang fp contract(off)
    if constexpr (NEOX) {
      uint4* pa = (uint4*)(h + u * 8);
      uint4* pb = (uint4*)(h + D / 2 + u * 8);
      const uint4 va = *pa, vb = *pb;
      const uint32_t wa[4] = {va.x, va.y, va.z, va.w}, wb[4] = {vb.x, vb.y, vb.z, vb.w};
      uint32_t oa[4], ob[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float a0 = bf16_lo(wa[i]), a1 = bf16_hi(wa[i]), b0 = bf16_lo(wb[i]), b1 = bf16_hi(wb[i]);
        const int e0 = 2 * i, e1 = 2 * i + 1;
        oa[i] = pack_bf16x2(a0 * c[e0] - b0 * s[e0], a1 * c[e1] - b1 * s[e1]);
        ob[i] = pack_bf16x2(b0 * c[e0] + a0 * s[e0], b1 * c[e1] + a1 * s[e1]);
      }
      *pa = make_uint4(oa[0], oa[1], oa[2], oa[3]);
      *pb = make_uint4(ob[0], ob[1], ob[2], ob[3]);
    } else {
      uint4* pp = (uint4*)(h + u * 16);
      const uint4 v0 = pp[0], v1 = pp[1];
      const uint32_t w[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
      uint32_t o[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x1 = bf16_lo(w[e]), x2 = bf16_hi(w[e]);
        o[e] = pack_bf16x2(x1 * c[e] - x2 * s[e], x2 * c[e] + x1 * s[e]);
      }
      pp[0] = make_uint4(o[0], o[1], o[2], o[3]);
      pp[1] = make_uint4(o[4], o[5], o[6], o[7]);
    }
  };
  for (int h = 0; h < Hq; ++h) rotate_head(q + (t * Hq + h) * D);
  for (int h = 0; h < Hkv; ++h) rotate_head(k + (t * Hkv + h) * D);
}

// ---------------------------------------------------------------------------------------------
// SwiGLU activation of listed rows (slot-indexed): gu row = [gate (f) | up (f)] -> y row (f).
// silu(g) = g / (1 + e^-g) in float32.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void silu_mul_rows_kernel(const ReqDev* __restrict__ reqs,
                                                            const int32_t* __restrict__ n_rows, int max_rows,
                                                            const uint16_t* __restrict__ gu, int f,
                                                            uint16_t* __restrict__ y) {
  const ReqDev rq = reqs[blockIdx.y];
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int upr = f / 8;
  const int64_t n = g / upr;
  const int c = (int)(g - n * upr) * 8;
  if (n >= n_rows[blockIdx.y] || n >= max_rows) return;
  const int64_t row = (int64_t)rq.tok_off + n;
  const uint4 gv = *(const uint4*)(gu + row * 2 * f + c);
  const uint4 uv = *(const uint4*)(gu + row * 2 * f + f + c);
  const uint32_t gw[4] = {gv.x, gv.y, gv.z, gv.w}, uw[4] = {uv.x, uv.y, uv.z, uv.w};
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float g0 = bf16_lo(gw[i]), g1 = bf16_hi(gw[i]);
    const float s0 = g0 / (1.0f + expf(-g0)), s1 = g1 / (1.0f + expf(-g1));
    o[i] = pack_bf16x2(s0 * bf16_lo(uw[i]), s1 * bf16_hi(uw[i]));
  }
  *(uint4*)(y + row * f + c) = make_uint4(o[0], o[1], o[2], o[3]);
}

}  // namespace

hipError_t launch_gemm_rows(const sx_plan* p, const RowsArg& r, const void* x, int x_tok, const void* w, int k,
                            int n_parts, const int* part_n, void* const* ys, const void* res, int y_tok, hipStream_t s) {
  if (n_parts < 1 || n_parts > kGemmMaxParts) return hipErrorInvalidValue;
  GemmRowsK a{};
  a.reqs = p->d_req;
  a.rows = r.rows;
  a.n_rows = r.n_rows;
  a.x = (const uint16_t*)x;
  a.w = (const uint16_t*)w;
  a.res = (const uint16_t*)res;
  a.n_parts = n_parts;
  int n = 0;
  for (int i = 0; i < n_parts; ++i) {
    a.y[i] = (uint16_t*)ys[i];
    a.pn[i] = n;
    n += part_n[i];
  }
  a.pn[n_parts] = n;
  a.K = k;
  a.N = n;
  a.n_req = p->n_req;
  a.m_tiles = (r.max_rows + GBM - 1) / GBM;
  a.max_rows = r.max_rows;
  constexpr int BK = SX_GEMM_BK, NST = SX_GEMM_NST, GM = SX_GEMM_GM, NW = SX_GEMM_NW, MF = SX_GEMM_MF;
  a.x_tok = x_tok;
  a.y_tok = y_tok;
  const int64_t tiles = (int64_t)a.m_tiles * p->n_req * (n / GBN);
  const int64_t blocks = (tiles + kGemmXcds - 1) / kGemmXcds * kGemmXcds;
  hipLaunchKernelGGL((gemm_rows_kernel<BK, NST, GM, NW, MF>), dim3((unsigned)blocks), dim3(NW * 64), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_rmsnorm_rows(const sx_plan* p, const RowsArg& r, const void* x, int x_tok, const void* gamma,
                               float eps, int h, void* y, int y_tok, hipStream_t s) {
  const dim3 grid((unsigned)((r.max_rows + 3) / 4), (unsigned)p->n_req);
  hipLaunchKernelGGL(rmsnorm_rows_kernel, grid, dim3(256), 0, s, p->d_req, r.rows, r.n_rows, r.max_rows, (const uint16_t*)x, x_tok,
                     (const uint16_t*)gamma, eps, h, (uint16_t*)y, y_tok);
  return hipGetLastError();
}

hipError_t launch_rope_rows(const sx_plan* p, const RowsArg& r, void* q, void* k, hipStream_t s) {
  const int D = p->desc.head_dim;
  const int64_t threads = (int64_t)r.max_rows * (D / 16);
  const dim3 grid((unsigned)((threads + 255) / 256), (unsigned)p->n_req);
  const bool neox = p->desc.rope_style == SX_ROPE_NEOX;
  const int Hq = p->desc.n_q_heads, Hkv = p->desc.n_kv_heads;
#define SX_ROPE(D_, N_)                                                                                               \
  hipLaunchKernelGGL((rope_rows_kernel<D_, N_>), grid, dim3(256), 0, s, p->d_req, r.rows, r.n_rows, r.max_rows, p->d_tok_pos,   \
                     p->d_theta, (uint16_t*)q, (uint16_t*)k, Hq, Hkv)
  if (D == 128) {
    if (neox) SX_ROPE(128, true); else SX_ROPE(128, false);
  } else {
    if (neox) SX_ROPE(64, true); else SX_ROPE(64, false);
  }
#undef SX_ROPE
  return hipGetLastError();
}

hipError_t launch_silu_mul_rows(const sx_plan* p, const RowsArg& r, const void* gu, int f, void* y, hipStream_t s) {
  const int64_t threads = (int64_t)r.max_rows * (f / 8);
  const dim3 grid((unsigned)((threads + 255) / 256), (unsigned)p->n_req);
  hipLaunchKernelGGL(silu_mul_rows_kernel, grid, dim3(256), 0, s, p->d_req, r.n_rows, r.max_rows, (const uint16_t*)gu, f,
                     (uint16_t*)y);
  return hipGetLastError();
}

}  // namespace sx
