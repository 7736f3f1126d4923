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
#include <type_traits>

#include "sx_device.h"
#include "sx_internal.h"

namespace sx {
namespace {

constexpr int KT = 64;     // keys per tile
constexpr int COLS = 256;  // query columns per workgroup (8 waves x 32)

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

typedef short shortx4_t __attribute__((ext_vector_type(4)));

// XOR applied to the 16-byte chunk index of row r of a V tile.  Each transposed read touches 4
// consecutive rows; this spreads their 32-byte (per 16 lanes) and 64-byte (per 32 lanes) pieces over
// distinct banks for both 128- and 256-byte-per-clock LDS service.  D = 64 rows have 8 chunks.
template <int NCH>
__device__ __forceinline__ int v_swz(int r) {
  return NCH >= 16 ? ((0xCA60 >> ((r & 3) * 4)) & 15) : ((0x4260 >> ((r & 3) * 4)) & 7);
}
typedef __attribute__((address_space(3))) shortx4_t lds_shortx4_t;

// s_waitcnt with vmcnt <= n (n < 16), expcnt and lgkmcnt left unconstrained (gfx9 encoding).
#define SX_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt(((n) & 0xF) | (0x7 << 4) | (0xF << 8))

template <int D, bool PAGED, bool PV>
__global__ __launch_bounds__(512, 1) void attn_mfma_kernel(AttnK a) {
  constexpr int NW = 8;                       // waves: two groups of 4
  constexpr int ROWB = D * 2;                 // bytes of one key row
  constexpr int NCH = ROWB / 16;              // 16-byte chunks per row
  constexpr int TILEB = KT * ROWB;            // bytes of one K (or V) tile
  constexpr int RPK = 1024 / ROWB;            // rows per 1 KB transfer instruction
  constexpr int IPW = TILEB / 1024 / NW;      // transfer instructions per wave per matrix
  // LDS: two buffers of K and V tiles, rows row-major; chunk c of row r of K sits at chunk
  // c ^ (r mod NCH) (conflict-free 16-byte row reads), of V at c ^ v_swz(r) (conflict-free
  // transposed 8-byte reads).
  __shared__ __attribute__((aligned(1024))) char K0[TILEB];
  __shared__ __attribute__((aligned(1024))) char K1[TILEB];
  __shared__ __attribute__((aligned(1024))) char V0[PV ? TILEB : 16];
  __shared__ __attribute__((aligned(1024))) char V1[PV ? TILEB : 16];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int wu = __builtin_amdgcn_readfirstlane(w);
  const int grp = wu >> 2;                    // 0: group X, 1: group Y
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
  const int row_tile = ntiles - 1 - rank;
  const int row0 = row_tile * rpw;
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
  // Q must be complete before any tile transfer is issued: the compiler does not see those
  // transfers, so a later wait of its own for Q would also wait for them.
  SX_WAIT_VMCNT(0);

  f32x16_t o[PV ? D / 32 : 1];
#pragma unroll
  for (int i = 0; i < (PV ? D / 32 : 1); ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[i][e] = 0.f;
  float m_run = -INFINITY;
  float l_run = 0.f;
  const float c2 = a.scale_log2;

  // ---- global -> LDS tile transfers (16 bytes per lane, all 8 waves share each tile).
  // Transfer q (1 KB) of a tile holds rows RPK*q .. RPK*q + RPK - 1, all inside one 16-key block;
  // keys past the end read row T-1 (they are masked: every query row is < T). ----
  const int last_key = T - 1;
  const int lrow_in = lane / NCH;     // row of this lane inside its 1 KB piece
  const int pchunk = lane % NCH;      // physical chunk this lane fills
  auto block_base = [&](const uint16_t* base, int key16) -> const uint16_t* {
    if constexpr (PAGED) {
      // the block table is read-only here: read it through the constant address space (scalar loads)
      const __attribute__((address_space(4))) int32_t* btc = (const __attribute__((address_space(4))) int32_t*)a.bt;
      const int32_t blk = btc[__builtin_amdgcn_readfirstlane(bt_off + key16)];
      return base + (((int64_t)blk * a.Hkv + kvh) * 16) * D;
    } else {
      return base + ((int64_t)(tok_off + key16 * 16) * a.Hkv + kvh) * D;
    }
  };
  constexpr int64_t kRowPaged = D;
  const int64_t rstride = PAGED ? kRowPaged : (int64_t)a.Hkv * D;   // elements between rows of a block
  const uint16_t* k_last = block_base(a.k, last_key >> 4) + (last_key & 15) * rstride;
  const uint16_t* v_last = PV ? block_base(a.v, last_key >> 4) + (last_key & 15) * rstride : nullptr;
  // One 16-byte global -> LDS transfer per lane; the destination (M0) is wave-uniform and lane l
  // lands at dst + 16 l.  Issued as inline assembly so the compiler does not order every later
  // LDS read behind it: the wait for these transfers is explicit (vmcnt(0) + barrier before a
  // tile is read).  The statement is volatile, so it stays between the barriers around it; it
  // declares no memory clobber, which keeps the read-only index loads on the scalar unit.
  auto dma16 = [&](const void* src, const char* dst) {
    const uint32_t m0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const char*)dst;
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(m0) : "m0");
  };
  auto dma16_sb = [&](const uint16_t* sbase, uint32_t voffset, const char* dst) {
    const uint32_t m0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const char*)dst;
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voffset), "s"(sbase), "s"(m0) : "m0");
  };
  // per-lane byte offsets of the transfers inside a (block, head) run; tiles start at multiples
  // of 64 keys, so they are the same for every tile
  uint32_t koff[IPW], voff[IPW];
#pragma unroll
  for (int i = 0; i < IPW; ++i) {
    const int rr = (wu * IPW + i) * RPK + lrow_in;
    koff[i] = (uint32_t)(((rr & 15) * rstride + (pchunk ^ (rr & (NCH - 1))) * 8) * 2);
    voff[i] = (uint32_t)(((rr & 15) * rstride + (pchunk ^ v_swz<NCH>(rr)) * 8) * 2);
  }
  // transfer of one matrix (K or V) tile kt into dst
  auto issue = [&](const uint16_t* base, const uint16_t* row_last, int kt, char* dst, bool is_v) {
    const int kbase = kt * KT;
    if (kbase + KT - 1 <= last_key) {
#pragma unroll
      for (int i = 0; i < IPW; ++i) {
        const int q = wu * IPW + i;
        const int kb16 = __builtin_amdgcn_readfirstlane((kbase + q * RPK) >> 4);
        dma16_sb(block_base(base, kb16), is_v ? voff[i] : koff[i], dst + q * 1024);
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < IPW; ++i) {
      const int q = wu * IPW + i;
      const int rr = q * RPK + lrow_in;
      const int key = kbase + rr;
      const int kb16 = __builtin_amdgcn_readfirstlane(min((kbase + q * RPK) >> 4, last_key >> 4));
      const int c = pchunk ^ (is_v ? v_swz<NCH>(rr) : (rr & (NCH - 1)));
      const uint16_t* blk = block_base(base, kb16);
      const uint16_t* row = key > last_key ? row_last : blk + (int64_t)(key & 15) * rstride;
      dma16(row + c * 8, dst + q * 1024);
    }
  };

  // ---- tile computations ----
  // S^T = K Q^T for the 64 keys of a tile (two 32-key M tiles)
  f32x16_t sacc[2];
  auto s_tile = [&](const char* Kb) {
    const f32x16_t zero16 = {};
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      const int rr = mt * 32 + l32;
#pragma unroll
      for (int s = 0; s < D / 16; ++s) {
        const int c = 2 * s + hg;
        const bf16x8_t ka = *(const bf16x8_t*)(Kb + rr * ROWB + ((c ^ (rr & (NCH - 1))) << 4));
        sacc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qb[s], s == 0 ? zero16 : sacc[mt], 0, 0, 0);
      }
    }
  };
  // online softmax of the tile in sacc (lane value e of M tile mt is key
  // kbase + 32 mt + 8 (e / 4) + 4 hg + e % 4 of the lane's column) -> P^T operands
  bf16x8_t pb[4];
  auto softmax_tile = [&](int kbase) {
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
    // the running max is raised only when it grows by more than 8: the O^T rescale is rare and
    // probabilities stay below 2^8
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
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      uint4 t;
      t.x = pack_bf16x2(x[8 * kk + 0], x[8 * kk + 1]);
      t.y = pack_bf16x2(x[8 * kk + 2], x[8 * kk + 3]);
      t.z = pack_bf16x2(x[8 * kk + 4], x[8 * kk + 5]);
      t.w = pack_bf16x2(x[8 * kk + 6], x[8 * kk + 7]);
      pb[kk] = __builtin_bit_cast(bf16x8_t, t);
    }
  };
  // V^T operand addressing (transposed 8-byte reads): lane 4k + c of each 16-lane group points
  // at row k, dims 4c .. 4c+3 of its 16-dim slice; the group's lane j receives dim j of 4 rows.
  const int tg = lane >> 4;
  const int tk = (lane & 15) >> 2;
  const int tc = lane & 3;
  // O^T += V^T P^T
  auto pv_tile = [&](const char* Vb) {
    if constexpr (PV) {
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) {
          // dims 32 dt + 16 (tg & 1) + 4 tc .. +3 -> 16-byte chunk, 8-byte half
          const int dchunk = 4 * dt + 2 * (tg & 1) + (tc >> 1);
          const int dhalf = (tc & 1) * 8;
          shortx4_t h2[2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            // slots 8 hg + 4h + k <-> key 16 kk + 8 h + 4 hg + k (the P^T operand order)
            const int rr = 16 * kk + 8 * h + 4 * (tg >> 1) + tk;
            const int off = rr * ROWB + ((dchunk ^ v_swz<NCH>(rr)) << 4) + dhalf;
            h2[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_shortx4_t*)(Vb + off));
          }
          const bf16x8_t va = __builtin_bit_cast(
              bf16x8_t, make_uint4(__builtin_bit_cast(uint2, h2[0]).x, __builtin_bit_cast(uint2, h2[0]).y,
                                   __builtin_bit_cast(uint2, h2[1]).x, __builtin_bit_cast(uint2, h2[1]).y));
          o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[kk], o[dt], 0, 0, 0);
        }
    }
  };

  // ---- ping-pong schedule.  Slots are separated by workgroup barriers.  Group X (waves 0-3)
  // runs its matrix phase M(j) = [P.V of tile j-1, S of tile j] in slot 2j and its softmax of tile
  // j in slot 2j+1; group Y is one slot behind.  So in every slot one wave of each SIMD issues
  // MFMAs while the other runs the softmax on the vector ALU.  Tile j's K is read in slots 2j and
  // 2j+1, its V in slots 2j+2 and 2j+3.  At the start of slot 2j the transfers of K(j+1) (into
  // the buffer of K(j-1)) and V(j) (into the buffer of V(j-2)) are issued; they are waited for at
  // the end of slot 2j+1. ----
  issue(a.k, k_last, 0, K0, false);
  SX_WAIT_VMCNT(0);
  __syncthreads();
  auto slot_start = [&](int j) {   // start of slot 2j: transfers of K(j+1) and V(j)
    if (j + 1 < nkt) issue(a.k, k_last, j + 1, ((j + 1) & 1) ? K1 : K0, false);
    if constexpr (PV) {
      if (j < nkt) issue(a.v, v_last, j, (j & 1) ? V1 : V0, true);
    }
  };
  auto matrix_phase = [&](int j) {   // M(j) = [P.V of tile j-1, S of tile j]
    if (j >= 1 && (j - 1) * KT <= wave_max) pv_tile(((j - 1) & 1) ? V1 : V0);
    if (j < nkt && j * KT <= wave_max) s_tile((j & 1) ? K1 : K0);
  };
  auto vector_phase = [&](int j) {   // softmax of tile j
    if (j >= 0 && j < nkt && j * KT <= wave_max) softmax_tile(j * KT);
  };
  // slots 2j and 2j+1 for j = 0 .. nkt; both groups pass the same barriers
  if (grp == 0) {
    for (int j = 0; j <= nkt; ++j) {
      slot_start(j);
      matrix_phase(j);
      __syncthreads();
      vector_phase(j);
      SX_WAIT_VMCNT(0);   // this wave's transfers of slot 2j have landed
      __syncthreads();
    }
  } else {
    for (int j = 0; j <= nkt; ++j) {
      slot_start(j);
      vector_phase(j - 1);
      __syncthreads();
      matrix_phase(j);
      SX_WAIT_VMCNT(0);
      __syncthreads();
    }
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
  hipLaunchKernelGGL((attn_mfma_kernel<D, PAGED, PV>), grid, dim3(512), 0, s, a);
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
