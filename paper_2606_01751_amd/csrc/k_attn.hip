// bfloat16 matrix-core kernels of the step:
//   * attention of a set of query rows over a paged or dense K/V (sparse attention of R,
//     Algorithm 1 step 21; full causal attention of the hybrid layers; and, without the PV
//     product, the log-sum-exp pass of Sparse-Q scoring, Eq. sparseq-attn);
//   * the per-key column sums of the Sparse-Q probabilities (Eq. sparseq-score).
//
// CDNA4 design (gfx950, wave64, v_mfma_f32_32x32x16_bf16):
//   * One workgroup = 8 waves = 256 query columns of one KV head; a column is a (query row,
//     query head) pair, so the G = Hq/Hkv heads that share a KV head share every K/V tile.
//   * Scores are formed transposed, S^T = K Q^T: each lane then owns one query column, so the
//     running max / sum of the online softmax stay in the lane (one cross-half exchange).
//   * The output is accumulated transposed, O^T += V^T P^T: the B operand P^T is exactly the
//     lane's own S^T accumulator registers (converted to bf16), no data movement.
//   * K and V tiles (64 keys) move global -> LDS directly (16 bytes per lane), triple-buffered;
//     they sit row-major with XOR-swizzled 16-byte chunks: conflict-free 16-byte K reads and
//     transposed 8-byte V^T reads.
//   * Ping-pong: two groups of 4 waves (one of each per SIMD) alternate a matrix phase
//     (MFMAs fed by pipelined LDS reads) and a softmax phase, so the matrix cores and the vector
//     ALU of a SIMD work at the same time; tile transfers are issued from the softmax phase.
//   * The 1-D grid is decoded KV head fastest, then request-major: the row tiles of request 0 from
//     the latest rows (most keys) to the earliest, then request 1, ...  With 8 KV heads the
//     round-robin dispatch keeps all tiles of one head on one XCD (one L2), and the workgroups
//     running there at one time mostly belong to one request, so they share its K/V tiles.
//     Sparse attention takes the same order from a per-KV-head work queue in a persistent grid
//     (about one workgroup per compute unit and KV head).
//   * Softmax in the log2 domain; the running max is raised only when a probability would reach
//     2^64, so the O^T rescale is rare and there is no max reduction on the common path.
#include <algorithm>
#include <type_traits>

#include "sx_device.h"
#include "sx_internal.h"

namespace sx {
namespace {

#ifndef SX_CS_NBUF
#define SX_CS_NBUF 3       // probe-chunk buffers of the column-sum kernel (3 to 5)
#endif
#ifndef SX_ATTN_NBUF
#define SX_ATTN_NBUF 3     // K/V tile buffers of the attention kernel (3 or 4; 4 measured no faster)
#endif
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
  int grid_rows;   // paged: rows of a request beyond this bound are not processed
  float scale_log2;
  int lse_base2;
  // log-sum-exp pass (paged, no P.V): each row tile's keys in nsplit pieces of whole 16-tile
  // groups; with nsplit > 1 every piece writes its (max, sum) to lse_part[piece][probe row][Hq]
  // (probe rows of all requests concatenated) and lse_merge_kernel forms the log-sum-exp
  int nsplit;
  float2* lse_part;
  int64_t n_part_rows;
  // persistent grids: per-KV-head work queues, [0, Hkv) items taken and [Hkv] the workgroups
  // finished, zero between launches (sparse attention: the plan's; full attention: slot qslot of
  // g_dense_queue)
  int32_t* queue;
  int qslot;
  // sparse attention: planned order of the queue items (tile_order_kernel; NULL or out[0] != the
  // item count: the queue's own order)
  const int32_t* order;
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
// Scheduling groups (instruction classes of the sched_group_barrier builtin): the next `n`
// instructions of class `mask` are placed here, in program order of the groups.
#define SX_SG(mask, n) __builtin_amdgcn_sched_group_barrier(mask, n, 0)
constexpr int kSgValu = 0x2, kSgMfma = 0x8, kSgDsRead = 0x100;
// Order of a matrix phase of NM MFMAs whose operands come from NR LDS reads each: the reads of
// the first PRE MFMAs go first, then every MFMA is followed by the reads of the MFMA PRE places
// later, so each read has PRE MFMAs (32 cycles each) to complete.
template <int NM, int NR, int PRE>
__device__ __forceinline__ void sched_pipelined() {
  SX_SG(kSgDsRead, NR * PRE);
#pragma unroll
  for (int i = 0; i < NM - PRE; ++i) {
    SX_SG(kSgMfma, 1);
    SX_SG(kSgDsRead, NR);
  }
  SX_SG(kSgMfma, PRE);
}

// The kernel arguments for one item of a persistent kernel: read from the kernel-argument segment
// (where the by-value argument sits at offset 0) through a pointer the compiler cannot follow, so
// the loads stay inside the item and nothing of them is kept across items.
template <bool RELOAD>
__device__ __forceinline__ AttnK item_args(const AttnK& k) {
  if constexpr (RELOAD) {
    typedef const __attribute__((address_space(4))) char* ArgPtr;
    ArgPtr p = (ArgPtr)__builtin_amdgcn_kernarg_segment_ptr();
    asm volatile("" : "+s"(p));
    return *(const AttnK*)(const char*)p;
  } else {
    return k;
  }
}

// Work-queue counters of persistent full attention, which has no plan: kDenseQueueSlots slots of
// kDenseQueueStride counters on every device, a launch using slot qslot (the host hands the slots
// out in turn, so launches that overlap in time use different slots; each launch leaves its slot
// zero).
__device__ int32_t g_dense_queue[kDenseQueueSlots * kDenseQueueStride];

template <int D, bool PAGED, bool PV, bool PERSIST>
__global__ __launch_bounds__(512, 1) void attn_mfma_kernel(AttnK ka) {
  constexpr int NW = 8;                       // waves: two groups of 4
  constexpr int ROWB = D * 2;                 // bytes of one key row
  constexpr int NCH = ROWB / 16;              // 16-byte chunks per row
  constexpr int TILEB = KT * ROWB;            // bytes of one K (or V) tile
  constexpr int RPK = 1024 / ROWB;            // rows per 1 KB transfer instruction
  constexpr int IPW = TILEB / 1024 / NW;      // transfer instructions per wave per matrix
  static_assert(IPW * RPK == 8, "a wave moves 8 consecutive rows of every tile");
  // LDS: NBUF buffers each of K and V tiles (tile t in buffer t mod NBUF), rows row-major; chunk c
  // of row r of K sits at chunk c ^ (r mod NCH) (conflict-free 16-byte row reads), of V at
  // c ^ v_swz(r) (conflict-free transposed 8-byte reads).  A tile is issued NBUF - 1 (K) or
  // NBUF - 2 (V) iterations before it is read.
  constexpr int NBUF = SX_ATTN_NBUF;
  static_assert(NBUF == 3 || NBUF == 4, "three or four tile buffers");
  __shared__ __attribute__((aligned(1024))) char smem[(PV ? 2 : 1) * NBUF * TILEB];
  char* const kbuf = smem;
  char* const vbuf = smem + (PV ? NBUF * TILEB : 0);

  // (the remainder is formed on the vector unit; in the paged kernel the empty asm keeps the uniform
  // result in a scalar register, so the block addresses built from it stay on the scalar unit)
  int kvh = __builtin_amdgcn_readfirstlane((int)(blockIdx.x % (unsigned)ka.Hkv));
  if constexpr (PAGED) asm("" : "+s"(kvh));
  // Request-major order: for each KV head, the row tiles of request 0 (latest rows, i.e. most keys,
  // first), then those of request 1, ...  The workgroups running together on one XCD then mostly
  // belong to one request and share its K/V tiles through that XCD's L2.  (Pieces of one row tile
  // are adjacent.)  The log-sum-exp pass launches one workgroup per item.  Attention with output
  // (sparse, and full attention outside graph capture) runs a persistent grid instead: about one
  // workgroup per compute unit and KV head, each taking its head's next item from that head's
  // queue whenever it finishes one.  The items then go to whichever compute unit frees first
  // (greedy longest-first, or the planned order of tile_order_kernel), with no gap for the
  // hardware to dispatch another workgroup; the hardware's own dispatch hands the workgroups of an
  // XCD to its shader engines in turn and holds the rest back while the next one's engine is full,
  // which left a tenth of the compute units idle in the tail.  A workgroup whose head's queue is
  // empty moves on to the head whose queue holds the most items (the XCDs do not run at one speed,
  // so the fast ones finish the slow ones' last, lightest items), and stops when every queue is
  // empty.  The last workgroup to stop resets the counters for the next launch.
  static_assert(!PERSIST || PV, "persistent grids run attention with output only");
  int32_t* const queue = PAGED ? ka.queue : g_dense_queue + ka.qslot * kDenseQueueStride;
  __shared__ int2 s_take[2];   // (head, item) taken by wave 0, alternating slots
  int item = (int)(blockIdx.x / (unsigned)ka.Hkv);
  int takes = 0, n_items = 0;
  if constexpr (PERSIST) {
    // items of one head (every head has the same): row tiles of all requests
    for (int c0 = 0; c0 < ka.n_req; c0 += 64) {
      const int rr = c0 + (int)(threadIdx.x & 63);
      const int nr = rr >= ka.n_req ? 0 : PAGED ? min(ka.n_rows[rr], ka.grid_rows) : ka.cu[rr + 1] - ka.cu[rr];
      int c = (nr + ka.rpw - 1) / ka.rpw;
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) c += __shfl_xor(c, o, 64);
      n_items += __builtin_amdgcn_readfirstlane(c);
    }
  }
  const bool use_order = PERSIST && PAGED && ka.order && ka.order[0] == n_items;
  for (;;) {
    if constexpr (PERSIST) {
      // wave 0 takes the next item: from head kvh's queue, else from the fullest other queue (the
      // counters read in one round trip, one lane per head); (-1, -1) when every queue is empty
      if (threadIdx.x < 64) {
        int2 t = make_int2(-1, -1);
        for (;;) {
          int v = 0;
          if (threadIdx.x == 0)
            v = __hip_atomic_fetch_add(queue + kvh, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          v = __builtin_amdgcn_readfirstlane(v);
          if (v < n_items) {
            t = make_int2(kvh, use_order ? ka.order[1 + v] : v);
            break;
          }
          int left = 0;
          for (int h0 = 0; h0 < ka.Hkv; h0 += 64) {
            const int h = h0 + (int)threadIdx.x;
            const int cnt =
                h < ka.Hkv ? __hip_atomic_load(queue + h, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : n_items;
            const int rem = n_items - min(cnt, n_items);
            int mx = rem;
#pragma unroll
            for (int o = 32; o >= 1; o >>= 1) mx = max(mx, __shfl_xor(mx, o, 64));
            mx = __builtin_amdgcn_readfirstlane(mx);
            if (mx > left) {   // most items left, then the lowest head
              left = mx;
              kvh = h0 + (int)__ffsll((unsigned long long)__ballot(rem == mx)) - 1;
            }
          }
          if (left == 0) break;
        }
        if (threadIdx.x == 0) s_take[takes & 1] = t;
      }
      __syncthreads();
      const int2 t = s_take[takes & 1];
      ++takes;
      kvh = __builtin_amdgcn_readfirstlane(t.x);
      asm("" : "+s"(kvh));
      item = __builtin_amdgcn_readfirstlane(t.y);
      if (kvh < 0) break;
    }
    // The kernel arguments and the lane values are formed again for every item (from the argument
    // segment and the thread index, both through opaque copies) rather than hoisted out of the item
    // loop and kept live through the tile loop, which would leave no registers for the pipelined
    // operand reads.
    const AttnK a = item_args<PERSIST>(ka);
    int tid = threadIdx.x;
    if constexpr (PERSIST) asm volatile("" : "+v"(tid));
    const int lane = tid & 63;
    const int w = tid >> 6;
    const int wu = __builtin_amdgcn_readfirstlane(w);
    const int grp = wu >> 2;                    // 0: group X, 1: group Y
    const int l32 = lane & 31;
    const int hg = lane >> 5;
    const int rpw = a.rpw;
    const int nsplit = (PAGED && !PV) ? a.nsplit : 1;
    // rows of request rr that are processed: the first min(n_rows, max_rows) rows (the rows the KV
    // write of the same row list covers), or every row of a dense request
    auto rows_of = [&](int rr) -> int {
      if constexpr (PAGED) return min(a.n_rows[rr], a.grid_rows);
      else return a.cu[rr + 1] - a.cu[rr];
    };
    int r, qi;
    locate_request(item, a.n_req, [&](int rr) { return (rows_of(rr) + rpw - 1) / rpw * nsplit; }, &r, &qi, lane);
    r = __builtin_amdgcn_readfirstlane(r);   // (uniform: the loop exit below is a uniform branch)
    qi = __builtin_amdgcn_readfirstlane(qi);
    if (r < 0) break;
    const int rank = qi / nsplit;
    const int piece = qi - rank * nsplit;

    int T, tok_off, bt_off = 0, nrows, p_off = 0;
    if constexpr (PAGED) {
      const ReqDev rq = a.reqs[r];
      T = rq.T;
      tok_off = rq.tok_off;
      bt_off = rq.bt_off;
      p_off = rq.p_off;
    } else {
      tok_off = a.cu[r];
      T = a.cu[r + 1] - tok_off;
    }
    if constexpr (PAGED) {
      // (request fields are workgroup-uniform: scalar registers keep the block address math on the
      // scalar unit)
      T = __builtin_amdgcn_readfirstlane(T);
      tok_off = __builtin_amdgcn_readfirstlane(tok_off);
      bt_off = __builtin_amdgcn_readfirstlane(bt_off);
      p_off = __builtin_amdgcn_readfirstlane(p_off);
    }
    nrows = rows_of(r);
    const int ntiles = (nrows + rpw - 1) / rpw;
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
    const int wave_max = wave_max_i(pos, lane);
    const int wave_min = wave_min_i(valid ? pos : 0x7fffffff, lane);
    const int qh = kvh * a.G + hh;
    const float c2 = a.scale_log2;
    // key tiles [kt0, kt0 + nkt) of this workgroup: all of them, or one piece of whole 16-tile groups
    const int nkt_all = wg_max / KT + 1;
    int kt0 = 0, nkt = nkt_all;
    if (nsplit > 1) {
      const int tpp = ((nkt_all + nsplit - 1) / nsplit + 15) & ~15;
      kt0 = piece * tpp;
      nkt = min(tpp, nkt_all - kt0);
      if (nkt <= 0) {   // no keys in this piece: an empty partial (uniform over the workgroup)
        if (valid && hg == 0)
          a.lse_part[((int64_t)piece * a.n_part_rows + p_off + ridx) * a.Hq + qh] = make_float2(-INFINITY, 0.f);
        return;
      }
    }

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
    // Block table (paged caches): a wave moves rows 8 wu .. 8 wu + 7 of every tile, all inside
    // logical block 4 t + wu / 2 of tile t, so one block id per wave and tile (a scalar load through
    // the constant address space, clamped to the request's last block for tiles past the end).
    const int nblk = (T + 15) >> 4;
    auto blk_of = [&](int kt) -> int32_t {
      if constexpr (PAGED) {
        const __attribute__((address_space(4))) int32_t* btc = (const __attribute__((address_space(4))) int32_t*)a.bt;
        return btc[__builtin_amdgcn_readfirstlane(bt_off + min(4 * kt + (wu >> 1), nblk - 1))];
      } else {
        return 0;
      }
    };
    // Q must be complete before any tile transfer is issued: the compiler does not see those
    // transfers, so a later wait of its own for Q would also wait for them.
    SX_WAIT_VMCNT(0);

    f32x16_t o[PV ? D / 32 : 1];
#pragma unroll
    for (int i = 0; i < (PV ? D / 32 : 1); ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[i][e] = 0.f;
    // running max (log2 domain); columns without a row start at 0 so their (unused) sums stay finite
    float m_run = valid ? -INFINITY : 0.f;
    float l_run = 0.f;

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
    // base of the rows this wave moves in key tile kt: the (block, head) run of block blk (paged), or
    // the tile's 16-row group of this wave (dense; rows past the end are not read through it)
    auto wave_base = [&](const uint16_t* base, int kt, int32_t blk) -> const uint16_t* {
      if constexpr (PAGED) return base + (((int64_t)blk * a.Hkv + kvh) * 16) * D;
      else return block_base(base, ((kt * KT) >> 4) + (wu >> 1));
    };
    constexpr int64_t kRowPaged = D;
    const int64_t rstride = PAGED ? kRowPaged : (int64_t)a.Hkv * D;   // elements between rows of a block
    const uint16_t* k_last = block_base(a.k, last_key >> 4) + (last_key & 15) * rstride;
    const uint16_t* v_last = PV ? block_base(a.v, last_key >> 4) + (last_key & 15) * rstride : nullptr;
    // One 16-byte global -> LDS transfer per lane; the destination (M0) is wave-uniform and lane l
    // lands at dst + 16 l.  Issued as inline assembly so the compiler does not order every later
    // LDS read behind it: the wait for these transfers is explicit (vmcnt + barrier before a tile
    // is read).  The statement is volatile, so it stays between the barriers around it; it
    // declares no memory clobber, which keeps the read-only index loads on the scalar unit.
    auto dma16 = [&](const void* src, const char* dst) {
      const uint32_t m0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const char*)dst;
      asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(m0) : "m0", "memory");
    };
    auto dma16_sb = [&](const uint16_t* sbase, uint32_t voffset, const char* dst) {
      const uint32_t m0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const char*)dst;
      // the base is wave-uniform; readfirstlane makes that visible where the compiler cannot prove it
      // (the instruction takes its base from an SGPR pair)
      // (the builtin returns a signed int: each half goes through uint32_t so that nothing is sign-extended)
      const uint64_t sb = (uint64_t)(uintptr_t)sbase;
      const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)sb);
      const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(sb >> 32));
      const uint64_t sbu = ((uint64_t)hi << 32) | (uint64_t)lo;
      asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voffset), "s"(sbu), "s"(m0)
                   : "m0", "memory");
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
    // transfer of this wave's share of one matrix (K or V) tile kt into dst; blk = blk_of(kt)
    auto issue = [&](const uint16_t* base, const uint16_t* row_last, int kt, char* dst, bool is_v, int32_t blk) {
      const int kbase = kt * KT;
      if (kbase + KT - 1 <= last_key) {
        const uint16_t* b = wave_base(base, kt, blk);
#pragma unroll
        for (int i = 0; i < IPW; ++i) {
          const int q = wu * IPW + i;
          dma16_sb(b, is_v ? voff[i] : koff[i], dst + q * 1024);
        }
        return;
      }
      // the tile crosses the end: the wave's rows past the last key read row T-1 (when the wave's
      // whole block is past the end, its block is clamped to the last one and every row reads row T-1)
#pragma unroll
      for (int i = 0; i < IPW; ++i) {
        const int q = wu * IPW + i;
        const int rr = q * RPK + lrow_in;
        const int key = kbase + rr;
        const int c = pchunk ^ (is_v ? v_swz<NCH>(rr) : (rr & (NCH - 1)));
        const uint16_t* b =
            PAGED ? wave_base(base, kt, blk)
                  : block_base(base, __builtin_amdgcn_readfirstlane(min((kbase + q * RPK) >> 4, last_key >> 4)));
        const uint16_t* row = key > last_key ? row_last : b + (int64_t)(key & 15) * rstride;
        dma16(row + c * 8, dst + q * 1024);
      }
    };
    auto ktile = [&](int t) { return kbuf + (t % NBUF) * TILEB; };
    auto vtile = [&](int t) { return vbuf + (t % NBUF) * TILEB; };
    constexpr int KD = NBUF - 1, VD = NBUF - 2;   // issue distances of K and V tiles (iterations)
    // the same buffers as LDS byte addresses (wave-uniform: the operand reads add a lane offset)
    const uint32_t kbuf_lds = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)kbuf;
    const uint32_t vbuf_lds = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)vbuf;
    auto ktile_lds = [&](int t) { return kbuf_lds + (uint32_t)((t % NBUF) * TILEB); };
    auto vtile_lds = [&](int t) { return vbuf_lds + (uint32_t)((t % NBUF) * TILEB); };
    // wait until at most n of this wave's tile transfers (the youngest) are still in flight
    auto wait_vm = [&](int n) {
      switch (n) {
        case 0: SX_WAIT_VMCNT(0); break;
        case 1: SX_WAIT_VMCNT(1); break;
        case 2: SX_WAIT_VMCNT(2); break;
        case 3: SX_WAIT_VMCNT(3); break;
        case 4: SX_WAIT_VMCNT(4); break;
        case 5: SX_WAIT_VMCNT(5); break;
        case 6: SX_WAIT_VMCNT(6); break;
        case 7: SX_WAIT_VMCNT(7); break;
        case 8: SX_WAIT_VMCNT(8); break;
        case 9: SX_WAIT_VMCNT(9); break;
        default: SX_WAIT_VMCNT(10); break;
      }
    };
    static_assert((NBUF - 2) * (2 * IPW + 1) <= 10, "transfers in flight exceed the wait table");

    // ---- tile computations ----
    // S^T = K Q^T for the 64 keys of a tile (two 32-key M tiles)
    f32x16_t sacc[2];
    // K operand addressing: lane reads row 32 mt + l32, logical chunk 2 s + hg.  The swizzle depends
    // on the row only through l32 mod NCH, so the lane part of the address is one value per k-slice
    // s (computed once) and the second row block adds a constant (an immediate offset).
    int k_off[D / 16];
#pragma unroll
    for (int s = 0; s < D / 16; ++s) k_off[s] = l32 * ROWB + (((2 * s + hg) ^ (l32 & (NCH - 1))) << 4);
    // Kb: the tile's LDS address; `fixed` when it is a compile-time constant (the buffer offset then
    // folds into the reads' immediate offsets), else made opaque (one add per k-slice, no
    // strength-reduced variants)
    auto s_body = [&](uint32_t Kb, auto fixed) {
      if constexpr (!decltype(fixed)::value) asm volatile("" : "+s"(Kb));
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int e = 0; e < 16; ++e) sacc[mt][e] = 0.f;
#pragma unroll
      for (int s = 0; s < D / 16; ++s) {
        uint32_t kbase = Kb + (uint32_t)k_off[s];
        if constexpr (!decltype(fixed)::value) asm volatile("" : "+v"(kbase));
#pragma unroll
        for (int mt = 0; mt < 2; ++mt) {
          const bf16x8_t ka =
              *(const __attribute__((address_space(3))) bf16x8_t*)(uintptr_t)(kbase + (uint32_t)(mt * 32 * ROWB));
          sacc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qb[s], sacc[mt], 0, 0, 0);
        }
      }
    };
    auto s_tile = [&](uint32_t Kb, auto fixed) {
      s_body(Kb, fixed);
      sched_pipelined<D / 8, 1, 4>();
    };
    // online softmax of the tile in sacc (lane value e of M tile mt is key
    // kbase + 32 mt + 8 (e / 4) + 4 hg + e % 4 of the lane's column) -> P^T operands.
    // The running max m_run is not raised tile by tile: p is formed against the current m_run and
    // m_run is raised (with the O^T / l rescale) only when some p of the wave reaches 2^64 or is not
    // finite -- on the first tile of a column and when scores grow by more than about 59 in log2
    // units.  Every p then stays below 2^64, so P, l and O^T keep their float32 / bfloat16
    // relative precision and cannot overflow; the result is the same softmax.
    bf16x8_t pb[4];
    auto softmax_tile = [&](int kbase) {
      if (kbase + KT - 1 > wave_min) {
        // keys with offset > lim get -inf; a per-element bit select (no lane-mask registers)
        const int lim = pos - kbase - hg * 4;
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int koff = mt * 32 + (e >> 2) * 8 + (e & 3);
            const uint32_t m = (uint32_t)((lim - koff) >> 31);   // all ones where koff > lim
            sacc[mt][e] = __uint_as_float((__float_as_uint(sacc[mt][e]) & ~m) | (0xff800000u & m));
          }
      }
      float psum = 0.f;
      // 8 probabilities of slot group kk -> packed P^T operand, added to psum
      auto emit = [&](int kk, const float* x) {
        uint4 u;
        u.x = pack_bf16x2(x[0], x[1]);
        u.y = pack_bf16x2(x[2], x[3]);
        u.z = pack_bf16x2(x[4], x[5]);
        u.w = pack_bf16x2(x[6], x[7]);
        pb[kk] = __builtin_bit_cast(bf16x8_t, u);
        // l sums the float32 probabilities (exact denominators, also for the log-sum-exp output)
#pragma unroll
        for (int t = 0; t < 8; ++t) psum += x[t];
      };
      auto tile_max = [&]() {
        float mx = sacc[0][0];
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
          for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sacc[mt][e]);
        return fmaxf(mx, __shfl_xor(mx, 32, 64));
      };
      auto rescale = [&](float alpha) {
        l_run *= alpha;
        if constexpr (PV) {
#pragma unroll
          for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
            for (int e = 0; e < 16; ++e) o[dt][e] *= alpha;
        }
      };
      // p = 2^(c2 s - m_run)
      auto expo = [&](float mneg) {
        psum = 0.f;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          float x[8];
#pragma unroll
          for (int t = 0; t < 8; ++t)
            x[t] = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kk >> 1][(kk & 1) * 8 + t], c2, mneg));
          emit(kk, x);
        }
      };
      expo(-m_run);
      if (__ballot(!(psum < 0x1p64f))) {
        const float m_new = fmaxf(m_run, tile_max() * c2);          // c2 > 0
        rescale(m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new));
        m_run = m_new;
        expo(m_new == -INFINITY ? 0.f : -m_new);
      }
      l_run += psum;
    };
    // V^T operand addressing (transposed 8-byte reads): lane 4k + c of each 16-lane group points
    // at row k, dims 4c .. 4c+3 of its 16-dim slice; the group's lane j receives dim j of 4 rows.
    const int tg = lane >> 4;
    const int tk = (lane & 15) >> 2;
    const int tc = lane & 3;
    // O^T += V^T P^T
    // Lane part of the V^T read offsets, one per 32-dim tile: row 4 (tg >> 1) + tk of an 8-row
    // group, dims 32 dt + 16 (tg & 1) + 4 tc .. +3 (16-byte chunk, 8-byte half).  The swizzle
    // depends on the row only through row mod 4 = tk, so rows 16 kk + 8 h add a constant.
    int vtr_off[D / 32];
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
      const int dchunk = 4 * dt + 2 * (tg & 1) + (tc >> 1);
      vtr_off[dt] = (4 * (tg >> 1) + tk) * ROWB + ((dchunk ^ v_swz<NCH>(tk)) << 4) + (tc & 1) * 8;
    }
    auto pv_body = [&](uint32_t Vb, auto fixed) {
      if constexpr (PV) {
        if constexpr (!decltype(fixed)::value) asm volatile("" : "+s"(Vb));
        // one base address per 32-dim tile for this tile's buffer (the empty asm keeps the compiler
        // from re-associating the sums into one precomputed register per read); every read then
        // adds its row constant as an immediate offset
        uint32_t vbase[D / 32];
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) {
          vbase[dt] = Vb + (uint32_t)vtr_off[dt];
          if constexpr (!decltype(fixed)::value) asm volatile("" : "+v"(vbase[dt]));
        }
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
#pragma unroll
          for (int dt = 0; dt < D / 32; ++dt) {
            shortx4_t h2[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              // slots 8 hg + 4h + k <-> key 16 kk + 8 h + 4 hg + k (the P^T operand order)
              h2[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                  (lds_shortx4_t*)(uintptr_t)(vbase[dt] + (uint32_t)((16 * kk + 8 * h) * ROWB)));
            }
            const bf16x8_t va = __builtin_bit_cast(
                bf16x8_t, make_uint4(__builtin_bit_cast(uint2, h2[0]).x, __builtin_bit_cast(uint2, h2[0]).y,
                                     __builtin_bit_cast(uint2, h2[1]).x, __builtin_bit_cast(uint2, h2[1]).y));
            o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[kk], o[dt], 0, 0, 0);
          }
      }
    };
    auto pv_tile = [&](uint32_t Vb, auto fixed) {
      if constexpr (PV) {
        pv_body(Vb, fixed);
        sched_pipelined<D / 8, 2, 4>();
      }
    };


    // ---- ping-pong schedule over iterations j = 0 .. nkt.  Iteration j has two slots separated by
    // workgroup barriers.  Group X (waves 0-3) runs its matrix phase M(j) = [P.V of tile j-1, S of
    // tile j] in the first slot and the softmax of tile j in the second; group Y runs the softmax of
    // tile j-1 in the first slot and M(j) in the second.  So in every slot one wave of each SIMD
    // issues MFMAs while the other runs the softmax on the vector ALU.
    // Tiles rotate through NBUF buffers: at the start of its softmax slot of iteration j each wave
    // issues its share of the transfers of K(j+KD) and V(j+VD) (an issue that waits for the address
    // unit then delays vector work, not MFMAs; issued at the end of the matrix phase instead they cost
    // both attention kernels about 6 %); they have NBUF - 2 iterations to land (waited for at the end
    // of iteration j + NBUF - 3) before they are read, and their buffers were last read in iteration
    // j-1. ----
    auto ncur = [&](int j) {   // transfers this wave issues in iteration j
      return (j + KD >= 0 && j + KD < nkt ? IPW : 0) + (PV && j + VD >= 0 && j + VD < nkt ? IPW : 0);
    };
    // transfers of iterations j - NBUF + 4 .. j may still be in flight at the end of iteration j
    auto inflight = [&](int j) {
      int n = ncur(j);
      if constexpr (NBUF == 4) n += ncur(j - 1);
      return n;
    };
    // (iteration j works on key tile kt0 + j; the LDS buffers rotate with j.)  Prologue: K(0), then
    // the transfers that iterations -(NBUF-2) .. -1 would have issued.
    issue(a.k, k_last, kt0, ktile(0), false, blk_of(kt0));
#pragma unroll
    for (int jj = -(NBUF - 2); jj < 0; ++jj) {
      if (jj + KD < nkt) issue(a.k, k_last, kt0 + jj + KD, ktile(jj + KD), false, blk_of(kt0 + jj + KD));
      if constexpr (PV) {
        if (jj + VD < nkt) issue(a.v, v_last, kt0 + jj + VD, vtile(jj + VD), true, blk_of(kt0 + jj + VD));
      }
    }
    // block ids of the next transfer phase (scalar loads one iteration ahead, so their wait is never
    // on the loop's critical path): V(j + VD) is the tile of the previous phase's K (VD = KD - 1)
    static_assert(VD == KD - 1, "the V tile of a transfer phase is the K tile of the one before");
    int32_t blk_k = blk_of(kt0 + KD), blk_v = blk_of(kt0 + KD - 1);
    wait_vm(inflight(-1));   // K(0) has landed
    __syncthreads();
    // `ph` is j mod NBUF when known at compile time (integral constant >= 0), else -1: the tile
    // buffers of the iteration are then constants
    auto matrix_phase = [&](int j, auto ph) {
      constexpr int PH = decltype(ph)::value;
      constexpr bool FX = PH >= 0;
      // the wave in its matrix phase issues first: its MFMAs are not held back by the other
      // wave's softmax on the same SIMD
      __builtin_amdgcn_s_setprio(2);
      if (j >= 1 && j - 1 < nkt && (kt0 + j - 1) * KT <= wave_max)
        pv_tile(FX ? vbuf_lds + (uint32_t)(((PH + NBUF - 1) % NBUF) * TILEB) : vtile_lds(j - 1),
                std::integral_constant<bool, FX>{});
      if (j < nkt && (kt0 + j) * KT <= wave_max)
        s_tile(FX ? kbuf_lds + (uint32_t)(PH * TILEB) : ktile_lds(j), std::integral_constant<bool, FX>{});
      __builtin_amdgcn_s_setprio(0);
    };
    // this wave's share of K(j+KD) and V(j+VD); tph = j mod NBUF (wave-uniform)
    auto transfer_phase = [&](int j, int tph) {
      const int kb = tph + KD >= NBUF ? tph + KD - NBUF : tph + KD;
      const int vb = tph + VD >= NBUF ? tph + VD - NBUF : tph + VD;
      if (j + KD < nkt) issue(a.k, k_last, kt0 + j + KD, kbuf + kb * TILEB, false, blk_k);
      if constexpr (PV) {
        if (j + VD < nkt) issue(a.v, v_last, kt0 + j + VD, vbuf + vb * TILEB, true, blk_v);
      }
      if constexpr (PAGED) {
        // a wave calls this once per iteration, in order: prefetch the next call's K block
        blk_v = blk_k;
        blk_k = blk_of(kt0 + j + 1 + KD);
      }
    };
    auto vector_phase = [&](int j) {   // softmax of tile j
      if (j >= 0 && j < nkt && (kt0 + j) * KT <= wave_max) softmax_tile((kt0 + j) * KT);
    };
    // Both groups run one loop body, U(j) = M(j) | barrier | T(j + grp), softmax of tile j | barrier.
    // Group Y (grp = 1) is half an iteration ahead: it issues T(0) and passes one barrier before its
    // first U, so its matrix phase M(j) runs beside group X's softmax of tile j - 1 and its softmax of
    // tile j beside X's M(j + 1).  A wave waits for its transfers of iteration j - NBUF + 3 (all but
    // those of T(j), the youngest) before the barrier that precedes its next matrix phase.  Every loop
    // trip runs NBUF iterations with static buffer phases (every LDS offset of the matrix phase an
    // immediate); iterations past nkt only pass their barriers.  Both groups pass the same number of
    // barriers: Y's extra one at the start, X's at the end.
    const int g1 = __builtin_amdgcn_readfirstlane(grp);
    if (g1) {
      transfer_phase(0, 0);
      __syncthreads();
    }
    auto iter_u = [&](int j, auto ph) {
      constexpr int PH = decltype(ph)::value;
      matrix_phase(j, ph);
      if (g1) wait_vm(inflight(j));
      __syncthreads();
      transfer_phase(j + g1, PH + g1 >= NBUF ? PH + g1 - NBUF : PH + g1);
      vector_phase(j);
      if (!g1) wait_vm(inflight(j));
      __syncthreads();
    };
    for (int j = 0; j <= nkt; j += NBUF) {
      iter_u(j, std::integral_constant<int, 0>{});
      iter_u(j + 1, std::integral_constant<int, 1>{});
      iter_u(j + 2, std::integral_constant<int, 2>{});
      if constexpr (NBUF == 4) iter_u(j + 3, std::integral_constant<int, 3>{});
    }
    if (!g1) __syncthreads();

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
    if (nsplit > 1) {
      if (valid && hg == 0)
        a.lse_part[((int64_t)piece * a.n_part_rows + p_off + ridx) * a.Hq + qh] = make_float2(m_run, l_tot);
    } else if (a.lse && valid && hg == 0) {
      const float lse2 = m_run + __log2f(l_tot);
      a.lse[(int64_t)(tok_off + ridx) * a.Hq + qh] = a.lse_base2 ? lse2 : lse2 * 0.69314718055994531f;
    }
    if constexpr (!PERSIST) break;
  }
  if constexpr (PERSIST) {
    if (threadIdx.x == 0) {
      const int done = __hip_atomic_fetch_add(queue + ka.Hkv, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (done == (int)gridDim.x - 1)
        for (int h = 0; h <= ka.Hkv; ++h)
          __hip_atomic_store(queue + h, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// Order in which persistent sparse attention takes its row tiles (the same for every KV head), from
// the tiles' estimated costs: key tiles up to the tile's last row plus kOrderCost0 for the work
// outside the tile loop.  Taking the tiles longest first (the queue's own order) is the greedy
// longest-processing-time schedule; this kernel plans a tighter one with Multifit (the smallest
// bin capacity for which first-fit-decreasing packs the tiles into m bins, m being the
// workgroups per head, found by a parallel search over candidate capacities), the m largest tiles
// opening the bins, and lists the tiles by their planned start, so that the workgroups, each
// taking the next tile when it finishes one, follow the plan.  One workgroup of 1024 threads; out[0] = number of tiles n, out[1 + k] = the
// queue item taken k-th; out[0] = -1 (the queue's order) when n > 8 m or m > 64.
// Every item index of [0, n) appears exactly once, whatever the costs.
constexpr int kOrderCost0 = 4;

// Position of key[i] among key[0, n) in ascending order (the keys are distinct; key is 16-byte
// aligned and holds 0xFFFFFFFF from n up to the next multiple of 4).
__device__ __forceinline__ int rank_of(const uint32_t* key, int n, int i) {
  const uint32_t k = key[i];
  int r = 0;
#pragma unroll 4
  for (int j = 0; j < n; j += 4) {
    const uint4 q = *(const uint4*)(key + j);
    r += (q.x < k ? 1 : 0) + (q.y < k ? 1 : 0) + (q.z < k ? 1 : 0) + (q.w < k ? 1 : 0);
  }
  return r;
}

__global__ __launch_bounds__(1024) void tile_order_kernel(const ReqDev* __restrict__ reqs,
                                                          const int32_t* __restrict__ rows,
                                                          const int32_t* __restrict__ n_rows, int max_rows,
                                                          int n_req, int rpw, int m, int32_t* __restrict__ out) {
  constexpr int NMAX = kOrderMax;   // items planned: at most 8 per bin, at most 64 bins
  static_assert(NMAX == 8 * 64, "eight items per bin, 64 bins");
  __shared__ __attribute__((aligned(16))) uint32_t key[NMAX];
  __shared__ int32_t item[NMAX];   // queue item of the k-th largest cost
  __shared__ int32_t cost[NMAX];   // its cost
  __shared__ uint32_t plan[16][NMAX];   // each wave's packing: planned start << 6 | bin per item
  __shared__ int s_n, s_sum, s_max, s_lo, s_hi, s_hi0, s_best, s_fail;
  __shared__ int s_ok[16];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  if (tid == 0) {
    int n = 0;
    for (int r = 0; r < n_req; ++r) n += (min(n_rows[r], max_rows) + rpw - 1) / rpw;
    s_n = n;
    s_sum = 0;
    s_max = 0;
  }
  __syncthreads();
  const int n = s_n;
  if (n > NMAX || n > 8 * m || m > 64 || m < 1 || n == 0) {
    if (tid == 0) out[0] = n == 0 ? 0 : -1;
    return;
  }
  // costs in the queue's item order (request-major, each request's last row tile first), keyed for
  // decreasing cost, then increasing item
  int base = 0;
  for (int r = 0; r < n_req; ++r) {
    const int nr = min(n_rows[r], max_rows);
    const int t = (nr + rpw - 1) / rpw;
    const int tok_off = reqs[r].tok_off;
    for (int rank = tid; rank < t; rank += blockDim.x) {
      const int row_tile = t - 1 - rank;
      const int last = min((row_tile + 1) * rpw, nr) - 1;
      const int c = rows[tok_off + last] / KT + 1 + kOrderCost0;
      key[base + rank] = ((uint32_t)(0xFFFF - min(c, 0xFFFF)) << 16) | (uint32_t)(base + rank);
      atomicAdd(&s_sum, c);
      atomicMax(&s_max, c);
    }
    base += t;
  }
  for (int i = n + tid; i < ((n + 3) & ~3); i += blockDim.x) key[i] = 0xFFFFFFFFu;
  __syncthreads();
  for (int i = tid; i < n; i += blockDim.x) {
    const int k = rank_of(key, n, i);
    item[k] = (int)(key[i] & 0xFFFF);
    cost[k] = 0xFFFF - (int)(key[i] >> 16);
  }
  if (tid == 0) {
    const int lb = max(s_max, (s_sum + m - 1) / m);
    s_lo = lb - 1;                                   // no packing fits below the lower bound
    s_hi0 = max(s_max, (2 * s_sum + m - 1) / m);     // first-fit decreasing always fits here
    s_hi = min(s_hi0, lb + lb / 4 + 1);              // where it usually fits already
    s_best = -1;
    s_fail = 0;
  }
  __syncthreads();
  // every wave holds the costs in registers: lane l has cost[l + 64 k] in creg[k]
  int creg[NMAX / 64];
#pragma unroll
  for (int k = 0; k < NMAX / 64; ++k) creg[k] = lane + 64 * k < n ? cost[lane + 64 * k] : 0;
  // first-fit decreasing into m bins of capacity C by one wave (lane b holds bin b's load), the m
  // largest items opening one bin each (so they start together, as longest-first would start them:
  // their workgroups stream the same keys through the L2 at the same time; letting first fit pack
  // two of them into one bin made the plan 1 % shorter but tripled the sparse attention's L2
  // misses); returns whether every item fitted.  With rec, the i-th item's planned start << 6 | bin.
  auto ffd = [&](int C, bool rec) -> bool {
    // branch-free per item (a branch per step made the pass several times slower); lanes past
    // the bins hold a load no item fits on
    int load = lane < m ? 0 : 0x3FFFFFFF;
    bool ok = true;
#pragma unroll
    for (int k = 0; k < NMAX / 64; ++k) {
      const int jn = min(64, n - 64 * k);
      for (int j = 0; j < jn; ++j) {
        const int c = __builtin_amdgcn_readlane(creg[k], j);
        const int cand = load + c;
        const uint64_t fits = 64 * k + j < m ? 1ull << (64 * k + j) : __ballot(cand <= C);
        ok = ok && fits != 0;
        const int b = fits ? (int)__builtin_ctzll(fits) : 64;
        if (rec) plan[wv][64 * k + j] = ((uint32_t)__builtin_amdgcn_readlane(load, b & 63) << 6) | (uint32_t)b;
        load = lane == b ? cand : load;
      }
    }
    return ok;
  };
  // parallel search: every wave packs at one capacity of (lo, hi] and keeps its packing; the
  // interval shrinks 16-fold per round, down to a step of 1/256 of the capacity.  If no capacity up
  // to the first guess fits, the search goes on up to the bound where first fit always fits.
  while (!s_fail && (s_hi - s_lo > max(1, s_hi >> 8) || s_best < 0)) {
    const int lo = s_lo, hi = s_hi;
    const int C = lo + (int)(((int64_t)(hi - lo) * (wv + 1) + 15) / 16);
    const bool ok = ffd(C, true);
    if (lane == 0) s_ok[wv] = ok ? C : -C;
    __syncthreads();
    if (tid == 0) {
      int nlo = lo, nhi = hi, best = -1;
      for (int w = 0; w < 16; ++w) {
        if (s_ok[w] > 0) {
          if (s_ok[w] <= nhi) {
            nhi = s_ok[w];
            best = w;
          }
        } else {
          nlo = max(nlo, -s_ok[w]);
        }
      }
      if (best < 0) {   // nothing fitted up to hi (its packing failed too): search above it
        if (hi >= s_hi0) s_fail = 1;   // (cannot happen: first fit always fits at s_hi0)
        nlo = hi;
        nhi = s_hi0;
      }
      s_lo = nlo;
      s_hi = nhi;
      s_best = best;
    }
    __syncthreads();
  }
  if (s_fail) {
    if (tid == 0) out[0] = -1;
    return;
  }
  // the chosen packing, its items in order of planned start
  const uint32_t* chosen = plan[s_best];
  for (int i = tid; i < n; i += blockDim.x) key[i] = chosen[i];
  for (int i = n + tid; i < ((n + 3) & ~3); i += blockDim.x) key[i] = 0xFFFFFFFFu;
  __syncthreads();
  for (int i = tid; i < n; i += blockDim.x) out[1 + rank_of(key, n, i)] = item[i];
  if (tid == 0) out[0] = n;
}

// Log-sum-exp of the pieces of the split log-sum-exp pass, for one (probe row, query head) per
// thread: lse2 = m + log2(sum_i l_i 2^(m_i - m)) over the pieces that saw a key (l_i > 0), with m
// their largest running max, combined in piece order.  blockIdx.y = request.
__global__ __launch_bounds__(256) void lse_merge_kernel(const ReqDev* __restrict__ reqs,
                                                        const float2* __restrict__ part, int nsplit,
                                                        int64_t n_part_rows, int Hq, float* __restrict__ lse,
                                                        int lse_base2) {
  const ReqDev rq = reqs[blockIdx.y];
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t i = g / Hq;
  if (i >= rq.n_probe) return;
  const int h = (int)(g - i * Hq);
  const float2* pp = part + ((int64_t)rq.p_off + i) * Hq + h;
  const int64_t step = n_part_rows * Hq;
  float m = -INFINITY;
  for (int s = 0; s < nsplit; ++s) {
    const float2 v = pp[s * step];
    if (v.y > 0.f) m = fmaxf(m, v.x);
  }
  float l = 0.f;
  for (int s = 0; s < nsplit; ++s) {
    const float2 v = pp[s * step];
    if (v.y > 0.f) l += v.y * __builtin_amdgcn_exp2f(v.x - m);
  }
  const float lse2 = m + __log2f(l);
  lse[(int64_t)(rq.tok_off + i) * Hq + h] = lse_base2 ? lse2 : lse2 * 0.69314718055994531f;
}

constexpr int CS_WAVE_KEYS = 32;   // keys per key tile of a column-sum wave

// Gather of the Sparse-Q probe columns for colsum_kernel: the query rows of every probe row
// and the base-2 log-sum-exp of every (probe row, query head), in probe order and grouped by KV
// head ([Hkv][probe row][G] for both, so a chunk of one KV head's columns is contiguous), so that
// the column-sum kernel computes every address from its registers (no load chains).
// Thread: one 16-byte piece of one (probe row, head); blockIdx.y = request.
template <int D>
__global__ __launch_bounds__(256) void probe_gather_kernel(const uint16_t* __restrict__ q, const float* __restrict__ lse,
                                                           int lse_tok, const ReqDev* __restrict__ reqs,
                                                           const int32_t* __restrict__ probe, int Hq, int Hkv,
                                                           int64_t n_probe_total, uint16_t* __restrict__ qp,
                                                           float* __restrict__ lse2p) {
  constexpr int PPH = D * 2 / 16;   // 16-byte pieces per head row
  const ReqDev rq = reqs[blockIdx.y];
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t per_row = (int64_t)Hq * PPH;
  const int64_t i = g / per_row;
  if (i >= rq.n_probe) return;
  const int rem = (int)(g - i * per_row);
  const int h = rem / PPH;
  const int pc = rem - h * PPH;
  const int pos = probe[rq.tok_off + i];
  const int64_t prow = (int64_t)rq.p_off + i;
  const int G = Hq / Hkv;
  const int kvh = h / G;
  ((uint4*)qp)[(((int64_t)kvh * (n_probe_total + kProbePad) + prow) * G + (h - kvh * G)) * PPH + pc] =
      ((const uint4*)q)[((int64_t)(rq.tok_off + pos) * Hq + h) * PPH + pc];
  if (pc == 0) {
    const float l2 = lse_tok ? lse[(int64_t)(rq.tok_off + pos) * Hq + h] * 1.4426950408889634f
                             : lse[(int64_t)(rq.tok_off + i) * Hq + h];
    lse2p[((int64_t)kvh * (n_probe_total + kProbePad) + prow) * G + (h - kvh * G)] = l2;
  }
}

// Sparse-Q column sums from the gathered probe columns, key-stationary: a workgroup owns
// 8 x 32 x NKT keys of one KV head (a wave's NKT tiles of 32 keys held in registers as the MFMA B
// operand) and computes S = Q K^T, p = 2^(scale*log2e*s - lse2) masked causally, summed per key.
// In this orientation a lane's accumulator elements all belong to one key (its lane) and 16 probe
// columns, so a key's sum is a per-lane sum: one fp32 partial per key tile, flushed every chunk
// into an fp64 total.  Each query-operand read from LDS feeds NKT MFMAs.  The probe columns (probe
// row x query head of the group) stream in chunks of RC probe rows x G heads (at most 64 columns,
// two 32-column MFMA groups) that move global -> LDS directly: the query rows (16 bytes per lane,
// XOR-swizzled 16-byte chunks), the chunk's 64 log-sum-exps and 64 probe positions (one per column
// slot, 4 bytes per lane), triple-buffered and issued two chunks ahead.  No global load in the loop
// feeds an address, so the loop waits only for transfers issued two chunks earlier.
struct ColsumK {
  const uint16_t* k;
  const uint16_t* qp;
  const float* lse2p;
  const ReqDev* reqs;
  const int32_t* bt;
  const int32_t* probe;
  double* colsum;
  int64_t total, n_probe_total;
  int Hq, Hkv, G, RC, n_req;
  float scale_log2;
};

template <int D, int NKT>
__global__ __launch_bounds__(512, 1) void colsum_kernel(ColsumK a) {
  constexpr int NW = 8;
  constexpr int KEYS = NW * CS_WAVE_KEYS * NKT;   // keys per workgroup
  constexpr int ROWB = D * 2;                 // bytes of one query row (one column)
  constexpr int NCH = ROWB / 16;              // 16-byte chunks per column
  constexpr int CPP = 1024 / ROWB;            // columns per 1 KB transfer
  constexpr int NC = 64;                      // column slots per chunk
  constexpr int NPC = NC / CPP;               // 1 KB transfers per chunk
  constexpr int PPW = (NPC + NW - 1) / NW;    // per wave
  constexpr int QB = NC * ROWB;
  constexpr int CHB = QB + 512;               // + 64 log-sum-exps + 64 positions
  constexpr int NBUF = SX_CS_NBUF;            // chunk buffers; chunk k + NBUF - 1 is issued with chunk k
  static_assert(NBUF >= 3 && NBUF <= 5, "three to five chunk buffers");
  static_assert(NPC % NW == 0, "query transfers spread evenly over the waves");
  __shared__ __attribute__((aligned(1024))) char smem[NBUF * CHB];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int wu = __builtin_amdgcn_readfirstlane(w);
  const int l32 = lane & 31;
  const int hg = lane >> 5;
  const int kvh = (int)(blockIdx.x % (unsigned)a.Hkv);
  // request-major grid (per KV head: the key tiles of request 0 from the first keys, which the most
  // probe rows see, then request 1, ...), so the workgroups running together on one XCD mostly
  // stream the same request's probe columns
  int r, kt;
  locate_request((int)(blockIdx.x / (unsigned)a.Hkv), a.n_req,
                 [&](int rr) { return (a.reqs[rr].T + KEYS - 1) / KEYS; }, &r, &kt, lane);
  if (r < 0) return;
  r = __builtin_amdgcn_readfirstlane(r);
  kt = __builtin_amdgcn_readfirstlane(kt);
  const ReqDev rq = a.reqs[r];
  const int T = rq.T;
  const int j0 = kt * KEYS;
  const int jw = j0 + w * (CS_WAVE_KEYS * NKT);   // the wave's first key
  const int G = a.G;
  const int RC = a.RC;
  const int ncol = RC * G;                    // columns of a full chunk (<= 64)
  // B operand of key tile t: lane (l32, hg) holds dims 16 s + 8 hg .. + 7 of key jw + 32 t + l32
  bf16x8_t kb[NKT][D / 16];
#pragma unroll
  for (int t = 0; t < NKT; ++t) {
    const int key = jw + CS_WAVE_KEYS * t + l32;
    const uint16_t* kp = nullptr;
    if (key < T) {
      const int32_t blk = a.bt[rq.bt_off + (key >> 4)];
      kp = a.k + (((int64_t)blk * a.Hkv + kvh) * 16 + (key & 15)) * D + hg * 8;
    }
#pragma unroll
    for (int s = 0; s < D / 16; ++s) {
      uint4 v = kp ? *(const uint4*)(kp + 16 * s) : make_uint4(0, 0, 0, 0);
      kb[t][s] = __builtin_bit_cast(bf16x8_t, v);
    }
  }
  const int32_t* probe = a.probe + rq.tok_off;
  const int np = rq.n_probe;
  int lo = 0, hi = np;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (probe[mid] < j0) lo = mid + 1; else hi = mid;
  }
  const int nchunk = (np - lo + RC - 1) / RC;
  // ---- transfers of chunk k into buffer k mod NBUF (this wave's share).  Rows past the request's
  // probe rows read the padding (at most RC - 1 < kProbePad rows), so no clamping.  A chunk's query
  // rows are contiguous (column c of the chunk at c * D from its start); each 1 KB query piece is
  // a wave-uniform chunk base (scalar) plus a fixed per-lane offset. ----
  // query pieces: slot column qc = CPP * piece + lane / NCH, physical chunk lane % NCH holding
  // logical chunk (lane % NCH) ^ (qc mod NCH); slot columns past RC * G repeat column RC * G - 1
  uint32_t q_voff[PPW];
#pragma unroll
  for (int i = 0; i < PPW; ++i) {
    const int qc = CPP * (wu + NW * i) + lane / NCH;
    const int cc = min(qc, ncol - 1);
    const int lc = (lane % NCH) ^ (qc & (NCH - 1));
    q_voff[i] = (uint32_t)((cc * D + lc * 8) * 2);
  }
  const uint16_t* q_base = a.qp + ((int64_t)kvh * (a.n_probe_total + kProbePad) + rq.p_off + lo) * G * D;
  const int64_t q_step = (int64_t)RC * G * D;   // one chunk further
  // per-column metadata (column slot = lane): log-sum-exp (wave NW-1) and probe position (wave NW-2).
  // Slots past RC * G (G not dividing 64) read the log-sum-exp padding, +inf, so they add 0.
  const int m_col = min(lane, ncol - 1);
  const int m_row = m_col / G;
  const float* l_src =
      lane < ncol
          ? a.lse2p + ((int64_t)kvh * (a.n_probe_total + kProbePad) + rq.p_off + lo + m_row) * G + (m_col - m_row * G)
          : a.lse2p + ((int64_t)kvh * (a.n_probe_total + kProbePad) + a.n_probe_total) * G;
  const int l_step = lane < ncol ? RC * G : 0;
  const uint32_t p_voff = (uint32_t)(m_row * 4);
  const bool lse_wave = wu == NW - 1, pos_wave = wu == NW - 2;
  const int n_mine = PPW + (lse_wave ? 1 : 0) + (pos_wave ? 1 : 0);
  // wave-uniform 64-bit base in an SGPR pair (readfirstlane makes the uniformity visible; each half
  // goes through uint32_t so that nothing is sign-extended)
  auto sgpr_base = [](const void* ptr) -> uint64_t {
    const uint64_t sb = (uint64_t)(uintptr_t)ptr;
    const uint32_t lo32 = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)sb);
    const uint32_t hi32 = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(sb >> 32));
    return ((uint64_t)hi32 << 32) | (uint64_t)lo32;
  };
  // (dst: LDS byte address, wave-uniform)
  auto dma16_sb = [&](uint64_t sbase, uint32_t voffset, uint32_t dst) {
    const uint32_t m0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)dst);
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voffset), "s"(sbase), "s"(m0)
                 : "m0", "memory");
  };
  auto dma4_sb = [&](uint64_t sbase, uint32_t voffset, uint32_t dst) {
    const uint32_t m0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)dst);
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dword %0, %1" ::"v"(voffset), "s"(sbase), "s"(m0)
                 : "m0", "memory");
  };
  auto dma4 = [&](const void* src, uint32_t dst) {
    const uint32_t m0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)dst);
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off" ::"v"(src), "s"(m0) : "m0", "memory");
  };
  const uint32_t smem_lds = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)smem;
  auto issue = [&](int k) {
    if (k >= nchunk) return;
    const uint32_t b = smem_lds + (uint32_t)((k % NBUF) * CHB);
    const uint64_t qb = sgpr_base(q_base + k * q_step);
#pragma unroll
    for (int i = 0; i < PPW; ++i) dma16_sb(qb, q_voff[i], b + (uint32_t)((wu + NW * i) * 1024));
    if (lse_wave) dma4(l_src + k * l_step, b + QB);
    if (pos_wave) dma4_sb(sgpr_base(probe + lo + k * RC), p_voff, b + QB + 256);
  };
  auto wait_vm = [&](int n) {
    switch (n) {
      case 0: SX_WAIT_VMCNT(0); break;
      case 1: SX_WAIT_VMCNT(1); break;
      case 2: SX_WAIT_VMCNT(2); break;
      case 3: SX_WAIT_VMCNT(3); break;
      case 4: SX_WAIT_VMCNT(4); break;
      case 5: SX_WAIT_VMCNT(5); break;
      case 6: SX_WAIT_VMCNT(6); break;
      case 7: SX_WAIT_VMCNT(7); break;
      case 8: SX_WAIT_VMCNT(8); break;
      default: SX_WAIT_VMCNT(9); break;
    }
  };
  static_assert((NBUF - 2) * (PPW + 1) <= 9, "transfers in flight exceed the wait table");
  // this wave's transfers still allowed in flight once chunk k + 1 must have landed: those of
  // chunks k + 2 .. k + NBUF - 1
  auto inflight = [&](int k) {
    int n = 0;
#pragma unroll
    for (int c = 2; c < NBUF; ++c) n += k + c < nchunk ? n_mine : 0;
    return n;
  };
  // Chunks whose first probe row lies before the workgroup's last key may miss keys (causal mask),
  // and the last chunk may hold fewer than RC probe rows; both take the checked path.  Probe rows
  // ascend, so the masked chunks come first: nmask of them.
  int hm = lo, hx = np;
  while (hm < hx) {
    const int mid = (hm + hx) >> 1;
    if (probe[mid] < j0 + KEYS - 1) hm = mid + 1; else hx = mid;
  }
  const int nmask = min(nchunk, (hm - lo + RC - 1) / RC);
  const bool last_partial = (np - lo) % RC != 0;
  const int nfast = last_partial ? nchunk - 1 : nchunk;   // chunks [nmask, nfast) take the fast path

  double acc64[NKT];
  float acc32[NKT];
#pragma unroll
  for (int t = 0; t < NKT; ++t) {
    acc64[t] = 0.0;
    acc32[t] = 0.f;
  }
  // K must be in registers before the first transfer wait (the compiler does not count the
  // transfers, so a later wait of its own for K would also wait for them)
  SX_WAIT_VMCNT(0);
#pragma unroll
  for (int c = 0; c < NBUF - 1; ++c) issue(c);
  wait_vm(inflight(-1));   // chunk 0 has landed
  __syncthreads();
  const float c2 = a.scale_log2;
  // operand reads add a loop-invariant lane offset to a wave-uniform buffer address (one vector
  // add per k-step; the column group is an immediate)
  uint32_t q_off[D / 16];
#pragma unroll
  for (int st = 0; st < D / 16; ++st) {
    const int ci = 2 * st + hg;
    q_off[st] = (uint32_t)(l32 * ROWB + ((ci ^ (l32 & (NCH - 1))) << 4));
  }
  auto lds16 = [](uint32_t addr) -> bf16x8_t {
    return *(const __attribute__((address_space(3))) bf16x8_t*)(uintptr_t)addr;
  };
  // S of the chunk in the buffer at Cb against the NKT key tiles, column group gi in s[gi]: lane
  // (l32, hg), element e holds column 32 gi + 8 (e / 4) + 4 hg + e % 4 of the chunk and key
  // jw + 32 t + l32
  struct SG {
    f32x16_t s[NKT];
  };
  SG sg[2];
  auto matrix_phase = [&](int j) {
    if (j >= nchunk) return;
    uint32_t Cb = (uint32_t)__builtin_amdgcn_readfirstlane((int)(smem_lds + (uint32_t)((j % NBUF) * CHB)));
    asm volatile("" : "+s"(Cb));
    __builtin_amdgcn_s_setprio(2);
#pragma unroll
    for (int gi = 0; gi < 2; ++gi)
#pragma unroll
      for (int t = 0; t < NKT; ++t) sg[gi].s[t] = f32x16_t{};
#pragma unroll
    for (int st = 0; st < D / 16; ++st) {
      uint32_t qa_addr = Cb + q_off[st];
      asm volatile("" : "+v"(qa_addr));
#pragma unroll
      for (int gi = 0; gi < 2; ++gi) {
        const bf16x8_t qa = lds16(qa_addr + (uint32_t)(gi * 32 * ROWB));
#pragma unroll
        for (int t = 0; t < NKT; ++t)
          sg[gi].s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa, kb[t][st], sg[gi].s[t], 0, 0, 0);
      }
    }
    sched_pipelined<2 * NKT * (D / 16), 1, 4>();
    __builtin_amdgcn_s_setprio(0);
  };
  // sums of chunk j.  Fast path: every column valid, no mask.  Checked path: column c counts for
  // key j when c < nvalid and j <= its probe position.
  auto vector_phase = [&](int j, auto checked) {
    uint32_t Mb = (uint32_t)__builtin_amdgcn_readfirstlane((int)(smem_lds + (uint32_t)((j % NBUF) * CHB + QB)));
    asm volatile("" : "+s"(Mb));
    const uint32_t lb = Mb + (uint32_t)(16 * hg);
#pragma unroll
    for (int gi = 0; gi < 2; ++gi) {
      float l2[16];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        typedef float f32x4_t __attribute__((ext_vector_type(4)));
        const f32x4_t v = *(const __attribute__((address_space(3))) f32x4_t*)(uintptr_t)(lb + 4 * (32 * gi + 8 * q));
        l2[4 * q + 0] = v.x;
        l2[4 * q + 1] = v.y;
        l2[4 * q + 2] = v.z;
        l2[4 * q + 3] = v.w;
      }
      if constexpr (decltype(checked)::value) {
        const int nvalid = min(RC, np - (lo + j * RC)) * G;
        int pos[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          typedef int i32x4_t __attribute__((ext_vector_type(4)));
          const i32x4_t v = *(const __attribute__((address_space(3))) i32x4_t*)(uintptr_t)(lb + 256 + 4 * (32 * gi + 8 * q));
          const int c0 = 32 * gi + 8 * q + 4 * hg;
          pos[4 * q + 0] = c0 + 0 < nvalid ? v.x : -1;
          pos[4 * q + 1] = c0 + 1 < nvalid ? v.y : -1;
          pos[4 * q + 2] = c0 + 2 < nvalid ? v.z : -1;
          pos[4 * q + 3] = c0 + 3 < nvalid ? v.w : -1;
        }
#pragma unroll
        for (int t = 0; t < NKT; ++t) {
          const int key = jw + CS_WAVE_KEYS * t + l32;
          float sum = acc32[t];
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sg[gi].s[t][e], c2, -l2[e]));
            sum += key <= pos[e] ? p : 0.f;
          }
          acc32[t] = sum;
        }
      } else {
#pragma unroll
        for (int t = 0; t < NKT; ++t) {
          float sum = acc32[t];
#pragma unroll
          for (int e = 0; e < 16; ++e) sum += __builtin_amdgcn_exp2f(__builtin_fmaf(sg[gi].s[t][e], c2, -l2[e]));
          acc32[t] = sum;
        }
      }
    }
#pragma unroll
    for (int t = 0; t < NKT; ++t) {
      acc64[t] += (double)acc32[t];
      acc32[t] = 0.f;
    }
  };
  auto vphase = [&](int j) {
    if (j < 0 || j >= nchunk) return;
    if (j < nmask || j >= nfast) vector_phase(j, std::true_type{});
    else vector_phase(j, std::false_type{});
  };
  // ---- ping-pong: iteration j = 0 .. nchunk has two slots separated by workgroup barriers.  Group
  // X (waves 0-3) runs the matrix phase of chunk j in slot 1 and its sums in slot 2; group Y (waves
  // 4-7) the sums of chunk j-1 in slot 1 and the matrix phase of chunk j in slot 2, so in every slot
  // one wave of each SIMD issues MFMAs while the other exponentiates.  Chunk j + NBUF - 1 is issued
  // in slot 2 into the buffer of chunk j - 1, whose last reader (Y's sums) ran in slot 1; each wave
  // waits for its own transfers of chunk j + 1 before the barrier that closes iteration j. ----
  const int grp = wu >> 2;
  if (grp == 0) {
    for (int j = 0; j <= nchunk; ++j) {
      matrix_phase(j);
      __syncthreads();
      issue(j + NBUF - 1);
      vphase(j);
      wait_vm(inflight(j));
      __syncthreads();
    }
  } else {
    for (int j = 0; j <= nchunk; ++j) {
      vphase(j - 1);
      __syncthreads();
      issue(j + NBUF - 1);
      matrix_phase(j);
      wait_vm(inflight(j));
      __syncthreads();
    }
  }
  // the two lane halves hold the same keys (different columns)
#pragma unroll
  for (int t = 0; t < NKT; ++t) {
    const double tot = acc64[t] + __shfl_xor(acc64[t], 32, 64);
    const int key = jw + CS_WAVE_KEYS * t + l32;
    if (hg == 0 && key < T) a.colsum[(int64_t)kvh * a.total + rq.tok_off + key] = tot;
  }
}

template <int D, bool PAGED, bool PV>
hipError_t launch_mfma(const AttnLaunch& L, hipStream_t s) {
  // persistent grid: sparse attention always (the plan's counters), full attention when the host
  // gave it a queue slot
  constexpr bool kCanPersist = PV;
  const bool persist = kCanPersist && (PAGED || L.qslot >= 0);
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
  a.grid_rows = L.grid_rows;
  const int64_t ntiles = (L.grid_rows + a.rpw - 1) / a.rpw;
  // the log-sum-exp pass of the Sparse-Q probe rows has few row tiles: split each row tile's keys
  // into up to kLseSplit pieces until the grid has about 1024 workgroups
  int ns = 1;
  if (PAGED && !PV && L.lse_part) {
    while (ns < kLseSplit && ntiles * L.Hkv * L.n_req * ns < 1024) ns *= 2;
  }
  a.nsplit = ns;
  a.lse_part = L.lse_part;
  a.n_part_rows = L.n_part_rows;
  a.queue = L.queue;
  a.qslot = L.qslot;
  a.order = L.order;
  int64_t per_head = ntiles * ns * L.n_req;   // items of one KV head (an upper bound: empty ones end at once)
  if (persist) {
    // about one workgroup per compute unit and KV head, never more than the items
    if (PAGED ? !L.queue : (L.qslot >= kDenseQueueSlots || L.Hkv >= kDenseQueueStride)) return hipErrorInvalidValue;
    per_head = std::min<int64_t>(per_head, std::max(1, L.n_cu / L.Hkv));
  }
  const dim3 grid((unsigned)(per_head * L.Hkv));
  if (persist)
    hipLaunchKernelGGL((attn_mfma_kernel<D, PAGED, PV, kCanPersist>), grid, dim3(512), 0, s, a);
  else
    hipLaunchKernelGGL((attn_mfma_kernel<D, PAGED, PV, false>), grid, dim3(512), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || ns == 1) return e;
  const dim3 mg((unsigned)((L.grid_rows * (int64_t)L.Hq + 255) / 256), (unsigned)L.n_req);
  hipLaunchKernelGGL(lse_merge_kernel, mg, dim3(256), 0, s, L.reqs, L.lse_part, ns, L.n_part_rows, L.Hq, L.lse,
                     L.lse_base2);
  return hipGetLastError();
}

}  // namespace

// float32 variants (vector ALU), defined in k_attn_f32.hip
hipError_t launch_attn_f32(const AttnLaunch& a, bool paged, hipStream_t s);
hipError_t launch_colsum_f32(const sx_plan* p, double* colsum, const void* q, const void* kc, const float* lse,
                             int lse_tok, hipStream_t s);

hipError_t launch_attn_paged(const AttnLaunch& a, hipStream_t s) {
  if (a.dtype == SX_F32) return launch_attn_f32(a, true, s);
  const bool pv = a.out != nullptr;
  if (pv && a.lse != nullptr) return hipErrorInvalidValue;
  if (a.D == 128) return pv ? launch_mfma<128, true, true>(a, s) : launch_mfma<128, true, false>(a, s);
  return pv ? launch_mfma<64, true, true>(a, s) : launch_mfma<64, true, false>(a, s);
}

hipError_t launch_tile_order(const sx_plan* p, const int32_t* rows, const int32_t* n_rows, int32_t max_rows,
                             hipStream_t s) {
  const int G = p->desc.n_q_heads / p->desc.n_kv_heads;
  const int rpw = COLS / G;
  const int64_t items = (int64_t)(max_rows + rpw - 1) / rpw * p->n_req;   // as the attention launch bounds them
  const int m = (int)std::min<int64_t>(items, std::max(1, p->n_cu / p->desc.n_kv_heads));
  hipLaunchKernelGGL(tile_order_kernel, dim3(1), dim3(1024), 0, s, p->d_req, rows, n_rows, max_rows, p->n_req, rpw,
                     std::max(m, 1), p->d_order);
  return hipGetLastError();
}

hipError_t launch_attn_dense(const AttnLaunch& a, hipStream_t s) {
  if (a.dtype == SX_F32) return launch_attn_f32(a, false, s);
  if (a.D == 128) return launch_mfma<128, false, true>(a, s);
  return launch_mfma<64, false, true>(a, s);
}

hipError_t launch_colsum(const sx_plan* p, const ScoreScratch& sc, const void* q, const void* kc, const float* lse,
                         int lse_tok, hipStream_t s) {
  if (p->desc.dtype == SX_F32) return launch_colsum_f32(p, sc.colsum, q, kc, lse, lse_tok, s);
  const int G = p->desc.n_q_heads / p->desc.n_kv_heads;   // <= 64 (checked on the host)
  // gather the probe columns, then the column sums from them
  const int D = p->desc.head_dim;
  const int64_t threads = (int64_t)p->max_probe * p->desc.n_q_heads * (D * 2 / 16);
  if (threads > 0) {
    const dim3 gg((unsigned)((threads + 255) / 256), (unsigned)p->n_req);
    if (D == 128)
      hipLaunchKernelGGL(probe_gather_kernel<128>, gg, dim3(256), 0, s, (const uint16_t*)q, lse, lse_tok, p->d_req,
                         p->d_probe, p->desc.n_q_heads, p->desc.n_kv_heads, p->n_probe, (uint16_t*)sc.qp,
                         sc.lse2p);
    else
      hipLaunchKernelGGL(probe_gather_kernel<64>, gg, dim3(256), 0, s, (const uint16_t*)q, lse, lse_tok, p->d_req,
                         p->d_probe, p->desc.n_q_heads, p->desc.n_kv_heads, p->n_probe, (uint16_t*)sc.qp,
                         sc.lse2p);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  ColsumK c{};
  c.k = (const uint16_t*)kc;
  c.qp = (const uint16_t*)sc.qp;
  c.lse2p = sc.lse2p;
  c.reqs = p->d_req;
  c.bt = p->d_bt;
  c.probe = p->d_probe;
  c.colsum = sc.colsum;
  c.total = p->total;
  c.n_probe_total = p->n_probe;
  c.Hq = p->desc.n_q_heads;
  c.Hkv = p->desc.n_kv_heads;
  c.G = G;
  c.RC = 64 / G;
  c.n_req = p->n_req;
  c.scale_log2 = p->scale * 1.4426950408889634f;
  // two key tiles per wave (each staged query column feeds twice the MFMAs and the probe columns
  // stream half as often) while that still leaves two workgroups per CU, else one
  const int64_t wg2 = ((p->max_T + 511) / 512) * c.Hkv * p->n_req;
  if (wg2 >= 512) {
    const dim3 grid((unsigned)wg2);
    if (D == 128) hipLaunchKernelGGL((colsum_kernel<128, 2>), grid, dim3(512), 0, s, c);
    else hipLaunchKernelGGL((colsum_kernel<64, 2>), grid, dim3(512), 0, s, c);
  } else {
    const dim3 grid((unsigned)(((p->max_T + 255) / 256) * c.Hkv * p->n_req));
    if (D == 128) hipLaunchKernelGGL((colsum_kernel<128, 1>), grid, dim3(512), 0, s, c);
    else hipLaunchKernelGGL((colsum_kernel<64, 1>), grid, dim3(512), 0, s, c);
  }
  return hipGetLastError();
}

}  // namespace sx
