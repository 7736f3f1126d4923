// Internal declarations shared by the host library and the HIP kernels of libsx.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "sx.h"

namespace sx {

constexpr int kBlock = 16;     // paged-cache block size supported by the kernels
constexpr int kTail = 64;      // tail-fallback rows (Section 3.2)
constexpr int kProbePad = 64;  // padding rows past the probe lists and gathered probe columns

// Per-request device metadata.
struct ReqDev {
  int32_t T;        // tokens of the request
  int32_t tok_off;  // first token in the concatenation of all requests
  int32_t bt_off;   // first entry of its block table in the concatenated tables
  int32_t n_reuse;  // top-k candidates: |I_reuse|, or T with SX_TOPK_ALL_POSITIONS
  int32_t n_probe;  // |I_nr U S_tail|: Sparse-Q rows
  int32_t n_nr;     // |I_nr|
  int32_t n_base;   // |I_nr U S_ov U S_tail|
  int32_t p_off;    // first probe row of the request in the concatenation of all probe rows
};

// One reused token of the re-alignment pass.  Slots are pool-wide: block * kBlock + slot.
struct RealignRow {
  int32_t src_slot;
  int32_t dst_slot;
  int32_t cs_row;   // row of the cos/sin table (one row per cached segment)
  int32_t pad;
};

// Selection scratch (plan-owned; the histograms are zeroed when the plan is made and cleared again
// by every call's last pass): per request the fine and coarse histograms of the first digit
// [kTopkFine + 256] and the selection state (first digit, candidates still needed) [4]; per chunk
// of kTopkChunk tokens the rows surely in R and the number of boundary entries [2]; per token a
// boundary-list slot (index with a base-row flag, key), a chunk's list filling the slots of its own
// tokens.
constexpr int kTopkChunk = 2048;
constexpr int kTopkFine = 65536;       // first digit: the top 16 bits of a 32-bit key
constexpr int kTopkMaxChunks = 1024;   // chunks per request: requests up to 2097152 tokens
struct TopkScratch {
  uint32_t* hist;    // [n_req][kTopkFine + 256]
  uint32_t* state;   // [n_req][4]
  int32_t* cnt;      // [n_req][max_chunks][2]
  uint2* list;       // [sum T]
  int32_t max_chunks;
};

// Token flags used by the selection kernel.
enum : uint8_t { kFlagCandidate = 1, kFlagBase = 2 };

struct HostReq {
  int32_t T, tok_off, bt_off, n_reuse, n_probe, n_nr, n_base;
};

}  // namespace sx

struct sx_plan {
  sx_layer_desc desc;
  float scale;                    // softmax scale actually used
  int32_t n_req = 0;
  int64_t total = 0;              // sum T
  int32_t max_T = 0;
  int64_t n_dst_blocks = 0, n_src_blocks = 0;
  int32_t device = 0;
  std::vector<sx::HostReq> reqs;
  int64_t n_reuse = 0, n_nr = 0, n_probe = 0, n_base = 0;
  int32_t max_nr = 0, max_probe = 0;
  int64_t n_realign = 0;
  int64_t device_bytes = 0;
  // device memory owned by the plan
  sx::ReqDev* d_req = nullptr;
  int32_t* d_bt = nullptr;
  sx::RealignRow* d_ra = nullptr;
  float2* d_cs = nullptr;         // [cached segments][d/2] (cos, sin)
  int32_t* d_probe = nullptr;     // row-list layout
  int32_t* d_nr = nullptr;        // row-list layout
  int32_t* d_n_nr = nullptr;      // [n_req]
  int32_t* d_n_probe = nullptr;   // [n_req]
  uint8_t* d_flags = nullptr;     // [sum T]
  // [sum T] every token's slots in one record: dst_slot (block * b + slot), and for a reused token
  // its source slot and cos/sin row (src_slot = -1 for an uncached token)
  sx::RealignRow* d_tok_row = nullptr;
  uint32_t* d_rmark = nullptr;    // [sum T] row-set generation marks (sx_realign_scatter)
  mutable uint32_t rgen = 0;      // last generation used
  float* d_lse = nullptr;         // scratch [sum T][Hq]
  double* d_colsum = nullptr;     // scratch [Hkv][sum T]
  int32_t* d_tok_pos = nullptr;   // [sum T] RoPE position of every token in the new sequence
  double* d_theta = nullptr;      // [d/2] RoPE frequencies base^(-2i/d), float64
  void* d_qp = nullptr;           // scratch [Hkv][n_probe][Hq / Hkv][d]: query rows of the probe rows (bf16 plans)
  float* d_lse2p = nullptr;       // scratch [Hkv][n_probe][Hq / Hkv]: their base-2 log-sum-exp
  float2* d_lsep = nullptr;       // scratch [kLseSplit][n_probe][Hq]: partials of the split pass (bf16 plans)
  uint32_t* d_topk = nullptr;     // selection scratch, carved into `topk`
  sx::TopkScratch topk{};
  int32_t* d_queue = nullptr;     // [Hkv + 1] work-queue counters of sparse attention, zero between calls
  int32_t n_cu = 0;               // compute units of the plan's device
  // [1 + kOrderMax] planned row-tile order of sparse attention, written by sx_rows_mask for the row
  // list it was given (bf16 plans); sx_sparse_attn uses it for the same rows / n_rows / max_rows
  int32_t* d_order = nullptr;
  mutable const int32_t* order_rows = nullptr;
  mutable const int32_t* order_n_rows = nullptr;
  mutable int32_t order_max_rows = -1;
};

namespace sx {

// Kernel launchers (defined in the .hip files).  Each returns the launch status.
hipError_t launch_realign(const sx_plan* p, const void* src_k, const void* src_v, void* kc, void* vc,
                          hipStream_t s);
hipError_t launch_scatter(const sx_plan* p, const void* k_new, const void* v_new, const int32_t* rows,
                          const int32_t* n_rows, int32_t max_rows, void* kc, void* vc, hipStream_t s);
// Scratch of the Sparse-Q column sums: per-KV-head float64 sums [Hkv][sum T]; (bf16 plans) the
// gathered probe columns, queries [Hkv][n_probe + kProbePad][Hq / Hkv][d] and base-2 log-sum-exps
// [Hkv][n_probe + kProbePad][Hq / Hkv], whose kProbePad padding rows must hold zero queries and
// +inf log-sum-exps (a column read there adds exp2(-inf) = 0).
constexpr uint32_t kProbePadLse = 0x7f800000u;   // +inf
struct ScoreScratch {
  double* colsum;
  void* qp;
  float* lse2p;
};
hipError_t launch_head_reduce(const sx_plan* p, const double* colsum, float* scores, hipStream_t s);
// sets the padding rows of the gathered probe columns in `sc` (zero queries, +inf log-sum-exps)
hipError_t launch_probe_pad_clear(const sx_plan* p, const ScoreScratch& sc, hipStream_t s);
// fused re-alignment + KV write of n_layers layers (host array of per-layer pointers): marks the
// rows with `gen` (after clearing every mark when clear_marks), then writes every token's slot of
// every layer once
// (sel != null: membership in R from the caller's byte mask instead; rows, gen and clear_marks unused)
hipError_t launch_realign_scatter(const sx_plan* p, int32_t n_layers, const sx_layer_kv* layers, const int32_t* rows,
                                  const int32_t* n_rows, int32_t max_rows, uint32_t gen, bool clear_marks,
                                  const uint8_t* sel, hipStream_t s);
// mask[off_r + t] = 1 for every listed row t, 0 for every other token of the plan
hipError_t launch_rows_mask(const sx_plan* p, const int32_t* rows, const int32_t* n_rows, int32_t max_rows,
                            uint8_t* mask, hipStream_t s);
hipError_t launch_topk(const sx_plan* p, const float* scores, double ratio, int32_t* rows, int32_t* n_rows,
                       hipStream_t s);

// Row-sparse layer body (defined in k_layer.hip).  Rows are the listed rows of every request in
// the row-list layout; an operand row is addressed by slot (off_r + n) or by token
// (off_r + rows[off_r + n]).
// Device-side validation (checked library): launches the checks on `s`, synchronises it and fills
// verdict = {code (0 = valid), request, index, value}.  Row lists: rows may be NULL (counts only).
hipError_t device_check_rows(const sx_plan* p, const int32_t* rows, const int32_t* n_rows, int32_t max_rows,
                             hipStream_t s, int verdict[4]);
hipError_t device_check_cu(const int32_t* cu, int32_t n_req, int32_t max_seqlen, hipStream_t s, int verdict[4]);

// Sets the thread-local error message read by sx_last_error and returns st (for host-only
// translation units without the dispatcher's helpers).
sx_status report(sx_status st, const char* msg);

struct RowsArg {
  const int32_t* rows;
  const int32_t* n_rows;
  int32_t max_rows;
};
// y = x w^T on the listed rows; w is [sum part_n][k], output part i (columns of w's rows
// sum_{j<i} part_n[j] ..) goes to ys[i] with row stride part_n[i]; 1 <= n_parts <= 4, residual
// (nullable) addressed like part 0
hipError_t launch_gemm_rows(const sx_plan* p, const RowsArg& r, const void* x, int x_tok, const void* w, int k,
                            int n_parts, const int* part_n, void* const* ys, const void* res, int y_tok, hipStream_t s);
hipError_t launch_rmsnorm_rows(const sx_plan* p, const RowsArg& r, const void* x, int x_tok, const void* gamma,
                               float eps, int h, void* y, int y_tok, hipStream_t s);
hipError_t launch_rope_rows(const sx_plan* p, const RowsArg& r, void* q, void* k, hipStream_t s);
hipError_t launch_silu_mul_rows(const sx_plan* p, const RowsArg& r, const void* gu, int f, void* y, hipStream_t s);

// Attention family.  Mode selects the query rows and the key source.
struct AttnLaunch {
  int Hq, Hkv, D, n_req, grid_rows;   // grid_rows: max query rows of any request
  int dtype;
  float scale;
  const void* q;
  const void* k;
  const void* v;
  void* out;          // null in LSE-only mode
  float* lse;         // optional
  int lse_base2;      // 1: base-2 LSE of scale*q.k (score pass); 0: natural log
  // paged mode
  const ReqDev* reqs;
  const int32_t* bt;
  const int32_t* rows;
  const int32_t* n_rows;
  // dense mode
  const int32_t* cu;
  // paged log-sum-exp pass: scratch for the (max, sum) partials of a split pass,
  // [kLseSplit][n_part_rows][Hq] (n_part_rows = probe rows of all requests); NULL: no split
  float2* lse_part;
  int64_t n_part_rows;
  // persistent attention grids (about one workgroup per compute unit and KV head): sparse
  // attention's work-queue counters (the plan's), full attention's queue slot (-1: one workgroup per
  // item, as under graph capture), and the device's compute units
  int32_t* queue;
  int qslot;
  int n_cu;
  const int32_t* order;   // sparse attention: the plan's planned tile order, or NULL
};
constexpr int kOrderMax = 512;   // most row tiles the tile order is planned for (8 per workgroup, 64 workgroups)
// planned order of sparse attention's row tiles for the row list (plan->d_order)
hipError_t launch_tile_order(const sx_plan* p, const int32_t* rows, const int32_t* n_rows, int32_t max_rows,
                             hipStream_t s);
// queue slots of persistent full attention on one device, and counters per slot (KV heads + 1)
constexpr int kDenseQueueSlots = 64;
constexpr int kDenseQueueStride = 256;
constexpr int kLseSplit = 4;   // most key pieces per row tile of the log-sum-exp pass
hipError_t launch_attn_paged(const AttnLaunch& a, hipStream_t s);   // rows over a paged cache
hipError_t launch_attn_dense(const AttnLaunch& a, hipStream_t s);   // all rows, dense K/V
// column sums of the Sparse-Q probabilities; lse: base-2 sums indexed by probe (lse_tok = 0, the
// plan's pass-1 scratch) or natural-log sums indexed by token (lse_tok = 1, a caller's input)
hipError_t launch_colsum(const sx_plan* p, const ScoreScratch& sc, const void* q, const void* kc, const float* lse,
                         int lse_tok, hipStream_t s);

}  // namespace sx
