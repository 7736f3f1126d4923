// Device-side validation of the index arrays a caller hands over in device memory, compiled into
// the checked library only (SX_DEVICE_CHECKS; the release library has none of it).  The host
// validates everything it can see in sx_plan_create (segment tables, block tables, source block
// ids); what lives on the device -- the row lists of R that sx_topk_select or the caller wrote, and
// the cu_seqlens of sx_full_attn -- is checked here before any compute kernel reads it, so a bad
// list becomes SX_EDEVICE instead of out-of-range reads and writes.  The entry point synchronises
// its stream to read the verdict, which a debug build accepts.
//
// Row lists (row-list layout of include/sx.h), per request r with n = n_rows[r]:
//   0 <= n <= T_r; the first min(n, max_rows) rows are in [0, T_r) and strictly ascending.
// cu_seqlens: cu[0] = 0 and 0 <= cu[r + 1] - cu[r] <= max_seqlen.
// The checks read only in-bounds entries: at most T_r rows of a request's own region.
#include "sx_internal.h"

namespace sx {
namespace {

// verdict of the last check: code (0 = valid), request, index, value
__device__ int g_check[4];

enum { kBadCount = 1, kRowRange = 2, kRowOrder = 3, kCuStart = 4, kCuLength = 5 };

__device__ void report_bad(int code, int r, int i, int v) {
  if (atomicCAS(&g_check[0], 0, code) == 0) {
    g_check[1] = r;
    g_check[2] = i;
    g_check[3] = v;
  }
}

__global__ void check_clear_kernel() {
  if (threadIdx.x < 4) g_check[threadIdx.x] = 0;
}

__global__ __launch_bounds__(256) void check_rows_kernel(const ReqDev* __restrict__ reqs,
                                                         const int32_t* __restrict__ rows,
                                                         const int32_t* __restrict__ n_rows, int max_rows) {
  const ReqDev rq = reqs[blockIdx.y];
  const int n = n_rows[blockIdx.y];
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0 && (n < 0 || n > rq.T)) report_bad(kBadCount, blockIdx.y, -1, n);
  if (!rows) return;
  const int lim = min(min(max(n, 0), max_rows), rq.T);
  if (i >= lim) return;
  const int v = rows[rq.tok_off + i];
  if (v < 0 || v >= rq.T) report_bad(kRowRange, blockIdx.y, i, v);
  else if (i > 0 && rows[rq.tok_off + i - 1] >= v) report_bad(kRowOrder, blockIdx.y, i, v);
}

__global__ __launch_bounds__(256) void check_cu_kernel(const int32_t* __restrict__ cu, int n_req, int max_seqlen) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r == 0 && cu[0] != 0) report_bad(kCuStart, 0, 0, cu[0]);
  if (r >= n_req) return;
  const int len = cu[r + 1] - cu[r];
  if (len < 0 || len > max_seqlen) report_bad(kCuLength, r, r, len);
}

// Launch status, then the verdict (synchronises the stream).  *code = 0 when valid.
hipError_t read_verdict(hipStream_t s, int out[4]) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = hipMemcpyFromSymbolAsync(out, HIP_SYMBOL(g_check), 4 * sizeof(int), 0, hipMemcpyDeviceToHost, s);
  if (e != hipSuccess) return e;
  return hipStreamSynchronize(s);
}

}  // namespace

hipError_t device_check_rows(const sx_plan* p, const int32_t* rows, const int32_t* n_rows, int32_t max_rows,
                             hipStream_t s, int verdict[4]) {
  hipLaunchKernelGGL(check_clear_kernel, dim3(1), dim3(64), 0, s);
  const int lim = max_rows < p->max_T ? max_rows : p->max_T;
  const dim3 grid((unsigned)((lim > 0 ? lim : 1) + 255) / 256, (unsigned)p->n_req);
  hipLaunchKernelGGL(check_rows_kernel, grid, dim3(256), 0, s, p->d_req, rows, n_rows, max_rows);
  return read_verdict(s, verdict);
}

hipError_t device_check_cu(const int32_t* cu, int32_t n_req, int32_t max_seqlen, hipStream_t s, int verdict[4]) {
  hipLaunchKernelGGL(check_clear_kernel, dim3(1), dim3(64), 0, s);
  hipLaunchKernelGGL(check_cu_kernel, dim3((unsigned)((n_req + 255) / 256)), dim3(256), 0, s, cu, n_req, max_seqlen);
  return read_verdict(s, verdict);
}

}  // namespace sx
