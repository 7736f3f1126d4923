// Device helpers shared by the libsx kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace sx {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// bfloat16 stored as the upper half of a float32: widening is exact.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Two float32 -> packed bfloat16, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  bf16x2_t v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Value of v in lane src of the wave (src taken mod 64).
__device__ __forceinline__ int lane_value(int v, int src) { return __builtin_amdgcn_ds_bpermute(src << 2, v); }

// Request-major position of a workgroup: position idx of the concatenation of every request's
// items (cnt(r) items of request r, requests in order) -> request *r and item *q inside it; *r = -1
// past the last item.  Every wave computes the same answer (no LDS, no barrier); cnt is called for
// requests in runs of 64, one per lane.  lane: the caller's lane index (threadIdx.x & 63; a kernel
// that loops over items passes a copy the compiler cannot hoist, so the shuffle indices built from
// it are not kept live across the loop).
template <typename CountF>
__device__ __forceinline__ void locate_request(int idx, int n_req, CountF cnt, int* r, int* q, int lane) {
  int base = 0;
  for (int c0 = 0; c0 < n_req; c0 += 64) {
    const int rr = c0 + lane;
    const int c = rr < n_req ? cnt(rr) : 0;
    int x = c;   // inclusive prefix over the lanes
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = lane_value(x, lane - o);
      if (lane >= o) x += y;
    }
    const int tot = __builtin_amdgcn_readlane(x, 63);
    if (idx < base + tot) {
      const uint64_t m = __ballot(base + x > idx);
      const int l = __ffsll((unsigned long long)m) - 1;
      *r = c0 + l;
      *q = idx - (base + __builtin_amdgcn_readlane(x, l) - __builtin_amdgcn_readlane(c, l));
      return;
    }
    base += tot;
  }
  *r = -1;
  *q = 0;
}

// Largest and smallest v over the wave (lane as for locate_request).
__device__ __forceinline__ int wave_max_i(int v, int lane) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = max(v, lane_value(v, lane ^ o));
  return v;
}

__device__ __forceinline__ int wave_min_i(int v, int lane) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = min(v, lane_value(v, lane ^ o));
  return v;
}

// Pool offset (elements) of (slot, head) in a [blocks][Hkv][16][D] pool.
__device__ __forceinline__ int64_t pool_off(int32_t slot, int head, int Hkv, int D) {
  return ((((int64_t)(slot >> 4)) * Hkv + head) * 16 + (slot & 15)) * (int64_t)D;
}

}  // namespace sx
