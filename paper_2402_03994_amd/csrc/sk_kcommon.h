// sk_kcommon.h -- device helpers shared by the Walsh-Hadamard kernels.
#pragma once

#include "sk_internal.h"

namespace sk {

__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

__device__ __forceinline__ void store_out(void *out, int out_dtype, int64_t i, float v) {
  if (out_dtype == SK_BF16)
    ((uint16_t *)out)[i] = f32_to_bf16(v);
  else
    ((float *)out)[i] = v;
}

// Load up to 4 consecutive input elements starting at element e of a vector
// whose valid prefix has `lim` (>= 1) elements from e on; missing -> 0.
template <bool BF16, bool VEC>
__device__ __forceinline__ void load4(const void *x, int64_t e, int64_t lim, float v[4]) {
  if (VEC && lim >= 4) {
    if (BF16) {
      const uint2 u = *(const uint2 *)((const uint16_t *)x + e);
      v[0] = __uint_as_float(u.x << 16);
      v[1] = __uint_as_float(u.x & 0xFFFF0000u);
      v[2] = __uint_as_float(u.y << 16);
      v[3] = __uint_as_float(u.y & 0xFFFF0000u);
    } else {
      const float4 f = *(const float4 *)((const float *)x + e);
      v[0] = f.x;
      v[1] = f.y;
      v[2] = f.z;
      v[3] = f.w;
    }
    return;
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    if (q < lim)
      v[q] = BF16 ? bf16_to_f32(((const uint16_t *)x)[e + q]) : ((const float *)x)[e + q];
    else
      v[q] = 0.0f;
  }
}

// In-place unnormalised radix-2 Walsh-Hadamard transform along the rows of an
// LDS tile s[r << lgcs | c], 2^lgrows rows, 2^lgcs columns.  Ends synchronised.
__device__ __forceinline__ void lds_fwht(float *s, int lgrows, int lgcs) {
  const int npairs = 1 << (lgrows - 1 + lgcs);
  const int cmask = (1 << lgcs) - 1;
  for (int st = 0; st < lgrows; ++st) {
    __syncthreads();
    const int hmask = (1 << st) - 1;
    for (int p = threadIdx.x; p < npairs; p += blockDim.x) {
      const int q = p >> lgcs, c = p & cmask;
      const int r = ((q & ~hmask) << 1) | (q & hmask);
      float *a = s + ((r << lgcs) | c);
      float *b = a + (1 << (st + lgcs));
      const float u = *a, w = *b;
      *a = u + w;
      *b = u - w;
    }
  }
  __syncthreads();
}

// Unnormalised Walsh-Hadamard transform of N values held in registers.
template <int N>
__device__ __forceinline__ void fwht_regs_t(float *v) {
#pragma unroll
  for (int h = 1; h < N; h <<= 1)
#pragma unroll
    for (int i = 0; i < N; i += 2 * h)
#pragma unroll
      for (int j = i; j < i + h; ++j) {
        const float a = v[j], b = v[j + h];
        v[j] = a + b;
        v[j + h] = a - b;
      }
}

}  // namespace sk
