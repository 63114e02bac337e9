// sk_fft.h -- batched complex FFTs held in LDS (Stockham autosort: radix-4
// stages, then one radix-2 stage when log2 L is odd), the transform engine of
// the Fourier pre-conditioner kernels.
//
// Layout: buf[pos * C + col], pos < L along the transform, col < C columns,
// both powers of two, L * C <= NT * MAXE.  Twiddles come from a table
// tw[m] = exp(-2 pi i m / S) (S a power of two multiple of L, computed in
// double precision on the host), so no transcendental is evaluated here.
// Forward: X[k] = sum_n x[n] exp(-2 pi i n k / L); inverse (INV): the same
// with exp(+...), unscaled.  Every thread of the block must call lds_fft; it
// synchronises the block before returning.
#pragma once

#include <hip/hip_runtime.h>

namespace sk {

__device__ __forceinline__ float2 cmul(float2 a, float2 b) {
  return make_float2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
__device__ __forceinline__ float2 cmulc(float2 a, float2 b) {  // a * conj(b)
  return make_float2(a.x * b.x + a.y * b.y, a.y * b.x - a.x * b.y);
}
__device__ __forceinline__ float2 cconj(float2 a) { return make_float2(a.x, -a.y); }
__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
__device__ __forceinline__ float2 cscale(float2 a, float s) { return make_float2(a.x * s, a.y * s); }

// exp(-+2 pi i m / 2^lgn) from the table (m reduced modulo 2^lgn)
template <bool INV>
__device__ __forceinline__ float2 twiddle(const float2 *__restrict__ tw, int lgS, int lgn, int64_t m) {
  const float2 w = tw[(m & ((1ll << lgn) - 1)) << (lgS - lgn)];
  return INV ? cconj(w) : w;
}
// the same for m < 2^lgn < 2^31 (32-bit index arithmetic)
template <bool INV>
__device__ __forceinline__ float2 twiddle32(const float2 *__restrict__ tw, int lgS, int lgn, uint32_t m) {
  const float2 w = tw[m << (lgS - lgn)];
  return INV ? cconj(w) : w;
}

// One Stockham stage of radix R over the whole block's butterflies.  OPQ: the
// thread index passes through an empty asm, so the index arithmetic stays
// inside the caller's loops instead of being hoisted out of them into
// registers that outlive the transform (for transforms inside a loop that
// keeps other loads in flight).
template <bool INV, int R, int NT, int MAXB, bool OPQ>
__device__ __forceinline__ void fft_stage(float2 *buf, int lgL, int lgC, int lgNs, const float2 *__restrict__ tw,
                                          int lgS) {
  constexpr int lgR = R == 4 ? 2 : 1;
  int tid = threadIdx.x;
  if (OPQ) asm volatile("" : "+v"(tid));
  const int C = 1 << lgC;
  const int nb = 1 << (lgL + lgC - lgR);  // butterflies of the stage
  const int q = 1 << (lgL - lgR);         // L / R
  float2 v[MAXB][R];
#pragma unroll
  for (int i = 0; i < MAXB; ++i) {
    const int e = tid + NT * i;
    if (e < nb) {
      const int col = e & (C - 1), j = e >> lgC;
#pragma unroll
      for (int r = 0; r < R; ++r) v[i][r] = buf[((j + r * q) << lgC) + col];
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < MAXB; ++i) {
    const int e = tid + NT * i;
    if (e < nb) {
      const int col = e & (C - 1), j = e >> lgC;
      const int k = j & ((1 << lgNs) - 1);
      if (k) {
        // w^k from the table, w^2k and w^3k by products (one load per butterfly)
        const float2 w1 = twiddle32<INV>(tw, lgS, lgNs + lgR, (uint32_t)k);
        v[i][1] = cmul(v[i][1], w1);
        if (R == 4) {
          const float2 w2 = cmul(w1, w1);
          v[i][2] = cmul(v[i][2], w2);
          v[i][3] = cmul(v[i][3], cmul(w1, w2));
        }
      }
      if (R == 4) {
        const float2 a0 = cadd(v[i][0], v[i][2]), a1 = csub(v[i][0], v[i][2]);
        const float2 a2 = cadd(v[i][1], v[i][3]), a3 = csub(v[i][1], v[i][3]);
        // forward: w4 = -i, inverse: +i
        const float2 ja3 = INV ? make_float2(-a3.y, a3.x) : make_float2(a3.y, -a3.x);
        v[i][0] = cadd(a0, a2);
        v[i][2] = csub(a0, a2);
        v[i][1] = cadd(a1, ja3);
        v[i][3] = csub(a1, ja3);
      } else {
        const float2 a0 = cadd(v[i][0], v[i][1]), a1 = csub(v[i][0], v[i][1]);
        v[i][0] = a0;
        v[i][1] = a1;
      }
      const int d = ((j >> lgNs) << (lgNs + lgR)) + k;
#pragma unroll
      for (int r = 0; r < R; ++r) buf[((d + (r << lgNs)) << lgC) + col] = v[i][r];
    }
  }
  __syncthreads();
}

// In-place FFT of length 2^lgL along pos for 2^lgC columns.
template <bool INV, int NT, int MAXE, bool OPQ = false>
__device__ __forceinline__ void lds_fft(float2 *buf, int lgL, int lgC, const float2 *__restrict__ tw, int lgS) {
  __syncthreads();  // the caller's writes to buf are visible to every thread
  int lgNs = 0;
  for (; lgNs + 2 <= lgL; lgNs += 2) fft_stage<INV, 4, NT, (MAXE + 3) / 4, OPQ>(buf, lgL, lgC, lgNs, tw, lgS);
  if (lgNs < lgL) fft_stage<INV, 2, NT, (MAXE + 1) / 2, OPQ>(buf, lgL, lgC, lgNs, tw, lgS);
}

}  // namespace sk
