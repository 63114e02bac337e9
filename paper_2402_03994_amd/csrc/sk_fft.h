// sk_fft.h -- batched complex FFTs held in LDS (Stockham autosort: radix-16
// stages, then radix-4, then one radix-2 stage where the bits run out), the
// transform engine of the Fourier pre-conditioner kernels.
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

// 4-point DFT in place (forward: X_m = sum_n x_n (-i)^{nm}; inverse: +i).
template <bool INV>
__device__ __forceinline__ void dft4(float2 &x0, float2 &x1, float2 &x2, float2 &x3) {
  const float2 a0 = cadd(x0, x2), a1 = csub(x0, x2), a2 = cadd(x1, x3), a3 = csub(x1, x3);
  const float2 ja3 = INV ? make_float2(-a3.y, a3.x) : make_float2(a3.y, -a3.x);
  x0 = cadd(a0, a2);
  x2 = csub(a0, a2);
  x1 = cadd(a1, ja3);
  x3 = csub(a1, ja3);
}

// exp(-+2 pi i m / 16) for the products r1 s2 (r1, s2 < 4) of a 16-point DFT
template <bool INV>
__device__ __forceinline__ float2 w16(int m) {
  constexpr float c1 = 0.92387953251128674f, s1 = 0.38268343236508977f, h = 0.70710678118654752f;
  float2 w;
  switch (m) {
    case 1: w = make_float2(c1, -s1); break;
    case 2: w = make_float2(h, -h); break;
    case 3: w = make_float2(s1, -c1); break;
    case 4: w = make_float2(0.f, -1.f); break;
    case 6: w = make_float2(-h, -h); break;
    case 9: w = make_float2(-c1, s1); break;
    default: w = make_float2(1.f, 0.f); break;
  }
  return INV ? cconj(w) : w;
}

// One Stockham stage of radix 16: the 16 inputs of a butterfly take the
// twiddles w^r (w = w_{16 Ns}^k; w and w^4 from the table, the other powers by
// products), then a 16-point DFT in registers as 4 x 4 (r = r1 + 4 r2,
// s = s2 + 4 s1: 4-point DFTs over r2, the twiddles w_16^{r1 s2}, 4-point DFTs
// over r1).  Half the LDS passes and barriers of two radix-4 stages.
template <bool INV, int NT, int MAXB, bool OPQ>
__device__ __forceinline__ void fft_stage16(float2 *buf, int lgL, int lgC, int lgNs, const float2 *__restrict__ tw,
                                            int lgS) {
  int tid = threadIdx.x;
  if (OPQ) asm volatile("" : "+v"(tid));
  const int C = 1 << lgC;
  const int nb = 1 << (lgL + lgC - 4);  // butterflies of the stage
  const int q = 1 << (lgL - 4);         // L / 16
  float2 v[MAXB][16];
#pragma unroll
  for (int i = 0; i < MAXB; ++i) {
    const int e = tid + NT * i;
    if (e < nb) {
      const int col = e & (C - 1), j = e >> lgC;
#pragma unroll
      for (int r = 0; r < 16; ++r) v[i][r] = buf[((j + r * q) << lgC) + col];
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
        const float2 w1 = twiddle32<INV>(tw, lgS, lgNs + 4, (uint32_t)k);
        const float2 w4 = twiddle32<INV>(tw, lgS, lgNs + 2, (uint32_t)k);  // w^4 = w_{4 Ns}^k
        const float2 w2 = cmul(w1, w1), w3 = cmul(w2, w1);
        const float2 w8 = cmul(w4, w4), w12 = cmul(w8, w4);
        v[i][1] = cmul(v[i][1], w1);
        v[i][2] = cmul(v[i][2], w2);
        v[i][3] = cmul(v[i][3], w3);
        v[i][4] = cmul(v[i][4], w4);
        v[i][8] = cmul(v[i][8], w8);
        v[i][12] = cmul(v[i][12], w12);
        v[i][5] = cmul(v[i][5], cmul(w4, w1));
        v[i][6] = cmul(v[i][6], cmul(w4, w2));
        v[i][7] = cmul(v[i][7], cmul(w4, w3));
        v[i][9] = cmul(v[i][9], cmul(w8, w1));
        v[i][10] = cmul(v[i][10], cmul(w8, w2));
        v[i][11] = cmul(v[i][11], cmul(w8, w3));
        v[i][13] = cmul(v[i][13], cmul(w12, w1));
        v[i][14] = cmul(v[i][14], cmul(w12, w2));
        v[i][15] = cmul(v[i][15], cmul(w12, w3));
      }
      // 4-point DFTs over r2 (inputs r1, r1 + 4, r1 + 8, r1 + 12 -> t[r1][s2] in slots r1 + 4 s2)
#pragma unroll
      for (int r1 = 0; r1 < 4; ++r1) dft4<INV>(v[i][r1], v[i][r1 + 4], v[i][r1 + 8], v[i][r1 + 12]);
#pragma unroll
      for (int r1 = 1; r1 < 4; ++r1)
#pragma unroll
        for (int s2 = 1; s2 < 4; ++s2) v[i][r1 + 4 * s2] = cmul(v[i][r1 + 4 * s2], w16<INV>(r1 * s2));
      // 4-point DFTs over r1 (slots 4 s2 .. 4 s2 + 3 -> y[s2 + 4 s1] in slot 4 s2 + s1)
#pragma unroll
      for (int s2 = 0; s2 < 4; ++s2) dft4<INV>(v[i][4 * s2], v[i][4 * s2 + 1], v[i][4 * s2 + 2], v[i][4 * s2 + 3]);
      const int d = ((j >> lgNs) << (lgNs + 4)) + k;
#pragma unroll
      for (int s2 = 0; s2 < 4; ++s2)
#pragma unroll
        for (int s1 = 0; s1 < 4; ++s1) buf[((d + ((s2 + 4 * s1) << lgNs)) << lgC) + col] = v[i][4 * s2 + s1];
    }
  }
  __syncthreads();
}

// In-place FFT of length 2^lgL along pos for 2^lgC columns: radix-16 stages
// (R16; they hold 16 complex values per butterfly in registers), then radix-4,
// then one radix-2 stage where the bits run out.
template <bool INV, int NT, int MAXE, bool OPQ = false, bool R16 = false>
__device__ __forceinline__ void lds_fft(float2 *buf, int lgL, int lgC, const float2 *__restrict__ tw, int lgS) {
  __syncthreads();  // the caller's writes to buf are visible to every thread
  int lgNs = 0;
  if (R16)
    for (; lgNs + 4 <= lgL; lgNs += 4) fft_stage16<INV, NT, (MAXE + 15) / 16, OPQ>(buf, lgL, lgC, lgNs, tw, lgS);
  for (; lgNs + 2 <= lgL; lgNs += 2) fft_stage<INV, 4, NT, (MAXE + 3) / 4, OPQ>(buf, lgL, lgC, lgNs, tw, lgS);
  if (lgNs < lgL) fft_stage<INV, 2, NT, (MAXE + 1) / 2, OPQ>(buf, lgL, lgC, lgNs, tw, lgS);
}

}  // namespace sk
