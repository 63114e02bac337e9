// sk_device.h -- random streams and small helpers shared by the host planner
// and the gfx950 kernels of the sketch library.
//
// Every random quantity of a sketch is a pure function of
// (seed, layer, stream, index) through Philox4x32-10 (Salmon et al., SC'11):
// key = (lo32 seed, hi32 seed), counter = (lo32 c, hi32 c, layer, stream).
//   signs      bit (j & 31) of word ((j >> 5) & 3) of block j >> 7; 1 -> -1
//   Gaussians  Box-Muller on the 24-bit uniforms of word pair ((j >> 1) & 1)
//              of block j >> 2: u1 = (top24 + 1) 2^-24, u2 = top24 2^-24,
//              g = sqrt(-2 ln u1) * (cos, sin)(2 pi u2) for even/odd j
//   indices    word (i & 3) of block i >> 2, masked to [0, N')
//   perms      8-round alternating Feistel network on [0, 2^w), split into
//              high ceil(w/2) / low floor(w/2) bits; round keys are the 8 words
//              of blocks 2 pid and 2 pid + 1; round function: 32-bit finaliser
//              of (half ^ key), masked to the updated half.
// The layout is version 1 of the stream specification.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define SK_HD __host__ __device__ __forceinline__

namespace sk {

constexpr int kRngVersion = 1;

enum Stream : uint32_t {
  ST_SIGN = 1,
  ST_GAUSS = 2,
  ST_INDEX = 3,
  ST_FFDPERM = 4,
  ST_PI1 = 5,
  ST_PI2 = 6,
  ST_QKA = 7,
  ST_QKB = 8,
  ST_QH = 9,
};

struct Key {
  uint32_t k0, k1;
};

SK_HD Key make_key(uint64_t seed) { return Key{(uint32_t)seed, (uint32_t)(seed >> 32)}; }

struct W4 {
  uint32_t w[4];
};

SK_HD W4 philox(uint64_t ctr, uint32_t layer, uint32_t stream, Key key) {
  uint32_t c0 = (uint32_t)ctr, c1 = (uint32_t)(ctr >> 32), c2 = layer, c3 = stream;
  uint32_t k0 = key.k0, k1 = key.k1;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
    const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
    c1 = (uint32_t)p1;
    c3 = (uint32_t)p0;
    c0 = n0;
    c2 = n2;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  W4 o;
  o.w[0] = c0;
  o.w[1] = c1;
  o.w[2] = c2;
  o.w[3] = c3;
  return o;
}

SK_HD uint32_t pick(const W4 &w, uint32_t i) {
  // i in [0,4); written as selects so that no private array is indexed
  return i == 0 ? w.w[0] : i == 1 ? w.w[1] : i == 2 ? w.w[2] : w.w[3];
}

// 32 sign bits covering coordinates [j & ~31, (j & ~31) + 32) of a layer.
SK_HD uint32_t sign_word(uint64_t j, uint32_t layer, Key key) {
  const W4 w = philox(j >> 7, layer, ST_SIGN, key);
  return pick(w, (uint32_t)(j >> 5) & 3u);
}

SK_HD float flip(float v, uint32_t bit) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __int_as_float(__float_as_int(v) ^ (int)(bit << 31));
#else
  return bit ? -v : v;
#endif
}

// Box-Muller on one word pair.
__device__ __forceinline__ float box_muller(uint32_t wa, uint32_t wb, bool odd) {
  const float u1 = (float)((wa >> 8) + 1u) * 5.9604644775390625e-8f;  // 2^-24, exact
  const float u2 = (float)(wb >> 8) * 5.9604644775390625e-8f;
  const float r = sqrtf(-2.0f * logf(u1));
  float s, c;
  sincospif(2.0f * u2, &s, &c);
  return odd ? r * s : r * c;
}

// Gaussian number j of (layer, stream).
__device__ __forceinline__ float gauss(uint64_t j, uint32_t layer, uint32_t stream, Key key) {
  const W4 w = philox(j >> 2, layer, stream, key);
  const bool hi = (j >> 1) & 1;
  return box_muller(hi ? w.w[2] : w.w[0], hi ? w.w[3] : w.w[1], j & 1);
}

// Four consecutive Gaussians 4q .. 4q+3 from one Philox block.
__device__ __forceinline__ void gauss4(uint64_t q, uint32_t layer, uint32_t stream, Key key, float g[4]) {
  const W4 w = philox(q, layer, stream, key);
  const float u1a = (float)((w.w[0] >> 8) + 1u) * 5.9604644775390625e-8f;
  const float u2a = (float)(w.w[1] >> 8) * 5.9604644775390625e-8f;
  const float u1b = (float)((w.w[2] >> 8) + 1u) * 5.9604644775390625e-8f;
  const float u2b = (float)(w.w[3] >> 8) * 5.9604644775390625e-8f;
  const float ra = sqrtf(-2.0f * logf(u1a)), rb = sqrtf(-2.0f * logf(u1b));
  float sa, ca, sb, cb;
  sincospif(2.0f * u2a, &sa, &ca);
  sincospif(2.0f * u2b, &sb, &cb);
  g[0] = ra * ca;
  g[1] = ra * sa;
  g[2] = rb * cb;
  g[3] = rb * sb;
}

SK_HD uint32_t sample_index(uint64_t i, uint32_t layer, Key key, uint64_t np) {
  const W4 w = philox(i >> 2, layer, ST_INDEX, key);
  return pick(w, (uint32_t)i & 3u) & (uint32_t)(np - 1);
}

SK_HD uint32_t fmix32(uint32_t h) {
  h ^= h >> 16;
  h *= 0x85EBCA6Bu;
  h ^= h >> 13;
  h *= 0xC2B2AE35u;
  h ^= h >> 16;
  return h;
}

struct PermKey {
  uint32_t k[8];
  uint32_t wl, ml, mh;
};

SK_HD PermKey perm_key(uint32_t layer, uint32_t stream, uint32_t pid, uint32_t w, Key key) {
  PermKey p;
  const W4 a = philox(2ull * pid, layer, stream, key);
  const W4 b = philox(2ull * pid + 1, layer, stream, key);
  for (int i = 0; i < 4; ++i) {
    p.k[i] = a.w[i];
    p.k[4 + i] = b.w[i];
  }
  p.wl = w / 2;
  p.ml = (1u << p.wl) - 1u;
  p.mh = (1u << (w - p.wl)) - 1u;
  return p;
}

SK_HD uint32_t perm_fwd(const PermKey &p, uint32_t x) {
  uint32_t hi = x >> p.wl, lo = x & p.ml;
#pragma unroll
  for (int r = 0; r < 8; r += 2) {
    hi ^= fmix32(lo ^ p.k[r]) & p.mh;
    lo ^= fmix32(hi ^ p.k[r + 1]) & p.ml;
  }
  return (hi << p.wl) | lo;
}

SK_HD uint32_t perm_inv(const PermKey &p, uint32_t y) {
  uint32_t hi = y >> p.wl, lo = y & p.ml;
#pragma unroll
  for (int r = 6; r >= 0; r -= 2) {
    lo ^= fmix32(hi ^ p.k[r + 1]) & p.ml;
    hi ^= fmix32(lo ^ p.k[r]) & p.mh;
  }
  return (hi << p.wl) | lo;
}

// Kronecker digits of N' = 2^lgn (Sec. 3, factors of at most 1024 columns):
// K = ceil(lgn / 10) digits, each of 10 bits except the most significant one,
// which holds the remaining lgn - 10 (K - 1) bits.  Returns K and fills
// lg[k] = log2 of digit k's range (k = 0 most significant).
SK_HD int kron_shapes_log2(int lgn, int lg[8]) {
  const int K = (lgn + 9) / 10;
  for (int k = 1; k < K; ++k) lg[k] = 10;
  if (K > 0) lg[0] = lgn - 10 * (K - 1);
  return K;
}

}  // namespace sk
