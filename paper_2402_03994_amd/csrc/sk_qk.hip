// sk_qk.hip -- QK (Kronecker) sketch kernels: per weight matrix X (m x n),
// Y = A X B^T with A (dA x m) ~ N(0, 1/dA) and B (dB x n) ~ N(0, 1/dB)
// (eq. straight with two Kronecker factors; the contraction is that of
// eq. qk_proof_tensor_dec).  Factors are generated on the device at creation
// in fp32.  A and B are kept in fp32 and, for the bf16 matrix-core
// contractions of bf16 inputs, also as two bf16 terms, hi = bf16(F) and
// lo = bf16(F - hi) (both rounded to nearest even), so that X B^T =
// X hi^T + X lo^T sees B to 16 mantissa bits.  fp32 inputs and the transpose
// multiply by the fp32 factors.  Products accumulate in fp32.
#include <algorithm>

#include "sk_launch.h"

namespace sk {

__device__ __forceinline__ uint16_t qk_f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float qk_bf2f(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// A in fp32 and as bf16 hi / lo terms (for the contraction that applies A first)
__global__ void k_qk_factor_a(float *__restrict__ dst, uint16_t *__restrict__ hi, uint16_t *__restrict__ lo,
                              int64_t count, uint32_t layer, float scale, Key key) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i >= count) return;
  const float g = gauss((uint64_t)i, layer, ST_QKA, key) * scale;
  dst[i] = g;
  const uint16_t h = qk_f2bf(g);
  hi[i] = h;
  lo[i] = qk_f2bf(g - qk_bf2f(h));
}

// B in fp32 and as bf16 hi / lo terms
__global__ void k_qk_factor_b(float *__restrict__ dst, uint16_t *__restrict__ hi, uint16_t *__restrict__ lo,
                              int64_t count, uint32_t layer, float scale, Key key) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i >= count) return;
  const float g = gauss((uint64_t)i, layer, ST_QKB, key) * scale;
  dst[i] = g;
  const uint16_t h = qk_f2bf(g);
  hi[i] = h;
  lo[i] = qk_f2bf(g - qk_bf2f(h));
}

void launch_qk_factors(const sk_sketch *s, hipStream_t st) {
  for (const LayerDesc &ld : s->layers) {
    const int64_t na = (int64_t)ld.da * ld.m, nb = (int64_t)ld.db * ld.nc;
    hipLaunchKernelGGL(k_qk_factor_a, dim3((unsigned)((na + 255) / 256)), dim3(256), 0, st, s->d_qka + ld.fa_off,
                       s->d_qkah + ld.fa_off, s->d_qkah + s->qk_a_elems + ld.fa_off, na, (uint32_t)ld.layer_id,
                       (float)(1.0 / sqrt((double)ld.da)), s->key);
    hipLaunchKernelGGL(k_qk_factor_b, dim3((unsigned)((nb + 255) / 256)), dim3(256), 0, st, s->d_qkbf + ld.fb_off,
                       s->d_qkb + ld.fb_off, s->d_qkb + s->qk_b_elems + ld.fb_off, nb, (uint32_t)ld.layer_id,
                       (float)(1.0 / sqrt((double)ld.db)), s->key);
  }
  (void)hipGetLastError();
}

int64_t qk_workspace_elems(const sk_sketch *s, int layer, int64_t bc) {
  const LayerDesc &ld = s->layers[layer];
  return bc * std::max((int64_t)ld.m * ld.db, (int64_t)ld.da * ld.nc);
}

// T[v][i][c] = sum_j X[v][i][j] B[c][j] with the fp32 B (inputs that the
// matrix-core path does not take: fp32, or shapes off its tiling).  These
// one-thread-per-output loops sum in fp64 and round once, so their error does
// not grow with the contraction length.
template <bool BF16>
__global__ void k_qk_xbt(const void *__restrict__ x, const float *__restrict__ B, int m, int n, int db,
                         int64_t b_begin, float *__restrict__ t) {
  const int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int64_t v = blockIdx.y;
  if (e >= (int64_t)m * db) return;
  const int64_t i = e / db, c = e - (e / db) * db;
  const int64_t xo = ((b_begin + v) * m + i) * (int64_t)n;
  double acc = 0.0;
  for (int64_t j = 0; j < n; ++j) {
    const float xv = BF16 ? qk_bf2f(((const uint16_t *)x)[xo + j]) : ((const float *)x)[xo + j];
    acc = fma((double)xv, (double)B[c * n + j], acc);
  }
  t[(v * m + i) * db + c] = (float)acc;
}

// ---------------------------------------------------------------------------
// MFMA path (bf16 X, n % 128 == 0, dA and dB multiples of 16, dB <= 128).
// Stage 1: T^T[v][c][i] = sum_j X[v][i][j] B[c][j], a tall-skinny GEMM over
// the stacked rows of the batch (M = bc m, N = dB, K = n) on
// v_mfma_f32_16x16x32_bf16.  Each wave owns 16 rows; each lane streams 64
// contiguous bytes of its row per 128-wide K step and splits them over four
// MFMAs.  The pairing of K positions to MFMA slots is a fixed permutation of
// the contraction index applied identically to X and B, so it does not change
// the sum.  Stage 2: Y[v][a][c] = sum_i A[a][i] T^T[v][c][i] on
// v_mfma_f32_16x16x4f32 (fp32 T, bf16 A widened exactly).
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

union Pack8 {
  uint4 u;
  bf16x8 v;
};

constexpr int kQkMR = 4;                  // 16-row tiles per wave
constexpr int kQkRows = 4 * kQkMR * 16;   // stacked rows per workgroup (4 waves)
constexpr int kQkBRow = 128 * 2 + 16;     // bytes of one B row chunk in LDS (padded)

template <int NT>
__global__ __launch_bounds__(256) void k_qk_s1(const uint16_t *__restrict__ x, const uint16_t *__restrict__ B,
                                               const uint16_t *__restrict__ Blo, int64_t m, int64_t n,
                                               int64_t b_begin, int64_t rows, float *__restrict__ tt) {
  constexpr int DB = NT * 16;
  __shared__ __align__(16) unsigned char bs[2 * DB * kQkBRow];  // [hi|lo][row][128 bf16 + pad]
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int li = lane & 15, g = lane >> 4;
  const int64_t r0 = (int64_t)blockIdx.x * kQkRows + wave * (kQkMR * 16);
  const uint16_t *xr[kQkMR];
  bool rv[kQkMR];
#pragma unroll
  for (int mr = 0; mr < kQkMR; ++mr) {
    const int64_t row = r0 + mr * 16 + li;
    rv[mr] = row < rows;
    xr[mr] = x + (b_begin * m + (rv[mr] ? row : 0)) * n + g * 8;
  }
  floatx4 acc[kQkMR][NT];
#pragma unroll
  for (int mr = 0; mr < kQkMR; ++mr)
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[mr][t] = floatx4{0.f, 0.f, 0.f, 0.f};
  for (int64_t k0 = 0; k0 < n; k0 += 128) {
    // this wave's X fragments: MFMA cc takes k = k0 + 32 cc + 8 g .. + 7 in lane (li, g), so each load
    // instruction reads 64 contiguous bytes of each of 16 rows (16 cache lines, not 32 half-used ones:
    // the address units bound this loop)
    Pack8 a[kQkMR][4];
#pragma unroll
    for (int mr = 0; mr < kQkMR; ++mr)
#pragma unroll
      for (int cc = 0; cc < 4; ++cc)
        a[mr][cc].u = rv[mr] ? *(const uint4 *)(xr[mr] + k0 + cc * 32) : make_uint4(0, 0, 0, 0);
    __syncthreads();  // previous chunk of B consumed
    // B[hi|lo][row][k0 .. k0+127] -> LDS, 16 bytes per thread per step
    for (int e = threadIdx.x; e < 2 * DB * 16; e += 256) {
      const int arr = e / (DB * 16), rem = e - arr * (DB * 16);
      const int row = rem >> 4, c16 = rem & 15;
      const uint16_t *src = (arr ? Blo : B) + (int64_t)row * n + k0 + c16 * 8;
      *(uint4 *)(bs + (arr * DB + row) * kQkBRow + c16 * 16) = *(const uint4 *)src;
    }
    __syncthreads();
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const unsigned char *bh = bs + (t * 16 + li) * kQkBRow + g * 16;
      const unsigned char *bl = bh + DB * kQkBRow;
#pragma unroll
      for (int cc = 0; cc < 4; ++cc) {
        Pack8 vh, vl;
        vh.u = *(const uint4 *)(bh + cc * 64);
        vl.u = *(const uint4 *)(bl + cc * 64);
#pragma unroll
        for (int mr = 0; mr < kQkMR; ++mr)
          acc[mr][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mr][cc].v, vh.v, acc[mr][t], 0, 0, 0);
#pragma unroll
        for (int mr = 0; mr < kQkMR; ++mr)
          acc[mr][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mr][cc].v, vl.v, acc[mr][t], 0, 0, 0);
      }
    }
  }
  // D layout: lane holds rows 4 g .. 4 g + 3 of column li of each 16 x 16 tile
#pragma unroll
  for (int mr = 0; mr < kQkMR; ++mr)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t R = r0 + mr * 16 + g * 4 + i;
      if (R >= rows) continue;
      const int64_t v = R / m, ii = R - (R / m) * m;
#pragma unroll
      for (int t = 0; t < NT; ++t) tt[(v * DB + t * 16 + li) * m + ii] = acc[mr][t][i];
    }
}

// A first (dA < dB, so A X costs fewer products than X B^T): stage 1
// U[v][a][j] = sum_i A[a][i] X[v][i][j] on v_mfma_f32_16x16x32_bf16 with A as
// bf16 hi + lo.  X's contiguous index j is the output column, so each lane
// reads 8 bytes (columns j0 .. j0 + 3) of 8 consecutive rows and packs the
// 16-bit halves into the K fragments of four MFMAs (one per column), i.e. four
// 16-column sets interleaved with stride 4.  Each step takes 64 rows; the
// next step's rows load during the current MFMAs.  Stage 2 is k_qk_s2 with U
// per vector and B in fp32.
template <int MT>
__global__ __launch_bounds__(256) void k_qk_s1a(const uint16_t *__restrict__ x, const uint16_t *__restrict__ Ah,
                                                const uint16_t *__restrict__ Al, int64_t m, int64_t n,
                                                int64_t b_begin, float *__restrict__ u) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int li = lane & 15, g = lane >> 4;
  const int64_t v = blockIdx.y;
  const int64_t j0 = (int64_t)blockIdx.x * 256 + wave * 64 + 4 * li;  // this lane's four columns
  const uint16_t *xc = x + (b_begin + v) * m * n + j0 + (int64_t)(g * 8) * n;
  const uint16_t *ah = Ah + (int64_t)li * m + g * 8;
  const uint16_t *al = Al + (int64_t)li * m + g * 8;
  floatx4 acc[MT][4];
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[t][q] = floatx4{0.f, 0.f, 0.f, 0.f};
  uint2 w[2][8];  // rows k0 + 32 h + 8 g + r
  auto fetch = [&](int64_t k0) {
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int r = 0; r < 8; ++r) w[h][r] = *(const uint2 *)(xc + (k0 + 32 * h + r) * n);
  };
  fetch(0);
  for (int64_t k0 = 0; k0 < m; k0 += 64) {
    uint2 c[2][8];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int r = 0; r < 8; ++r) c[h][r] = w[h][r];
    if (k0 + 64 < m) fetch(k0 + 64);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      // K fragments (rows k0 + 32 h + 8 g .. + 7) of columns j0 + q
      Pack8 f[4];
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        uint32_t e[8];
#pragma unroll
        for (int r = 0; r < 8; ++r) e[r] = p ? c[h][r].y : c[h][r].x;
        f[2 * p].u = make_uint4(__builtin_amdgcn_perm(e[1], e[0], 0x05040100u),
                                __builtin_amdgcn_perm(e[3], e[2], 0x05040100u),
                                __builtin_amdgcn_perm(e[5], e[4], 0x05040100u),
                                __builtin_amdgcn_perm(e[7], e[6], 0x05040100u));
        f[2 * p + 1].u = make_uint4(__builtin_amdgcn_perm(e[1], e[0], 0x07060302u),
                                    __builtin_amdgcn_perm(e[3], e[2], 0x07060302u),
                                    __builtin_amdgcn_perm(e[5], e[4], 0x07060302u),
                                    __builtin_amdgcn_perm(e[7], e[6], 0x07060302u));
      }
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        Pack8 hv, lv;
        hv.u = *(const uint4 *)(ah + (int64_t)(t * 16) * m + k0 + 32 * h);
        lv.u = *(const uint4 *)(al + (int64_t)(t * 16) * m + k0 + 32 * h);
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[t][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(hv.v, f[q].v, acc[t][q], 0, 0, 0);
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[t][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lv.v, f[q].v, acc[t][q], 0, 0, 0);
      }
    }
  }
  // D layout: lane holds rows 4 g .. 4 g + 3 (a) of its column in each set
  float *ub = u + v * (int64_t)(MT * 16) * n + j0;
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t a = t * 16 + g * 4 + i;
      *(float4 *)(ub + a * n) = make_float4(acc[t][0][i], acc[t][1][i], acc[t][2][i], acc[t][3][i]);
    }
}

// The same stage with 16-byte loads: each lane reads eight columns j0 .. j0 + 7
// (two 128-byte lines per row for 16 lanes, half the load instructions of the
// 8-byte form for the same bytes), which gives eight 16-column sets per MFMA
// group; steps of 32 rows, the next step's rows loading during the MFMAs.
template <int MT>
__global__ __launch_bounds__(256) void k_qk_s1aw(const uint16_t *__restrict__ x, const uint16_t *__restrict__ Ah,
                                                 const uint16_t *__restrict__ Al, int64_t m, int64_t n,
                                                 int64_t b_begin, float *__restrict__ u) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int li = lane & 15, g = lane >> 4;
  const int64_t v = blockIdx.y;
  const int64_t j0 = (int64_t)blockIdx.x * 512 + wave * 128 + 8 * li;  // this lane's eight columns
  const uint16_t *xc = x + (b_begin + v) * m * n + j0 + (int64_t)(g * 8) * n;
  const uint16_t *ah = Ah + (int64_t)li * m + g * 8;
  const uint16_t *al = Al + (int64_t)li * m + g * 8;
  floatx4 acc[MT][8];
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[t][q] = floatx4{0.f, 0.f, 0.f, 0.f};
  uint4 w[8];  // rows k0 + 8 g + r, columns j0 .. j0 + 7
  auto fetch = [&](int64_t k0) {
#pragma unroll
    for (int r = 0; r < 8; ++r) w[r] = *(const uint4 *)(xc + (k0 + r) * n);
  };
  fetch(0);
  for (int64_t k0 = 0; k0 < m; k0 += 32) {
    // K fragments (rows k0 + 8 g .. + 7) of columns j0 + q, q < 8
    Pack8 f[8];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      uint32_t e[8];
#pragma unroll
      for (int r = 0; r < 8; ++r) e[r] = p == 0 ? w[r].x : p == 1 ? w[r].y : p == 2 ? w[r].z : w[r].w;
      f[2 * p].u = make_uint4(__builtin_amdgcn_perm(e[1], e[0], 0x05040100u),
                              __builtin_amdgcn_perm(e[3], e[2], 0x05040100u),
                              __builtin_amdgcn_perm(e[5], e[4], 0x05040100u),
                              __builtin_amdgcn_perm(e[7], e[6], 0x05040100u));
      f[2 * p + 1].u = make_uint4(__builtin_amdgcn_perm(e[1], e[0], 0x07060302u),
                                  __builtin_amdgcn_perm(e[3], e[2], 0x07060302u),
                                  __builtin_amdgcn_perm(e[5], e[4], 0x07060302u),
                                  __builtin_amdgcn_perm(e[7], e[6], 0x07060302u));
    }
    if (k0 + 32 < m) fetch(k0 + 32);  // w is free once packed
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      Pack8 hv, lv;
      hv.u = *(const uint4 *)(ah + (int64_t)(t * 16) * m + k0);
      lv.u = *(const uint4 *)(al + (int64_t)(t * 16) * m + k0);
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[t][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(hv.v, f[q].v, acc[t][q], 0, 0, 0);
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[t][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lv.v, f[q].v, acc[t][q], 0, 0, 0);
    }
  }
  // D layout: lane holds rows 4 g .. 4 g + 3 (a) of its column in each set
  float *ub = u + v * (int64_t)(MT * 16) * n + j0;
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t a = t * 16 + g * 4 + i;
      *(float4 *)(ub + a * n) = make_float4(acc[t][0][i], acc[t][1][i], acc[t][2][i], acc[t][3][i]);
      *(float4 *)(ub + a * n + 4) = make_float4(acc[t][4][i], acc[t][5][i], acc[t][6][i], acc[t][7][i]);
    }
}

// A first when it makes fewer products, and also when the 16-byte-load
// A-first kernel applies at most twice the products of the B-first order
// (the matrix cores are far from busy there; its whole-line X loads are not).
bool qk_afirst_ok(const LayerDesc &ld, int dtype) {
  if (dtype != SK_BF16 || ld.da % 16 != 0 || ld.db % 16 != 0 || ld.m % 64 != 0 || ld.nc % 256 != 0) return false;
  return (ld.da < ld.db && ld.da <= 64) || (ld.da <= 32 && ld.da <= 2 * ld.db && ld.nc % 512 == 0);
}

// Stage 2: Y[v][a][c] = sum_k P[a][k] Q[c][k] (P: dA rows, Q: dB rows, both
// with the contraction index contiguous; each may be per vector) on
// v_mfma_f32_16x16x4f32.  One workgroup per (vector, block of TA x TB output
// tiles of 16 x 16): each wave keeps the TA x TB accumulators of the block over
// a quarter of K, so every P and Q row is read once per workgroup, and the four
// partial blocks are added in a fixed order through LDS.
template <int TA, int TB>
__global__ __launch_bounds__(256) void k_qk_s2(const float *__restrict__ P, int64_t p_vs,
                                               const float *__restrict__ Q, int64_t q_vs, int64_t K, int da, int db,
                                               int64_t D, int64_t col, int64_t b_begin, float *__restrict__ out,
                                               int accumulate) {
  __shared__ float red[4][TA * TB][64][4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nbb = db / (16 * TB);
  const int ba = blockIdx.x / nbb, bb = blockIdx.x - (blockIdx.x / nbb) * nbb;
  const int64_t v = blockIdx.y;
  const int li = lane & 15, g = lane >> 4;
  const float *pr = P + v * p_vs + (int64_t)(ba * TA * 16 + li) * K + g * 4;
  const float *qr = Q + v * q_vs + (int64_t)(bb * TB * 16 + li) * K + g * 4;
  const int64_t per = ((K + 63) / 64) * 16;  // K range per wave, a multiple of 16
  const int64_t kb = wave * per, ke = kb + per < K ? kb + per : K;
  floatx4 acc[TA][TB];
#pragma unroll
  for (int i = 0; i < TA; ++i)
#pragma unroll
    for (int j = 0; j < TB; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  // U steps of 16 per iteration: all of an iteration's loads are in flight together
  constexpr int U = TA * TB >= 8 ? 2 : 4;
  int64_t k0 = kb;
  for (; k0 + 16 * U <= ke; k0 += 16 * U) {
    float4 pv[U][TA], qv[U][TB];
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int i = 0; i < TA; ++i) pv[u][i] = *(const float4 *)(pr + (int64_t)(i * 16) * K + k0 + 16 * u);
#pragma unroll
      for (int j = 0; j < TB; ++j) qv[u][j] = *(const float4 *)(qr + (int64_t)(j * 16) * K + k0 + 16 * u);
    }
    // consecutive MFMAs go to different accumulators so none waits on the last
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int i = 0; i < TA; ++i)
#pragma unroll
        for (int j = 0; j < TB; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(pv[u][i].x, qv[u][j].x, acc[i][j], 0, 0, 0);
#pragma unroll
      for (int i = 0; i < TA; ++i)
#pragma unroll
        for (int j = 0; j < TB; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(pv[u][i].y, qv[u][j].y, acc[i][j], 0, 0, 0);
#pragma unroll
      for (int i = 0; i < TA; ++i)
#pragma unroll
        for (int j = 0; j < TB; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(pv[u][i].z, qv[u][j].z, acc[i][j], 0, 0, 0);
#pragma unroll
      for (int i = 0; i < TA; ++i)
#pragma unroll
        for (int j = 0; j < TB; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(pv[u][i].w, qv[u][j].w, acc[i][j], 0, 0, 0);
    }
  }
  for (; k0 + 16 <= ke; k0 += 16) {
    float4 pv[TA], qv[TB];
#pragma unroll
    for (int i = 0; i < TA; ++i) pv[i] = *(const float4 *)(pr + (int64_t)(i * 16) * K + k0);
#pragma unroll
    for (int j = 0; j < TB; ++j) qv[j] = *(const float4 *)(qr + (int64_t)(j * 16) * K + k0);
#pragma unroll
    for (int i = 0; i < TA; ++i)
#pragma unroll
      for (int j = 0; j < TB; ++j) {
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(pv[i].x, qv[j].x, acc[i][j], 0, 0, 0);
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(pv[i].y, qv[j].y, acc[i][j], 0, 0, 0);
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(pv[i].z, qv[j].z, acc[i][j], 0, 0, 0);
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(pv[i].w, qv[j].w, acc[i][j], 0, 0, 0);
      }
  }
  if (k0 < ke) {  // ragged end of K (K not a multiple of 16)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool ok = k0 + g * 4 + e < ke;
      float pe[TA], qe[TB];
#pragma unroll
      for (int i = 0; i < TA; ++i) pe[i] = ok ? pr[(int64_t)(i * 16) * K + k0 + e] : 0.0f;
#pragma unroll
      for (int j = 0; j < TB; ++j) qe[j] = ok ? qr[(int64_t)(j * 16) * K + k0 + e] : 0.0f;
#pragma unroll
      for (int i = 0; i < TA; ++i)
#pragma unroll
        for (int j = 0; j < TB; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(pe[i], qe[j], acc[i][j], 0, 0, 0);
    }
  }
#pragma unroll
  for (int i = 0; i < TA; ++i)
#pragma unroll
    for (int j = 0; j < TB; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) red[wave][i * TB + j][lane][q] = acc[i][j][q];
  __syncthreads();
  // lane (li, g) of tile (i, j): rows 4 g .. 4 g + 3 of column li
  for (int e = threadIdx.x; e < TA * TB * 64; e += 256) {
    const int tile = e >> 6, ln = e & 63;
    const int i = tile / TB, j = tile - (tile / TB) * TB;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float y = ((red[0][tile][ln][q] + red[1][tile][ln][q]) + red[2][tile][ln][q]) + red[3][tile][ln][q];
      const int a = (ba * TA + i) * 16 + (ln >> 4) * 4 + q, c = (bb * TB + j) * 16 + (ln & 15);
      float *o = out + (b_begin + v) * D + col + (int64_t)a * db + c;
      *o = accumulate ? *o + y : y;
    }
  }
}

// Tiles per block along a side of n16 tiles: the largest of 4, 2, 1 dividing it.
static int qk_block_tiles(int n16) { return n16 % 4 == 0 ? 4 : n16 % 2 == 0 ? 2 : 1; }

static void launch_qk_s2(const float *P, int64_t p_vs, const float *Q, int64_t q_vs, int64_t K, int da, int db,
                         int64_t D, int64_t col, int64_t b_begin, int64_t bc, float *out, bool accumulate,
                         hipStream_t st) {
  const int ta = qk_block_tiles(da / 16), tb = qk_block_tiles(db / 16);
  const dim3 grid((unsigned)((da / (16 * ta)) * (db / (16 * tb))), (unsigned)bc);
#define SK_S2(A, B)                                                                                      \
  if (ta == A && tb == B)                                                                                \
  hipLaunchKernelGGL((k_qk_s2<A, B>), grid, dim3(256), 0, st, P, p_vs, Q, q_vs, K, da, db, D, col, b_begin, out, \
                     (int)accumulate)
  SK_S2(1, 1); SK_S2(1, 2); SK_S2(1, 4); SK_S2(2, 1); SK_S2(2, 2); SK_S2(2, 4); SK_S2(4, 1); SK_S2(4, 2); SK_S2(4, 4);
#undef SK_S2
}

bool qk_mfma_ok(const LayerDesc &ld, int dtype) {
  return dtype == SK_BF16 && ld.nc % 128 == 0 && ld.m % 16 == 0 && ld.da % 16 == 0 && ld.db % 16 == 0 && ld.db <= 128;
}

// Y[v][a][c] = sum_i A[a][i] T[v][i][c]
__global__ void k_qk_at(const float *__restrict__ A, const float *__restrict__ t, int m, int da, int db,
                        int64_t D, int64_t col, int64_t b_begin, float *__restrict__ out, int accumulate) {
  const int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int64_t v = blockIdx.y;
  if (e >= (int64_t)da * db) return;
  const int64_t a = e / db, c = e - (e / db) * db;
  double acc = 0.0;
  for (int64_t i = 0; i < m; ++i) acc = fma((double)A[a * m + i], (double)t[(v * m + i) * db + c], acc);
  float *o = out + (b_begin + v) * D + col + e;
  *o = accumulate ? *o + (float)acc : (float)acc;
}

void launch_qk_apply(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc,
                     float *t_ws, int stages, float *out, bool accumulate, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const float *A = s->d_qka + ld.fa_off;
  const uint16_t *B = s->d_qkb + ld.fb_off, *Blo = s->d_qkb + s->qk_b_elems + ld.fb_off;
  if (qk_afirst_ok(ld, dtype)) {
    if (stages & 1) {
      const uint16_t *Ah = s->d_qkah + ld.fa_off, *Al = s->d_qkah + s->qk_a_elems + ld.fa_off;
      const dim3 g1((unsigned)(ld.nc / 256), (unsigned)bc);
      if (ld.nc % 512 == 0 && ld.da <= 32) {
        // eight columns per lane (16-byte loads)
        const dim3 g1w((unsigned)(ld.nc / 512), (unsigned)bc);
        if (ld.da == 16)
          hipLaunchKernelGGL(k_qk_s1aw<1>, g1w, dim3(256), 0, st, (const uint16_t *)x, Ah, Al, (int64_t)ld.m,
                             (int64_t)ld.nc, b_begin, t_ws);
        else
          hipLaunchKernelGGL(k_qk_s1aw<2>, g1w, dim3(256), 0, st, (const uint16_t *)x, Ah, Al, (int64_t)ld.m,
                             (int64_t)ld.nc, b_begin, t_ws);
      } else switch (ld.da / 16) {
        case 1: hipLaunchKernelGGL(k_qk_s1a<1>, g1, dim3(256), 0, st, (const uint16_t *)x, Ah, Al, (int64_t)ld.m,
                                   (int64_t)ld.nc, b_begin, t_ws); break;
        case 2: hipLaunchKernelGGL(k_qk_s1a<2>, g1, dim3(256), 0, st, (const uint16_t *)x, Ah, Al, (int64_t)ld.m,
                                   (int64_t)ld.nc, b_begin, t_ws); break;
        case 3: hipLaunchKernelGGL(k_qk_s1a<3>, g1, dim3(256), 0, st, (const uint16_t *)x, Ah, Al, (int64_t)ld.m,
                                   (int64_t)ld.nc, b_begin, t_ws); break;
        default: hipLaunchKernelGGL(k_qk_s1a<4>, g1, dim3(256), 0, st, (const uint16_t *)x, Ah, Al, (int64_t)ld.m,
                                    (int64_t)ld.nc, b_begin, t_ws); break;
      }
    }
    if (stages & 2) {
      // Y[v][a][c] = sum_j U[v][a][j] B[c][j]
      launch_qk_s2(t_ws, (int64_t)ld.da * ld.nc, s->d_qkbf + ld.fb_off, 0, (int64_t)ld.nc, ld.da, ld.db, s->D,
                   ld.qk_col, b_begin, bc, out, accumulate, st);
    }
    (void)hipGetLastError();
    return;
  }
  if (qk_mfma_ok(ld, dtype)) {
    const int64_t rows = bc * (int64_t)ld.m;
    dim3 g1((unsigned)((rows + kQkRows - 1) / kQkRows));
    if (stages & 1) {
#define SK_S1(NT)                                                                                              \
  case NT:                                                                                                     \
    hipLaunchKernelGGL(k_qk_s1<NT>, g1, dim3(256), 0, st, (const uint16_t *)x, B, Blo, (int64_t)ld.m,           \
                       (int64_t)ld.nc,                                                                         \
                       b_begin, rows, t_ws);                                                                   \
    break;
    switch (ld.db / 16) {
      SK_S1(1) SK_S1(2) SK_S1(3) SK_S1(4) SK_S1(5) SK_S1(6) SK_S1(7) SK_S1(8)
      default: break;
    }
#undef SK_S1
    }
    if (stages & 2) {
      launch_qk_s2(A, 0, t_ws, (int64_t)ld.db * ld.m, (int64_t)ld.m, ld.da, ld.db, s->D, ld.qk_col, b_begin, bc, out,
                   accumulate, st);
    }
    (void)hipGetLastError();
    return;
  }
  if (stages & 1) {
    dim3 g1((unsigned)(((int64_t)ld.m * ld.db + 255) / 256), (unsigned)bc);
    const float *Bf = s->d_qkbf + ld.fb_off;
    if (dtype == SK_BF16)
      hipLaunchKernelGGL(k_qk_xbt<true>, g1, dim3(256), 0, st, x, Bf, ld.m, ld.nc, ld.db, b_begin, t_ws);
    else
      hipLaunchKernelGGL(k_qk_xbt<false>, g1, dim3(256), 0, st, x, Bf, ld.m, ld.nc, ld.db, b_begin, t_ws);
  }
  if (stages & 2) {
    dim3 g2((unsigned)(((int64_t)ld.da * ld.db + 255) / 256), (unsigned)bc);
    hipLaunchKernelGGL(k_qk_at, g2, dim3(256), 0, st, A, t_ws, ld.m, ld.da, ld.db, s->D, ld.qk_col, b_begin, out,
                       (int)accumulate);
  }
  (void)hipGetLastError();
}

// U[v][i][c] = sum_a A[a][i] Z[v][a][c]
__global__ void k_qk_atz(const float *__restrict__ A, const float *__restrict__ z, int m, int da, int db, int64_t D,
                         int64_t col, int64_t b_begin, float *__restrict__ u) {
  const int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int64_t v = blockIdx.y;
  if (e >= (int64_t)m * db) return;
  const int64_t i = e / db, c = e - (e / db) * db;
  double acc = 0.0;
  for (int64_t a = 0; a < da; ++a) acc = fma((double)A[a * m + i], (double)z[(b_begin + v) * D + col + a * db + c], acc);
  u[(v * m + i) * db + c] = (float)acc;
}

// X'[v][i][j] = sum_c U[v][i][c] B[c][j] (+ theta0), fp32 B
__global__ void k_qk_ub(const float *__restrict__ B, const float *__restrict__ u, int m, int n, int db,
                        int64_t b_begin, void *__restrict__ out, int out_dtype, const float *__restrict__ theta0) {
  const int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int64_t v = blockIdx.y;
  if (e >= (int64_t)m * n) return;
  const int64_t i = e / n, j = e - (e / n) * n;
  double acc = 0.0;
  for (int64_t c = 0; c < db; ++c) acc = fma((double)u[(v * m + i) * db + c], (double)B[c * n + j], acc);
  if (theta0) acc += theta0[e];
  const float r = (float)acc;
  const int64_t o = (b_begin + v) * (int64_t)m * n + e;
  if (out_dtype == SK_BF16)
    ((uint16_t *)out)[o] = qk_f2bf(r);
  else
    ((float *)out)[o] = r;
}

void launch_qk_apply_T(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, float *t_ws,
                       void *out, int out_dtype, const float *theta0, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const float *A = s->d_qka + ld.fa_off;
  const float *Bf = s->d_qkbf + ld.fb_off;
  dim3 g1((unsigned)(((int64_t)ld.m * ld.db + 255) / 256), (unsigned)bc);
  hipLaunchKernelGGL(k_qk_atz, g1, dim3(256), 0, st, A, z, ld.m, ld.da, ld.db, s->D, ld.qk_col, b_begin, t_ws);
  dim3 g2((unsigned)(((int64_t)ld.m * ld.nc + 255) / 256), (unsigned)bc);
  hipLaunchKernelGGL(k_qk_ub, g2, dim3(256), 0, st, Bf, t_ws, ld.m, ld.nc, ld.db, b_begin, out, out_dtype, theta0);
  (void)hipGetLastError();
}

}  // namespace sk
