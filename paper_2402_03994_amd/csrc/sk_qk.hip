// sk_qk.hip -- QK (Kronecker) sketch kernels: per weight matrix X (m x n),
// Y = A X B^T with A (dA x m) ~ N(0, 1/dA) and B (dB x n) ~ N(0, 1/dB)
// (eq. straight with two Kronecker factors; the contraction is that of
// eq. qk_proof_tensor_dec).  Factors are generated on the device at creation
// in fp32 and rounded to nearest even into bf16; products accumulate in fp32.
#include "sk_launch.h"

namespace sk {

__device__ __forceinline__ uint16_t qk_f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float qk_bf2f(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

__global__ void k_qk_factor(uint16_t *__restrict__ dst, int64_t count, uint32_t layer, uint32_t stream, float scale,
                            Key key) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i >= count) return;
  dst[i] = qk_f2bf(gauss((uint64_t)i, layer, stream, key) * scale);
}

void launch_qk_factors(const sk_sketch *s, hipStream_t st) {
  for (const LayerDesc &ld : s->layers) {
    const int64_t na = (int64_t)ld.da * ld.m, nb = (int64_t)ld.db * ld.nc;
    hipLaunchKernelGGL(k_qk_factor, dim3((unsigned)((na + 255) / 256)), dim3(256), 0, st, s->d_qkfac + ld.fa_off, na,
                       (uint32_t)ld.layer_id, (uint32_t)ST_QKA, (float)(1.0 / sqrt((double)ld.da)), s->key);
    hipLaunchKernelGGL(k_qk_factor, dim3((unsigned)((nb + 255) / 256)), dim3(256), 0, st, s->d_qkfac + ld.fb_off, nb,
                       (uint32_t)ld.layer_id, (uint32_t)ST_QKB, (float)(1.0 / sqrt((double)ld.db)), s->key);
  }
  (void)hipGetLastError();
}

int64_t qk_workspace_elems(const sk_sketch *s, int layer, int64_t bc) {
  const LayerDesc &ld = s->layers[layer];
  return bc * (int64_t)ld.m * ld.db;
}

// T[v][i][c] = sum_j X[v][i][j] B[c][j]
template <bool BF16>
__global__ void k_qk_xbt(const void *__restrict__ x, const uint16_t *__restrict__ B, int m, int n, int db,
                         int64_t b_begin, float *__restrict__ t) {
  const int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int64_t v = blockIdx.y;
  if (e >= (int64_t)m * db) return;
  const int64_t i = e / db, c = e - (e / db) * db;
  const int64_t xo = ((b_begin + v) * m + i) * (int64_t)n;
  float acc = 0.0f;
  for (int64_t j = 0; j < n; ++j) {
    const float xv = BF16 ? qk_bf2f(((const uint16_t *)x)[xo + j]) : ((const float *)x)[xo + j];
    acc += xv * qk_bf2f(B[c * n + j]);
  }
  t[(v * m + i) * db + c] = acc;
}

// Y[v][a][c] = sum_i A[a][i] T[v][i][c]
__global__ void k_qk_at(const uint16_t *__restrict__ A, const float *__restrict__ t, int m, int da, int db,
                        int64_t D, int64_t col, int64_t b_begin, float *__restrict__ out, int accumulate) {
  const int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int64_t v = blockIdx.y;
  if (e >= (int64_t)da * db) return;
  const int64_t a = e / db, c = e - (e / db) * db;
  float acc = 0.0f;
  for (int64_t i = 0; i < m; ++i) acc += qk_bf2f(A[a * m + i]) * t[(v * m + i) * db + c];
  float *o = out + (b_begin + v) * D + col + e;
  *o = accumulate ? *o + acc : acc;
}

void launch_qk_apply(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc,
                     float *t_ws, int64_t batch_total, float *out, bool accumulate, hipStream_t st) {
  (void)batch_total;
  const LayerDesc &ld = s->layers[layer];
  const uint16_t *A = s->d_qkfac + ld.fa_off, *B = s->d_qkfac + ld.fb_off;
  dim3 g1((unsigned)(((int64_t)ld.m * ld.db + 255) / 256), (unsigned)bc);
  if (dtype == SK_BF16)
    hipLaunchKernelGGL(k_qk_xbt<true>, g1, dim3(256), 0, st, x, B, ld.m, ld.nc, ld.db, b_begin, t_ws);
  else
    hipLaunchKernelGGL(k_qk_xbt<false>, g1, dim3(256), 0, st, x, B, ld.m, ld.nc, ld.db, b_begin, t_ws);
  dim3 g2((unsigned)(((int64_t)ld.da * ld.db + 255) / 256), (unsigned)bc);
  hipLaunchKernelGGL(k_qk_at, g2, dim3(256), 0, st, A, t_ws, ld.m, ld.da, ld.db, s->D, ld.qk_col, b_begin, out,
                     (int)accumulate);
  (void)hipGetLastError();
}

// U[v][i][c] = sum_a A[a][i] Z[v][a][c]
__global__ void k_qk_atz(const uint16_t *__restrict__ A, const float *__restrict__ z, int m, int da, int db, int64_t D,
                         int64_t col, int64_t b_begin, float *__restrict__ u) {
  const int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int64_t v = blockIdx.y;
  if (e >= (int64_t)m * db) return;
  const int64_t i = e / db, c = e - (e / db) * db;
  float acc = 0.0f;
  for (int64_t a = 0; a < da; ++a) acc += qk_bf2f(A[a * m + i]) * z[(b_begin + v) * D + col + a * db + c];
  u[(v * m + i) * db + c] = acc;
}

// X'[v][i][j] = sum_c U[v][i][c] B[c][j] (+ theta0)
__global__ void k_qk_ub(const uint16_t *__restrict__ B, const float *__restrict__ u, int m, int n, int db,
                        int64_t b_begin, void *__restrict__ out, int out_dtype, const float *__restrict__ theta0) {
  const int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int64_t v = blockIdx.y;
  if (e >= (int64_t)m * n) return;
  const int64_t i = e / n, j = e - (e / n) * n;
  float acc = 0.0f;
  for (int64_t c = 0; c < db; ++c) acc += u[(v * m + i) * db + c] * qk_bf2f(B[c * n + j]);
  if (theta0) acc += theta0[e];
  const int64_t o = (b_begin + v) * (int64_t)m * n + e;
  if (out_dtype == SK_BF16)
    ((uint16_t *)out)[o] = qk_f2bf(acc);
  else
    ((float *)out)[o] = acc;
}

void launch_qk_apply_T(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, float *t_ws,
                       void *out, int out_dtype, const float *theta0, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const uint16_t *A = s->d_qkfac + ld.fa_off, *B = s->d_qkfac + ld.fb_off;
  dim3 g1((unsigned)(((int64_t)ld.m * ld.db + 255) / 256), (unsigned)bc);
  hipLaunchKernelGGL(k_qk_atz, g1, dim3(256), 0, st, A, z, ld.m, ld.da, ld.db, s->D, ld.qk_col, b_begin, t_ws);
  dim3 g2((unsigned)(((int64_t)ld.m * ld.nc + 255) / 256), (unsigned)bc);
  hipLaunchKernelGGL(k_qk_ub, g2, dim3(256), 0, st, B, t_ws, ld.m, ld.nc, ld.db, b_begin, out, out_dtype, theta0);
  (void)hipGetLastError();
}

}  // namespace sk
