// sk_qhaar.hip -- sketches with the random-orthogonal Kronecker pre-conditioner
// Q (Sec. 3, paragraphs "Alternative pre-conditioners" and "Direct usage of the
// pre-conditioner Q"; eq. straight; Table tab:gains_design_choices, rows
// "H_N -> Q"):
//
//   QKH    y = sqrt(N/D) R_D Q_N x       eq. straight on the flattened layer
//   AFJLQ  y = sqrt(N/D) G R_D Q_N x     eq. frikadel with H_N replaced by Q
//
// Q_N = Q_0 (x) ... (x) Q_{K-1} over the Kronecker factor sizes of N (at most
// 1024 each).  Factor k of a layer is Haar on the orthogonal group: the Q of the
// QR factorisation, with R's diagonal made positive, of the b_k x b_k matrix of
// the layer's QH Gaussian stream (number k 2^20 + r b_k + c at row r, column
// c).  The text applies Q without the sign diagonal B; a Haar factor needs no
// digit permutation either.
//
// With 2048 <= D <= 2^20, R_D keeps all 1024 rows of the last factor (T =
// 1024), the first D_m = D / 1024 rows of factor m = K - 2 and the first row of
// every leading factor.  Per layer and vector, with X_t the t-th b_m x T slab
// of the padded layer (row-major) and P = N / (b_m T) slabs:
//   Y (D_m x T) = A X' Qt^T,   X' = sum_t w[t] X_t,
//   A = sqrt(N/D) Q_m[:D_m, :],  Qt = Q_{K-1},  w = (x)_{k<m} Q_k[0, :],
// and the layer adds g . vec(Y) (AFJLQ) or vec(Y) (QKH) to the output.  The
// transpose is X' = A^T (Z Qt) written w[t] X' into every slab t (Z = the
// output vector as D_m x T, times g for AFJLQ).
//
// The factors are generated at creation on the host in double precision
// (Householder QR of each Gaussian matrix, one factor per thread) and stored
// in fp32: A, A^T, Qt, Qt^T and w per layer.  The contractions run on
// v_mfma_f32_16x16x4f32 (fp32 products, fp32 accumulation).  Which operand is
// contracted first follows the cost: a layer with fewer live rows of X than
// D_m (P = 1: biases and norms padded to N = D) multiplies by Qt^T first and
// then by the live columns of A; on the transpose side the same layers form
// only their live output rows.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <thread>
#include <vector>

#include "sk_kcommon.h"
#include "sk_launch.h"

namespace sk {

namespace {

typedef float f4v __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- factors
// Householder QR of a (b x b, column-major, overwritten) and the explicit Q
// with the signs of its columns set so that R has a positive diagonal.
void haar_from_gaussian(double *a, int b, double *q) {
  std::vector<double> tau(b, 0.0), rdiag(b, 0.0);
  for (int j = 0; j < b; ++j) {
    double *aj = a + (int64_t)j * b;
    double nrm2 = 0.0;
    for (int i = j; i < b; ++i) nrm2 += aj[i] * aj[i];
    const double alpha = aj[j], nrm = std::sqrt(nrm2);
    if (nrm == 0.0) continue;  // probability zero for Gaussian data: H_j = I
    const double beta = alpha >= 0.0 ? -nrm : nrm;
    const double v0 = alpha - beta;
    tau[j] = (beta - alpha) / beta;
    for (int i = j + 1; i < b; ++i) aj[i] /= v0;
    aj[j] = beta;
    rdiag[j] = beta;
    for (int c = j + 1; c < b; ++c) {
      double *ac = a + (int64_t)c * b;
      double s = ac[j];
      for (int i = j + 1; i < b; ++i) s += aj[i] * ac[i];
      s *= tau[j];
      ac[j] -= s;
      for (int i = j + 1; i < b; ++i) ac[i] -= s * aj[i];
    }
  }
  // Q = H_0 H_1 ... H_{b-1}: accumulate backwards onto the identity
  std::fill(q, q + (int64_t)b * b, 0.0);
  for (int i = 0; i < b; ++i) q[(int64_t)i * b + i] = 1.0;
  for (int j = b - 1; j >= 0; --j) {
    if (tau[j] == 0.0) continue;
    const double *v = a + (int64_t)j * b;  // v[j] = 1 (implicit), v[i] for i > j
    for (int c = j; c < b; ++c) {
      double *qc = q + (int64_t)c * b;
      double s = qc[j];
      for (int i = j + 1; i < b; ++i) s += v[i] * qc[i];
      s *= tau[j];
      qc[j] -= s;
      for (int i = j + 1; i < b; ++i) qc[i] -= s * v[i];
    }
  }
  for (int c = 0; c < b; ++c)
    if (rdiag[c] < 0.0)
      for (int i = 0; i < b; ++i) q[(int64_t)c * b + i] = -q[(int64_t)c * b + i];
}

// Standard normal number j of a stream in double precision: the Box-Muller
// transform of the stream specification (two 24-bit uniforms of a word pair).
double gauss64(uint64_t j, uint32_t layer, uint32_t stream, Key key) {
  const W4 w = philox(j >> 2, layer, stream, key);
  const uint32_t wa = w.w[((j >> 1) & 1) * 2], wb = w.w[((j >> 1) & 1) * 2 + 1];
  const double u1 = ((double)(wa >> 8) + 1.0) * (1.0 / 16777216.0);
  const double u2 = (double)(wb >> 8) * (1.0 / 16777216.0);
  const double r = std::sqrt(-2.0 * std::log(u1));
  const double t = 2.0 * M_PI * u2;
  return (j & 1) ? r * std::sin(t) : r * std::cos(t);
}

// ---------------------------------------------------------------- kernels
// P operand: fp32 buffer / the layer's input, rows v r + h = row h of vector v
enum { kPBuf = 0, kPStacked = 1 };
// Q operand: rows N (K-contiguous) / rows K from a buffer / folded input / a
// buffer times the table at w, element by element
enum { kQNT = 0, kQNNBuf = 1, kQNNFold = 2, kQNNMul = 3 };
// epilogue: fp32 store / sketch output / parameter-vector write / fp32 (+)= table at g times the product
enum { kEStore = 0, kEOut = 1, kEBcast = 2, kEMulAcc = 3 };

struct QhArgs {
  // C (M x N) = P (M x K) . op(Q); batch index v = blockIdx.y
  int M, N, K;
  const void *p;  // P: fp32 rows of ldp, batch stride p_vs; or the input (dtype, n_in per vector)
  int64_t p_vs;
  int ldp;
  int p_vec;      // 16-byte loads of P allowed (ldp % 4 == 0, aligned base)
  int p_rows;     // kPStacked: rows per vector
  int64_t p_off;  // kPStacked: first element of the rows (a slab's offset)
  int64_t o_off;  // kEBcast: first element written (a slab's offset)
  int nvec;       // slot form: vectors stacked
  int q_vec;      // NN fold: 16-byte (fp32) / 8-byte (bf16) loads of the input allowed
  const void *q;  // Q: NT: fp32 N x K (ldq = K); NN buffer: fp32 K x N; NN fold: the input
  int64_t q_vs;
  int dtype;      // input dtype (kPInput, kQNNFold)
  int64_t n_in;   // input elements per vector
  int64_t b_in;   // first batch row of the input
  const float *w; // fold / broadcast weights (P slabs)
  int nslab;      // P
  int64_t slab;   // elements per slab (b_m T)
  // epilogue
  void *dst;
  int64_t c_vs;
  int ldc;
  int dst_dtype;
  int64_t n_out;  // kEBcast: elements of the parameter vector
  int64_t D;      // kEOut: output row length
  int64_t b_out;  // first batch row of the output
  const float *g;       // kEOut: per-element factor (nullable)
  const float *theta0;  // kEBcast: added (nullable)
  int accumulate;
};

// Up to kQhSlots layers of the Qt-first form in one launch (grid z = slot).
constexpr int kQhSlots = 32;
struct QhSlots {
  int n;
  const void *x[kQhSlots];  // input [batch, n_in]
  int64_t n_in[kQhSlots];
  int rows[kQhSlots];       // live rows r
  const float *qt[kQhSlots];
  const float *A[kQhSlots];  // A (D_m x b_m)
  int lda[kQhSlots];
  const float *g[kQhSlots];  // G over [0, D) or null
  int64_t uoff[kQhSlots];    // float offset of the slot's U (bc r x T) in the workspace
};

__device__ __forceinline__ float load_in(const void *x, int dtype, int64_t i) {
  return dtype == SK_BF16 ? bf16_to_f32(((const uint16_t *)x)[i]) : ((const float *)x)[i];
}

// Four values of P at row `row`, columns k .. k + 3 (zero outside M x K or the input).
template <int PM>
__device__ __forceinline__ f4v load_p4(const QhArgs &a, int64_t v, int row, int k) {
  f4v r = {0.f, 0.f, 0.f, 0.f};
  if (row >= a.M) return r;
  if (PM == kPBuf) {
    const float *p = (const float *)a.p + v * a.p_vs + (int64_t)row * a.ldp;
    if (a.p_vec && k + 3 < a.K) return *(const f4v *)(p + k);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (k + e < a.K) r[e] = p[k + e];
  } else {
    const int vv = row / a.p_rows, h = row - (row / a.p_rows) * a.p_rows;
    const int64_t base = (a.b_in + vv) * a.n_in;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t f = a.p_off + (int64_t)h * a.ldp + k + e;
      if (k + e < a.K && f < a.n_in) r[e] = load_in(a.p, a.dtype, base + f);
    }
  }
  (void)v;
  return r;
}

// NN forms: rows k0 .. k0 + 15, columns c0 .. c0 + 63 of the Q operand, raw.
// Lane L loads row 4 q + L / 16, columns c0 + 4 (L % 16) .. + 3 (q < 4) of
// each of the PF slabs: 16-byte loads, 256 contiguous bytes per row.
template <int QM, int PF>
__device__ __forceinline__ void load_tile(const QhArgs &a, int64_t v, int k0, int c0, int lane, f4v (&r)[PF][4]) {
  const int cc = c0 + 4 * (lane & 15);
  // a tile wholly inside K and the input (tested once, uniformly): every load
  // is issued without a branch, so they are all in flight together
  if (QM == kQNNFold && a.q_vec && k0 + 15 < a.K &&
      (int64_t)(PF - 1) * a.slab + (int64_t)(k0 + 15) * a.N + c0 + 63 < a.n_in) {
    const int64_t base = (a.b_in + v) * a.n_in;
    if (a.dtype == SK_BF16) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int t = 0; t < PF; ++t) {
          const uint2 u = *(const uint2 *)((const uint16_t *)a.q + base + t * a.slab +
                                           (int64_t)(k0 + 4 * q + (lane >> 4)) * a.N + cc);
          r[t][q] = f4v{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u), __uint_as_float(u.y << 16),
                        __uint_as_float(u.y & 0xFFFF0000u)};
        }
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int t = 0; t < PF; ++t)
          r[t][q] = *(const f4v *)((const float *)a.q + base + t * a.slab + (int64_t)(k0 + 4 * q + (lane >> 4)) * a.N +
                                   cc);
    }
    return;
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int k = k0 + 4 * q + (lane >> 4);
#pragma unroll
    for (int t = 0; t < PF; ++t) r[t][q] = f4v{0.f, 0.f, 0.f, 0.f};
    if (k >= a.K) continue;
    if (QM == kQNNBuf || QM == kQNNMul) {
      r[0][q] = *(const f4v *)((const float *)a.q + v * a.q_vs + (int64_t)k * a.N + cc);
      if (QM == kQNNMul) r[0][q] *= *(const f4v *)(a.w + (int64_t)k * a.N + cc);
      continue;
    }
    const int64_t base = (a.b_in + v) * a.n_in;
#pragma unroll
    for (int t = 0; t < PF; ++t) {
      const int64_t f = t * a.slab + (int64_t)k * a.N + cc;
      if (a.q_vec && f + 3 < a.n_in) {
        if (a.dtype == SK_BF16) {
          const uint2 u = *(const uint2 *)((const uint16_t *)a.q + base + f);
          r[t][q] = f4v{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u), __uint_as_float(u.y << 16),
                        __uint_as_float(u.y & 0xFFFF0000u)};
        } else {
          r[t][q] = *(const f4v *)((const float *)a.q + base + f);
        }
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (f + e < a.n_in) r[t][q][e] = load_in(a.q, a.dtype, base + f + e);
      }
    }
  }
}

constexpr int kStageLd = 68;  // floats per staged row (64 + 4: 16-byte aligned rows)

// One workgroup per (16 TA x 16 TB output block, vector); the four waves take
// quarters of K and their partial blocks are added in wave order through LDS.
// Lane (li, g) of a 16 x 16 tile: P row li and Q column li, K slice 4 g .. 4 g
// + 3 of each 16-wide step (one MFMA per slice element), output rows 4 g .. 4 g
// + 3 of column li.  In the NN forms each wave stages its 16 x 64 tile of the
// Q operand in its own part of the LDS block (loaded one step ahead, slabs
// summed with their weights on the way in) and reads the MFMA fragments from
// there.
template <int TA, int TB, int PM, int QM, int PF, int EP, bool SL = false>
__global__ __launch_bounds__(256) void k_qh_gemm(QhArgs a, QhSlots sl) {
  if (SL) {  // the slot's layer: Qt-first form, vectors' rows stacked
    const int z = blockIdx.z;
    a.p = sl.x[z];
    a.n_in = sl.n_in[z];
    a.p_rows = sl.rows[z];
    a.M = a.p_rows * a.nvec;
    a.q = sl.qt[z];
    a.dst = (float *)a.dst + sl.uoff[z];
    if ((int)(blockIdx.x / (a.N / (16 * TB))) * TA * 16 >= a.M) return;  // whole workgroup
    a.c_vs = 0;
  }
  constexpr int kRed = TA * TB * 256;
  constexpr int kWave = kRed > 16 * kStageLd ? kRed : 16 * kStageLd;
  __shared__ __align__(16) float red[4][kWave];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int li = lane & 15, g = lane >> 4;
  const int nbb = a.N / (16 * TB);
  const int ba = blockIdx.x / nbb, bb = blockIdx.x - (blockIdx.x / nbb) * nbb;
  const int64_t v = blockIdx.y;
  const int r0 = ba * TA * 16, c0 = bb * TB * 16;
  const int per = ((a.K + 63) / 64) * 16;
  const int kb = wave * per, ke = kb + per < a.K ? kb + per : a.K;
  float *stage = red[wave];
  f4v acc[TA][TB];
#pragma unroll
  for (int i = 0; i < TA; ++i)
#pragma unroll
    for (int j = 0; j < TB; ++j) acc[i][j] = f4v{0.f, 0.f, 0.f, 0.f};
  constexpr int NR = QM == kQNT ? 1 : PF;
  f4v raw[NR][4];
  if (QM != kQNT && kb < ke) load_tile<QM, NR>(a, v, kb, c0, lane, raw);
  for (int k0 = kb; k0 < ke; k0 += 16) {
    f4v pv[TA], qv[TB];
    if (PM == kPBuf && a.p_vec && r0 + 16 * TA <= a.M && k0 + 15 < a.K) {
      // the workgroup's rows and this step wholly inside P (tested once): no per-load branch
      const float *pb = (const float *)a.p + v * a.p_vs;
#pragma unroll
      for (int i = 0; i < TA; ++i) pv[i] = *(const f4v *)(pb + (int64_t)(r0 + 16 * i + li) * a.ldp + k0 + 4 * g);
    } else {
#pragma unroll
      for (int i = 0; i < TA; ++i) pv[i] = load_p4<PM>(a, v, r0 + 16 * i + li, k0 + 4 * g);
    }
    if (QM == kQNT) {
      // Q rows are output columns, K-contiguous; K is a multiple of 16 here
#pragma unroll
      for (int j = 0; j < TB; ++j)
        qv[j] = *(const f4v *)((const float *)a.q + v * a.q_vs + (int64_t)(c0 + 16 * j + li) * a.K + k0 + 4 * g);
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        f4v x = raw[0][q];
        if (PF > 1) {
          x = a.w[0] * x;
#pragma unroll
          for (int t = 1; t < NR; ++t) x += a.w[t] * raw[t][q];
        }
        *(f4v *)(stage + (4 * q + (lane >> 4)) * kStageLd + 4 * (lane & 15)) = x;
      }
      if (k0 + 16 < ke) load_tile<QM, NR>(a, v, k0 + 16, c0, lane, raw);
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int j = 0; j < TB; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) qv[j][e] = stage[(4 * g + e) * kStageLd + 16 * j + li];
      __builtin_amdgcn_wave_barrier();
    }
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
      for (int i = 0; i < TA; ++i)
#pragma unroll
        for (int j = 0; j < TB; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(pv[i][e], qv[j][e], acc[i][j], 0, 0, 0);
  }
#pragma unroll
  for (int i = 0; i < TA; ++i)
#pragma unroll
    for (int j = 0; j < TB; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) red[wave][((i * TB + j) * 64 + lane) * 4 + q] = acc[i][j][q];
  __syncthreads();
  for (int e = threadIdx.x; e < TA * TB * 64; e += 256) {
    const int tile = e >> 6, ln = e & 63;
    const int i = tile / TB, j = tile - (tile / TB) * TB;
    const int col = c0 + 16 * j + (ln & 15);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int row = r0 + 16 * i + (ln >> 4) * 4 + q;
      if (row >= a.M) continue;
      const int o = (tile * 64 + ln) * 4 + q;
      const float y = ((red[0][o] + red[1][o]) + red[2][o]) + red[3][o];
      if (EP == kEStore) {
        ((float *)a.dst)[v * a.c_vs + (int64_t)row * a.ldc + col] = y;
      } else if (EP == kEOut) {
        const int64_t idx = (int64_t)row * a.N + col;
        float *o = (float *)a.dst + (a.b_out + v) * a.D + idx;
        const float val = a.g ? a.g[idx] * y : y;
        *o = a.accumulate ? *o + val : val;
      } else if (EP == kEMulAcc) {
        float *o = (float *)a.dst + v * a.c_vs + (int64_t)row * a.ldc + col;
        const float val = a.g[(int64_t)row * a.N + col] * y;
        *o = a.accumulate ? *o + val : val;
      } else {
        const int64_t idx = (int64_t)row * a.N + col;
        for (int t = 0; t < a.nslab; ++t) {
          const int64_t f = a.o_off + t * a.slab + idx;
          if (f >= a.n_out) break;
          float val = a.w ? a.w[t] * y : y;
          if (a.theta0) val += a.theta0[f];
          store_out(a.dst, a.dst_dtype, (a.b_out + v) * a.n_out + f, val);
        }
      }
    }
  }
}

// X'[v] (K x N) = sum_t w[t] X_t of the input (P slabs of K N elements), fp32.
// The slabs are read with 16-byte (fp32) or 8-byte (bf16) loads when vec is
// set, four slabs in flight per step.
__global__ __launch_bounds__(256) void k_qh_fold(const void *x, int dtype, int64_t n_in, int64_t b_in,
                                                 const float *__restrict__ w, int nslab, int64_t slab, int vec,
                                                 float *__restrict__ dst) {
  const int64_t e = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) * 4;
  const int64_t v = blockIdx.y;
  if (e >= slab) return;
  const int64_t base = (b_in + v) * n_in;
  f4v s = {0.f, 0.f, 0.f, 0.f};
  for (int t0 = 0; t0 < nslab; t0 += 4) {
    f4v r[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int t = t0 + u;
      const int64_t f = t * slab + e;
      r[u] = f4v{0.f, 0.f, 0.f, 0.f};
      if (t >= nslab) continue;
      if (vec && f + 3 < n_in) {
        if (dtype == SK_BF16) {
          const uint2 q = *(const uint2 *)((const uint16_t *)x + base + f);
          r[u] = f4v{__uint_as_float(q.x << 16), __uint_as_float(q.x & 0xFFFF0000u), __uint_as_float(q.y << 16),
                     __uint_as_float(q.y & 0xFFFF0000u)};
        } else {
          r[u] = *(const f4v *)((const float *)x + base + f);
        }
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (f + q < n_in) r[u][q] = load_in(x, dtype, base + f + q);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (t0 + u < nslab) s += w[t0 + u] * r[u];
  }
  *(f4v *)(dst + v * slab + e) = s;
}

// Y[v] (M x T) = A[:, :r] U[v] (r x T), A row-major with lda; epilogue as k_qh_gemm's
// kEStore (dst rows of T) or kEOut (sketch output with g).
template <int EP>
__global__ __launch_bounds__(256) void k_qh_small(const float *__restrict__ A, int lda, int M, int r,
                                                  const float *__restrict__ U, int64_t u_vs, int T, void *dst,
                                                  int64_t c_vs, int64_t D, int64_t b_out, const float *g,
                                                  int accumulate) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  const int row = blockIdx.z;
  const int64_t v = blockIdx.y;
  if (c >= T) return;
  const float *u = U + v * u_vs + c;
  const float *ar = A + (int64_t)row * lda;
  float s = 0.0f;
  for (int h = 0; h < r; ++h) s += ar[h] * u[(int64_t)h * T];
  if (EP == kEStore) {
    ((float *)dst)[v * c_vs + (int64_t)row * T + c] = s;
  } else {
    const int64_t idx = (int64_t)row * T + c;
    float *o = (float *)dst + (b_out + v) * D + idx;
    const float val = g ? g[idx] * s : s;
    *o = accumulate ? *o + val : val;
  }
  (void)M;
}

// w[v][i] = z[b + v][i] (times g[i])
__global__ void k_qh_zg(const float *__restrict__ z, int64_t D, int64_t b_in, const float *g, float *__restrict__ w) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int64_t v = blockIdx.y;
  if (i >= D) return;
  const float zz = z[(b_in + v) * D + i];
  w[v * D + i] = g ? zz * g[i] : zz;
}

// AFFDQ: M[t][e] = sum_t' c[t'][t] g[t' slab + e] over the layer's G stream
// (e < slab = b_m 1024); one thread per e holds the P <= kQhMaxLead values of g.
__global__ __launch_bounds__(256) void k_qh_mtab(const float *__restrict__ c, int P, int64_t slab, uint32_t layer_id,
                                                 Key key, float *__restrict__ m) {
  const int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (e >= slab) return;
  float g[kQhMaxLead];
#pragma unroll
  for (int t = 0; t < kQhMaxLead; ++t) g[t] = t < P ? gauss((uint64_t)(t * slab + e), layer_id, ST_GAUSS, key) : 0.0f;
  for (int t = 0; t < P; ++t) {
    float acc = 0.0f;
#pragma unroll
    for (int tp = 0; tp < kQhMaxLead; ++tp)
      if (tp < P) acc += c[tp * P + t] * g[tp];
    m[t * slab + e] = acc;
  }
}

int tiles_for(int m) { return m >= 64 ? 4 : m > 16 ? 2 : 1; }

template <int PM, int QM, int PF, int EP>
void launch_gemm(const QhArgs &a, int64_t bc, hipStream_t st) {
  const int ta = tiles_for(a.M);
  constexpr int TB = 4;  // N = 1024
  const unsigned nba = (unsigned)((a.M + 16 * ta - 1) / (16 * ta));
  const dim3 grid(nba * (unsigned)(a.N / (16 * TB)), (unsigned)bc);
  const QhSlots none{};
  if (ta == 4)
    hipLaunchKernelGGL((k_qh_gemm<4, TB, PM, QM, PF, EP>), grid, dim3(256), 0, st, a, none);
  else if (ta == 2)
    hipLaunchKernelGGL((k_qh_gemm<2, TB, PM, QM, PF, EP>), grid, dim3(256), 0, st, a, none);
  else
    hipLaunchKernelGGL((k_qh_gemm<1, TB, PM, QM, PF, EP>), grid, dim3(256), 0, st, a, none);
}

// out[v][idx] (+)= sum over the slots in order of g . (A[:, :r] U): one thread per (column, vector, row).
__global__ __launch_bounds__(256) void k_qh_small_slots(QhSlots sl, int T, const float *__restrict__ ws, float *out,
                                                        int64_t D, int64_t b_out, int accumulate) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  const int row = blockIdx.z;
  const int64_t v = blockIdx.y;
  if (c >= T) return;
  const int64_t idx = (int64_t)row * T + c;
  float total = 0.0f;
  for (int z = 0; z < sl.n; ++z) {
    const int r = sl.rows[z];
    const float *u = ws + sl.uoff[z] + v * r * (int64_t)T + c;
    const float *ar = sl.A[z] + (int64_t)row * sl.lda[z];
    float sum = 0.0f;
    for (int h = 0; h < r; ++h) sum += ar[h] * u[(int64_t)h * T];
    total += sl.g[z] ? sl.g[z][idx] * sum : sum;
  }
  float *o = out + (b_out + v) * D + idx;
  *o = accumulate ? *o + total : total;
}

}  // namespace

// ---------------------------------------------------------------- plan
int qh_plan_layer(LayerDesc &ld, int64_t D, int kind) {
  // factor m = K - 2 keeps D / 1024 rows; the last factor all 1024
  if (ld.K < 2 || ld.lg[ld.K - 1] != 10) return SK_EUNSUPPORTED;
  ld.qbm = 1 << ld.lg[ld.K - 2];
  ld.qdm = (int32_t)(D >> 10);
  ld.qP = ld.np / ((int64_t)ld.qbm << 10);
  if (kind == SK_AFFDQ && ld.qP > kQhMaxLead) return SK_EUNSUPPORTED;
  return ld.qdm >= 1 && ld.qdm <= ld.qbm ? SK_OK : SK_EUNSUPPORTED;
}

QhLayout qh_layout(const LayerDesc &ld, int kind) {
  const int64_t T2 = 1024 * 1024, bm = ld.qbm, dm = ld.qdm, P = ld.qP;
  QhLayout o{};
  if (kind != SK_AFFDQ) {
    o.a = 0;
    o.at = dm * bm;
    o.qt = 2 * dm * bm;
    o.qtt = o.qt + T2;
    o.w = o.qtt + T2;
    o.total = o.w + P;
  } else {
    o.q1m = 0;
    o.q1mt = bm * bm;
    o.q1l = 2 * bm * bm;
    o.q1lt = o.q1l + T2;
    o.a = o.q1lt + T2;
    o.at = o.a + dm * bm;
    o.qt = o.at + dm * bm;
    o.qtt = o.qt + T2;
    o.c = o.qtt + T2;
    o.m = (o.c + P * P + 3) & ~3ll;
    o.total = o.m + P * bm * 1024;
  }
  return o;
}

int64_t qh_layer_floats(const LayerDesc &ld, int kind) { return qh_layout(ld, kind).total; }

// Generates every layer's factors (host, fp64, threads over factors) and
// writes them in fp32 into host[] at the layers' offsets (qh_layout): for
// QKH/AFJLQ A, A^T, Qt, Qt^T and w; for AFFDQ the first set's factor K - 2 and
// its transpose, last factor and its transpose, the second set's A, A^T, Qt,
// Qt^T, and c[t'][t] = w2[t'] Qlead[t'][t] (w2: the second set's leading first
// rows, Qlead: the first set's leading factors) from which the device forms M.
void qh_generate_factors(const sk_sketch *s, std::vector<float> &host) {
  struct Job {
    int layer, k, b;  // k: factor index in the stream (second set: kQhSecond + digit)
  };
  const bool affd = s->kind == SK_AFFDQ;
  std::vector<Job> jobs;
  for (int l = 0; l < (int)s->layers.size(); ++l) {
    const LayerDesc &ld = s->layers[l];
    for (int k = 0; k < ld.K; ++k) {
      jobs.push_back(Job{l, k, 1 << ld.lg[k]});
      if (affd) jobs.push_back(Job{l, kQhSecond + k, 1 << ld.lg[k]});
    }
  }
  // largest factors first so the threads finish together
  std::stable_sort(jobs.begin(), jobs.end(), [](const Job &x, const Job &y) { return x.b > y.b; });
  // per layer and digit: first rows (QKH/AFJLQ, AFFDQ second set) and whole
  // leading factors (AFFDQ first set), row-major
  std::vector<std::vector<std::vector<double>>> lead(s->layers.size()), whole(s->layers.size());
  for (size_t l = 0; l < s->layers.size(); ++l) {
    lead[l].resize(s->layers[l].K);
    whole[l].resize(s->layers[l].K);
  }
  std::atomic<size_t> next{0};
  auto work = [&]() {
    std::vector<double> a, q;
    for (;;) {
      const size_t j = next.fetch_add(1);
      if (j >= jobs.size()) return;
      const Job jb = jobs[j];
      const LayerDesc &ld = s->layers[jb.layer];
      const int b = jb.b;
      const bool second = jb.k >= kQhSecond;
      const int digit = second ? jb.k - kQhSecond : jb.k;
      a.resize((size_t)b * b);
      q.resize((size_t)b * b);
      // A[r][c] = number k 2^20 + r b + c, stored column-major
      for (int r = 0; r < b; ++r)
        for (int c = 0; c < b; ++c)
          a[(size_t)c * b + r] = gauss64(((uint64_t)jb.k << 20) + (uint64_t)r * b + c, (uint32_t)ld.layer_id, ST_QH,
                                         s->key);
      haar_from_gaussian(a.data(), b, q.data());
      // q is column-major: Q[r][c] = q[c b + r]
      float *base = host.data() + ld.qoff;
      const QhLayout o = qh_layout(ld, s->kind);
      const double sc = std::sqrt((double)ld.np / (double)s->D);
      auto put = [&](int64_t off, int64_t offt, int rows, double scale) {  // rows x b and its transpose
        for (int r = 0; r < rows; ++r)
          for (int c = 0; c < b; ++c) {
            const float x = (float)(scale * q[(size_t)c * b + r]);
            base[off + (int64_t)r * b + c] = x;
            base[offt + (int64_t)c * rows + r] = x;
          }
      };
      const bool restricted = !affd || second;  // the set R_D applies to
      if (digit == ld.K - 2) {
        if (restricted) put(o.a, o.at, ld.qdm, sc);
        else put(o.q1m, o.q1mt, b, 1.0);
      } else if (digit == ld.K - 1) {
        if (restricted) put(o.qt, o.qtt, b, 1.0);
        else put(o.q1l, o.q1lt, b, 1.0);
      } else if (restricted) {
        std::vector<double> row(b);
        for (int c = 0; c < b; ++c) row[c] = q[(size_t)c * b];
        lead[jb.layer][digit] = std::move(row);  // distinct slot per job
      } else {
        std::vector<double> m((size_t)b * b);
        for (int r = 0; r < b; ++r)
          for (int c = 0; c < b; ++c) m[(size_t)r * b + c] = q[(size_t)c * b + r];
        whole[jb.layer][digit] = std::move(m);
      }
    }
  };
  unsigned nt = std::max(1u, std::min(16u, std::thread::hardware_concurrency()));
  nt = (unsigned)std::min<size_t>(nt, jobs.size());
  std::vector<std::thread> th;
  for (unsigned i = 1; i < nt; ++i) th.emplace_back(work);
  work();
  for (auto &t : th) t.join();
  for (size_t l = 0; l < s->layers.size(); ++l) {
    const LayerDesc &ld = s->layers[l];
    const QhLayout o = qh_layout(ld, s->kind);
    // w = Kronecker product of the leading first rows (digit 0 most significant)
    std::vector<double> w(1, 1.0);
    for (int k = 0; k < ld.K - 2; ++k) {
      std::vector<double> nw(w.size() * lead[l][k].size());
      for (size_t i = 0; i < w.size(); ++i)
        for (size_t c = 0; c < lead[l][k].size(); ++c) nw[i * lead[l][k].size() + c] = w[i] * lead[l][k][c];
      w.swap(nw);
    }
    float *base = host.data() + ld.qoff;
    if (!affd) {
      for (int64_t t = 0; t < ld.qP; ++t) base[o.w + t] = (float)w[t];
      continue;
    }
    // Qlead = Kronecker product of the first set's leading factors (P x P)
    std::vector<double> ql(1, 1.0);
    int64_t dim = 1;
    for (int k = 0; k < ld.K - 2; ++k) {
      const int64_t b = 1ll << ld.lg[k];
      std::vector<double> nq((size_t)(dim * b) * (dim * b));
      for (int64_t i = 0; i < dim; ++i)
        for (int64_t j = 0; j < dim; ++j)
          for (int64_t r = 0; r < b; ++r)
            for (int64_t c = 0; c < b; ++c)
              nq[(size_t)((i * b + r) * dim * b + j * b + c)] = ql[(size_t)(i * dim + j)] * whole[l][k][(size_t)(r * b + c)];
      ql.swap(nq);
      dim *= b;
    }
    for (int64_t tp = 0; tp < ld.qP; ++tp)
      for (int64_t t = 0; t < ld.qP; ++t) base[o.c + tp * ld.qP + t] = (float)(w[tp] * ql[(size_t)(tp * ld.qP + t)]);
  }
}

// Live rows of X (P = 1): rows of 1024 that hold input elements.
static int64_t qh_live_rows(const LayerDesc &ld) { return (ld.n + 1023) / 1024; }

static bool qh_b_first(const LayerDesc &ld) { return ld.qP == 1 && qh_live_rows(ld) < ld.qdm; }

int64_t qh_bytes_per_vector(const sk_sketch *s, int layer, bool transpose) {
  const LayerDesc &ld = s->layers[layer];
  const int64_t T = 1024;
  if (s->kind == SK_AFFDQ) return (2ll * ld.qbm + ld.qdm) * T * 4;  // U + F + T2, or U2 + F' + W
  if (!transpose) {
    if (qh_b_first(ld)) return 0;  // grouped: qh_small_bytes_per_vector
    const bool fold = !(ld.qP == 1 || ld.qP == 2 || ld.qP == 4);
    return (ld.qdm * T + (fold ? (int64_t)ld.qbm * T : 0)) * 4;
  }
  const int64_t rows = std::max<int64_t>(ld.qdm, ld.qP == 1 ? std::min<int64_t>(qh_live_rows(ld), ld.qbm) : 0);
  return (s->D + rows * T) * 4;
}

bool qh_small_layer(const sk_sketch *s, int layer) { return qh_b_first(s->layers[layer]); }

// Groups of up to kQhSlots consecutive Qt-first layers (in list order).
static std::vector<std::vector<int>> qh_groups(const sk_sketch *s, int l0, int l1) {
  std::vector<std::vector<int>> gs;
  for (int l = l0; l < l1; ++l) {
    if (!qh_b_first(s->layers[l])) continue;
    if (gs.empty() || (int)gs.back().size() == kQhSlots) gs.emplace_back();
    gs.back().push_back(l);
  }
  return gs;
}

int64_t qh_small_bytes_per_vector(const sk_sketch *s, int l0, int l1) {
  int64_t need = 0;
  for (const auto &grp : qh_groups(s, l0, l1)) {
    int64_t b = 0;
    for (int l : grp) b += qh_live_rows(s->layers[l]) * 1024 * 4;
    need = std::max(need, b);
  }
  return need;
}

int qh_small_group_count(const sk_sketch *s, int l0, int l1) { return (int)qh_groups(s, l0, l1).size(); }

// Group gi of the Qt-first layers in [l0, l1): phase 1 forms every slot's U
// (one launch), phase 2 adds the slots' contributions to out in slot order
// (one launch).  x[l - l0] is layer l's input.
void run_qh_small_group(const sk_sketch *s, int l0, int l1, int gi, const void *const *x, int dtype,
                        int64_t b_begin, int64_t bc, float *ws, float *out, bool accumulate, int phases,
                        hipStream_t st) {
  const std::vector<int> grp = qh_groups(s, l0, l1)[gi];
  QhSlots sl{};
  sl.n = (int)grp.size();
  int64_t uoff = 0;
  int maxr = 0, dm = 0;
  for (int z = 0; z < sl.n; ++z) {
    const int l = grp[z];
    const LayerDesc &ld = s->layers[l];
    const float *base = s->d_qh + ld.qoff;
    const QhLayout o = qh_layout(ld, s->kind);
    sl.x[z] = x[l - l0];
    sl.n_in[z] = ld.n;
    sl.rows[z] = (int)qh_live_rows(ld);
    sl.qt[z] = base + o.qt;
    sl.A[z] = base + o.a;
    sl.lda[z] = ld.qbm;
    sl.g[z] = s->kind == SK_AFJLQ ? s->d_gtab + (int64_t)l * s->D : nullptr;
    sl.uoff[z] = uoff;
    uoff += bc * sl.rows[z] * 1024;
    maxr = std::max(maxr, sl.rows[z]);
    dm = ld.qdm;
  }
  const int T = 1024;
  if (phases & 1) {
    QhArgs a{};
    a.N = T;
    a.K = T;
    a.ldp = T;
    a.dtype = dtype;
    a.b_in = b_begin;
    a.nvec = (int)bc;
    a.dst = ws;
    a.ldc = T;
    const int mmax = (int)(bc * maxr);
    const int ta = tiles_for(mmax);
    const unsigned nba = (unsigned)((mmax + 16 * ta - 1) / (16 * ta));
    const dim3 grid(nba * (unsigned)(T / 64), 1u, (unsigned)sl.n);
    if (ta == 4)
      hipLaunchKernelGGL((k_qh_gemm<4, 4, kPStacked, kQNT, 1, kEStore, true>), grid, dim3(256), 0, st, a, sl);
    else if (ta == 2)
      hipLaunchKernelGGL((k_qh_gemm<2, 4, kPStacked, kQNT, 1, kEStore, true>), grid, dim3(256), 0, st, a, sl);
    else
      hipLaunchKernelGGL((k_qh_gemm<1, 4, kPStacked, kQNT, 1, kEStore, true>), grid, dim3(256), 0, st, a, sl);
  }
  if (phases & 2) {
    const dim3 grid(T / 256, (unsigned)bc, (unsigned)dm);
    hipLaunchKernelGGL(k_qh_small_slots, grid, dim3(256), 0, st, sl, T, (const float *)ws, out, s->D, b_begin,
                       (int)accumulate);
  }
}

void run_qh_apply(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc, float *ws,
                  float *out, bool accumulate, int phases, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const float *base = s->d_qh + ld.qoff;
  const QhLayout o = qh_layout(ld, s->kind);
  const float *A = base + o.a, *Qt = base + o.qt, *w = base + o.w;
  const float *g = s->kind == SK_AFJLQ ? s->d_gtab + (int64_t)layer * s->D : nullptr;
  const int T = 1024;
  QhArgs a{};
  a.dtype = dtype;
  a.n_in = ld.n;
  a.b_in = b_begin;
  a.D = s->D;
  a.b_out = b_begin;
  a.g = g;
  a.accumulate = accumulate;
  // (the Qt-first layers go through run_qh_small_group)
  float *tbuf = ws, *xf = ws + bc * (int64_t)ld.qdm * T;
  if (phases & 1) {  // T (D_m x T) = A X'
    a.M = ld.qdm;
    a.N = T;
    a.K = ld.qbm;
    a.p = A;
    a.p_vs = 0;
    a.ldp = ld.qbm;
    a.p_vec = ld.qbm % 4 == 0;
    a.dst = tbuf;
    a.c_vs = (int64_t)ld.qdm * T;
    a.ldc = T;
    a.q = x;
    a.q_vec = ld.n % 4 == 0 && ((uintptr_t)x & (dtype == SK_BF16 ? 7 : 15)) == 0;
    a.w = w;
    a.nslab = (int)ld.qP;
    a.slab = (int64_t)ld.qbm * T;
    if (ld.qP == 1) {
      launch_gemm<kPBuf, kQNNFold, 1, kEStore>(a, bc, st);
    } else if (ld.qP == 2) {
      launch_gemm<kPBuf, kQNNFold, 2, kEStore>(a, bc, st);
    } else if (ld.qP == 4) {
      launch_gemm<kPBuf, kQNNFold, 4, kEStore>(a, bc, st);
    } else {
      const dim3 fg((unsigned)((a.slab / 4 + 255) / 256), (unsigned)bc);
      hipLaunchKernelGGL(k_qh_fold, fg, dim3(256), 0, st, x, dtype, ld.n, b_begin, w, (int)ld.qP, a.slab, a.q_vec,
                         xf);
      a.q = xf;
      a.q_vs = a.slab;
      launch_gemm<kPBuf, kQNNBuf, 1, kEStore>(a, bc, st);
    }
  }
  if (phases & 2) {  // out (+)= g . (T Qt^T)
    QhArgs b = a;
    b.M = ld.qdm;
    b.N = T;
    b.K = T;
    b.p = tbuf;
    b.p_vs = (int64_t)ld.qdm * T;
    b.ldp = T;
    b.p_vec = 1;
    b.q = Qt;
    b.q_vs = 0;
    b.dst = out;
    launch_gemm<kPBuf, kQNT, 1, kEOut>(b, bc, st);
  }
}

void run_qh_apply_T(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, float *ws, void *out,
                    int out_dtype, const float *theta0, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const float *base = s->d_qh + ld.qoff;
  const QhLayout o = qh_layout(ld, s->kind);
  const float *At = base + o.at, *QtT = base + o.qtt, *w = base + o.w;
  const float *g = s->kind == SK_AFJLQ ? s->d_gtab + (int64_t)layer * s->D : nullptr;
  const int T = 1024;
  float *zg = ws, *u = ws + bc * s->D;
  {
    const dim3 grid((unsigned)((s->D + 255) / 256), (unsigned)bc);
    hipLaunchKernelGGL(k_qh_zg, grid, dim3(256), 0, st, z, s->D, b_begin, g, zg);
  }
  QhArgs a{};
  a.N = T;
  a.dst = out;
  a.dst_dtype = out_dtype;
  a.n_out = ld.n;
  a.b_out = b_begin;
  a.theta0 = theta0;
  a.slab = (int64_t)ld.qbm * T;
  const int64_t live = qh_live_rows(ld);
  if (ld.qP == 1 && live < ld.qdm) {
    // V (live x T) = A^T[:live] Zg, then out = V Qt (rows beyond n dropped)
    const int r = (int)live;
    const dim3 grid(T / 256, (unsigned)bc, (unsigned)r);
    hipLaunchKernelGGL(k_qh_small<kEStore>, grid, dim3(256), 0, st, At, ld.qdm, r, ld.qdm, zg, s->D, T, (void *)u,
                       (int64_t)r * T, s->D, (int64_t)0, (const float *)nullptr, 0);
    a.M = r;
    a.K = T;
    a.p = u;
    a.p_vs = (int64_t)r * T;
    a.ldp = T;
    a.p_vec = 1;
    a.q = QtT;
    a.nslab = 1;
    a.w = nullptr;
    launch_gemm<kPBuf, kQNT, 1, kEBcast>(a, bc, st);
    return;
  }
  // U (D_m x T) = Zg Qt, then every slab t gets w[t] A^T U
  QhArgs b{};
  b.M = ld.qdm;
  b.N = T;
  b.K = T;
  b.p = zg;
  b.p_vs = s->D;
  b.ldp = T;
  b.p_vec = 1;
  b.q = QtT;
  b.dst = u;
  b.c_vs = (int64_t)ld.qdm * T;
  b.ldc = T;
  launch_gemm<kPBuf, kQNT, 1, kEStore>(b, bc, st);
  a.M = ld.qbm;
  a.K = ld.qdm;
  a.p = At;
  a.p_vs = 0;
  a.ldp = ld.qdm;
  a.p_vec = ld.qdm % 4 == 0;
  a.q = u;
  a.q_vs = (int64_t)ld.qdm * T;
  a.nslab = (int)ld.qP;
  a.w = w;
  launch_gemm<kPBuf, kQNNBuf, 1, kEBcast>(a, bc, st);
}

// ---------------------------------------------------------------- AFFDQ
void launch_affdq_mtab(const sk_sketch *s, int layer, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const QhLayout o = qh_layout(ld, s->kind);
  const int64_t slab = (int64_t)ld.qbm * 1024;
  hipLaunchKernelGGL(k_qh_mtab, dim3((unsigned)((slab + 255) / 256)), dim3(256), 0, st, s->d_qh + ld.qoff + o.c,
                     (int)ld.qP, slab, (uint32_t)ld.layer_id, s->key, s->d_qh + ld.qoff + o.m);
}

// Live rows (of 1024) of slab t of a layer.
static int affdq_slab_rows(const LayerDesc &ld, int64_t t) {
  const int64_t slab = (int64_t)ld.qbm * 1024;
  const int64_t left = ld.n - t * slab;
  if (left <= 0) return 0;
  return (int)std::min<int64_t>(ld.qbm, (left + 1023) / 1024);
}

// Forward.  Phase 1: F = sum_t M_t . (Q1m X_t Q1L^T) over the live slabs (per
// slab U = X_t Q1L^T on the live rows with the vectors stacked, then
// F (+)= M_t . (Q1m[:, :r] U)).  Phase 2: T2 = A2 F, out (+)= T2 Q2L^T.
void run_affdq_apply(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc, float *ws,
                     float *out, bool accumulate, int phases, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const float *base = s->d_qh + ld.qoff;
  const QhLayout o = qh_layout(ld, s->kind);
  const int T = 1024, bm = ld.qbm;
  const int64_t slab = (int64_t)bm * T;
  float *u = ws, *f = ws + bc * slab, *t2 = f + bc * slab;
  if (phases & 1) {
    bool first = true;
    for (int64_t t = 0; t < ld.qP; ++t) {
      const int r = affdq_slab_rows(ld, t);
      if (r == 0) break;
      QhArgs a{};
      a.M = (int)(bc * r);
      a.N = T;
      a.K = T;
      a.p = x;
      a.ldp = T;
      a.p_rows = r;
      a.p_off = t * slab;
      a.dtype = dtype;
      a.n_in = ld.n;
      a.b_in = b_begin;
      a.q = base + o.q1l;
      a.dst = u;
      a.ldc = T;
      launch_gemm<kPStacked, kQNT, 1, kEStore>(a, 1, st);
      QhArgs b{};
      b.M = bm;
      b.N = T;
      b.K = r;
      b.p = base + o.q1m;
      b.ldp = bm;
      b.p_vec = bm % 4 == 0;
      b.q = u;
      b.q_vs = (int64_t)r * T;
      b.dst = f;
      b.c_vs = slab;
      b.ldc = T;
      b.g = base + o.m + t * slab;
      b.accumulate = !first;
      launch_gemm<kPBuf, kQNNBuf, 1, kEMulAcc>(b, bc, st);
      first = false;
    }
    if (first) launch_fill_zero(f, bc * slab, st);  // no live slab (empty layer cannot occur; kept total)
  }
  if (phases & 2) {
    QhArgs a{};
    a.M = ld.qdm;
    a.N = T;
    a.K = bm;
    a.p = base + o.a;
    a.ldp = bm;
    a.p_vec = bm % 4 == 0;
    a.q = f;
    a.q_vs = slab;
    a.dst = t2;
    a.c_vs = (int64_t)ld.qdm * T;
    a.ldc = T;
    launch_gemm<kPBuf, kQNNBuf, 1, kEStore>(a, bc, st);
    QhArgs b{};
    b.M = ld.qdm;
    b.N = T;
    b.K = T;
    b.p = t2;
    b.p_vs = (int64_t)ld.qdm * T;
    b.ldp = T;
    b.p_vec = 1;
    b.q = base + o.qt;
    b.dst = out;
    b.D = s->D;
    b.b_out = b_begin;
    b.accumulate = accumulate;
    launch_gemm<kPBuf, kQNT, 1, kEOut>(b, bc, st);
  }
}

// Transpose: U2 = Z Q2L, F' = A2^T U2, then per live slab t the output rows
// X'_t[:r] = Q1m^T[:r] (M_t . F') Q1L.
void run_affdq_apply_T(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, float *ws,
                       void *out, int out_dtype, const float *theta0, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const float *base = s->d_qh + ld.qoff;
  const QhLayout o = qh_layout(ld, s->kind);
  const int T = 1024, bm = ld.qbm;
  const int64_t slab = (int64_t)bm * T;
  float *u2 = ws, *fp = ws + bc * (int64_t)ld.qdm * T, *w = fp + bc * slab;
  QhArgs a{};
  a.M = ld.qdm;
  a.N = T;
  a.K = T;
  a.p = z + b_begin * s->D;
  a.p_vs = s->D;
  a.ldp = T;
  a.p_vec = 1;
  a.q = base + o.qtt;
  a.dst = u2;
  a.c_vs = (int64_t)ld.qdm * T;
  a.ldc = T;
  launch_gemm<kPBuf, kQNT, 1, kEStore>(a, bc, st);
  QhArgs b{};
  b.M = bm;
  b.N = T;
  b.K = ld.qdm;
  b.p = base + o.at;
  b.ldp = ld.qdm;
  b.p_vec = ld.qdm % 4 == 0;
  b.q = u2;
  b.q_vs = (int64_t)ld.qdm * T;
  b.dst = fp;
  b.c_vs = slab;
  b.ldc = T;
  launch_gemm<kPBuf, kQNNBuf, 1, kEStore>(b, bc, st);
  for (int64_t t = 0; t < ld.qP; ++t) {
    const int r = affdq_slab_rows(ld, t);
    if (r == 0) break;
    QhArgs c{};
    c.M = r;
    c.N = T;
    c.K = bm;
    c.p = base + o.q1mt;
    c.ldp = bm;
    c.p_vec = bm % 4 == 0;
    c.q = fp;
    c.q_vs = slab;
    c.w = base + o.m + t * slab;
    c.dst = w;
    c.c_vs = (int64_t)r * T;
    c.ldc = T;
    launch_gemm<kPBuf, kQNNMul, 1, kEStore>(c, bc, st);
    QhArgs d{};
    d.M = r;
    d.N = T;
    d.K = T;
    d.p = w;
    d.p_vs = (int64_t)r * T;
    d.ldp = T;
    d.p_vec = 1;
    d.q = base + o.q1lt;
    d.dst = out;
    d.dst_dtype = out_dtype;
    d.n_out = ld.n;
    d.b_out = b_begin;
    d.theta0 = theta0;
    d.nslab = 1;
    d.slab = slab;
    d.o_off = t * slab;
    launch_gemm<kPBuf, kQNT, 1, kEBcast>(d, bc, st);
  }
}

}  // namespace sk
