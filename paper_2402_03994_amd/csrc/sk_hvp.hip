// sk_hvp.hip -- the synthetic Hessian H = shift I + sum_j lambda_j v_j v_j^T
// (v_j = s_j / sqrt(N_tot), s_j regenerated Rademacher vectors), the sketched
// HVP operator v -> S H S^T v (Sec. 2, explicit form of the appendix on
// implicit vs explicit HVPs) and Arnoldi with full re-orthogonalisation in the
// sketched space (Sec. 4, "Scaling eigenvalue estimation").
//
// Kernels:
//  * k_hvp_dots / k_hvp_combine: one workgroup per 8192-element chunk of a
//    layer.  The chunk's sign words (64 Philox blocks x r vectors) are built
//    once in LDS; each thread owns 4 consecutive coordinates per 1024-element
//    step, so one 32-bit LDS word serves its 4 elements for one vector j.
//    dots: per-chunk fp32 inner products s_j . x (ordered workgroup
//    reduction); k_hvp_coef sums the chunks in fp64 in a fixed order and forms
//    lambda_j t_j / N_tot.  combine: y = shift x + sum_j coef_j s_j.  Both
//    passes stream x once (HBM bound for small r; about 4 VALU operations
//    per element and vector).
//  * Arnoldi (two classical Gram-Schmidt passes per step): k_arn_dots forms
//    the partial inner products of w with rows 0..j of Q (and with itself) per
//    2048-entry chunk, k_arn_reduce sums them in fp64 in a fixed order into
//    the coefficients and Hbar, k_arn_update subtracts Q^T c (four waves split
//    the rows, combined in a fixed order), k_arn_normalize divides by |w| or
//    zeroes the row on breakdown.  No atomics: results are deterministic.
//  * Intrinsic-dimension search (Sec. 4, the doubling search): conjugate
//    gradients on the free coordinates of omega for the quadratic
//    L(theta0 + S^T omega) (one sketched HVP per step; the vector updates and
//    their fp64 dot products in single-workgroup kernels), the metric from the
//    quadratic's expansion at theta0, the doubling decision on the host.
#include <cmath>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/sketch_hvp.h"
#include "sk_launch.h"

using namespace sk;

namespace {

constexpr int kChunk = 8192;               // coordinates per workgroup item
constexpr int kBlocksPerChunk = kChunk / 128;  // Philox sign blocks per item
constexpr int kArnChunk = 2048;            // Arnoldi dot chunk (256 threads x 8)
constexpr int kArnRows = 8;                // Q rows per Arnoldi dot workgroup

struct HvpItem {
  int32_t layer;  // index into the layer list (RNG layer id)
  int32_t len;    // coordinates in this item (<= kChunk)
  int64_t e0;     // first coordinate (a multiple of kChunk)
};

// Per-layer input and output of one H x pass (a device table, so that one
// launch covers every layer).
struct HvpLayerPtr {
  const float *x;
  float *y;
  int64_t n;
};

int fail(int code, const std::string &msg) {
  sk::set_error(code, msg);
  return code;
}

struct DeviceGuard {
  int prev = -1;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != dev) (void)hipSetDevice(dev);
  }
  ~DeviceGuard() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

}  // namespace

struct sk_hvp {
  int device = 0;
  int rank = 0;
  float shift = 0.0f;
  uint64_t seed = 0;
  Key key{};
  int64_t max_batch = 0;
  int64_t total = 0;               // N_tot
  std::vector<int64_t> n, off;     // per layer: elements, offset in the concatenation
  std::vector<float> lambdas;
  std::vector<HvpItem> items;
  HvpItem *d_items = nullptr;
  float *d_lambda = nullptr;
  float *d_part = nullptr;   // [items][batch][r] per-chunk inner products
  float *d_coef = nullptr;   // [batch][r]
  float *X = nullptr, *Y = nullptr;  // sketch_hvp workspace, ws_floats each (>= max_batch * N_tot)
  int64_t ws_floats = 0;
  // per-layer pointers into X and Y for the sketch entry points, and the device tables of the
  // H x passes: X -> Y (filled at creation) and the caller's buffers of sk_hvp_apply (uploaded per
  // call from pinned host memory; the upload's event guards the host copy's reuse)
  std::vector<void *> xsk;
  std::vector<const void *> ysk;
  HvpLayerPtr *d_ws_tab = nullptr, *d_user_tab = nullptr, *h_user_tab = nullptr;
  hipEvent_t user_ev = nullptr;
  bool user_ev_pending = false;
  // kernel timing
  struct Rec {
    int cls, ev;
    int64_t bytes;
  };
  uint32_t prof_mask = 0;
  std::vector<hipEvent_t> evpool;
  int evnext = 0;
  std::vector<Rec> recs;
};

namespace {

struct HvpProf {
  sk_hvp *h;
  int idx = -1;
  hipStream_t st;
  HvpProf(sk_hvp *h_, int cls, int64_t bytes, hipStream_t st_) : h(h_), st(st_) {
    if (!h || !((h->prof_mask >> cls) & 1u) || h->evnext + 2 > (int)h->evpool.size()) return;
    idx = h->evnext;
    h->evnext += 2;
    h->recs.push_back(sk_hvp::Rec{cls, idx, bytes});
    (void)hipEventRecord(h->evpool[idx], st);
  }
  ~HvpProf() {
    if (idx >= 0) (void)hipEventRecord(h->evpool[idx + 1], st);
  }
};

typedef float f4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float flip_sign(float v, uint32_t bit) {
  return __int_as_float(__float_as_int(v) ^ (int)(bit << 31));
}

// Sign words of the item's blocks for vectors 0..r-1: sw[(blk * r + j) * 4 + q].
__device__ __forceinline__ void build_sign_table(uint32_t *sw, const HvpItem &it, int r, Key key) {
  const int nblk = (it.len + 127) >> 7;
  const uint64_t b0 = (uint64_t)it.e0 >> 7;
  for (int u = threadIdx.x; u < nblk * r; u += blockDim.x) {
    const int blk = u / r, j = u - blk * r;
    const W4 w = philox(b0 + (uint64_t)blk, ((uint32_t)it.layer << 6) | (uint32_t)j, SK_STREAM_HVP, key);
    uint4 v;
    v.x = w.w[0];
    v.y = w.w[1];
    v.z = w.w[2];
    v.w = w.w[3];
    *reinterpret_cast<uint4 *>(&sw[u * 4]) = v;
  }
}

// Loads the thread's 4 consecutive coordinates starting at local position p of
// a row (zeros past len).
__device__ __forceinline__ void load4(const float *row, int64_t p, int len_left, float v[4], bool vec) {
  if (vec && len_left >= 4) {
    const f4v q = __builtin_nontemporal_load(reinterpret_cast<const f4v *>(row + p));
    v[0] = q.x;
    v[1] = q.y;
    v[2] = q.z;
    v[3] = q.w;
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = k < len_left ? row[p + k] : 0.0f;
  }
}

template <int RB>
__global__ __launch_bounds__(256) void k_hvp_dots(const HvpItem *__restrict__ items,
                                                  const HvpLayerPtr *__restrict__ tab, int r, int64_t batch, Key key,
                                                  float *__restrict__ part) {
  __shared__ __align__(16) uint32_t sw[kBlocksPerChunk * RB * 4];
  __shared__ float red[4][RB];
  const HvpItem it = items[blockIdx.x];
  build_sign_table(sw, it, r, key);
  __syncthreads();
  const HvpLayerPtr lp = tab[it.layer];
  const int64_t n = lp.n;
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int q = (t >> 3) & 3, sh = (t & 7) * 4;
  for (int64_t b = 0; b < batch; ++b) {
    const float *row = lp.x + b * n + it.e0;
    const bool vec = ((reinterpret_cast<uintptr_t>(row) & 15u) == 0);
    float acc[RB];
#pragma unroll
    for (int j = 0; j < RB; ++j) acc[j] = 0.0f;
    for (int i = 0; i < kChunk / 1024; ++i) {
      const int p = 1024 * i + 4 * t;
      if (p >= it.len) break;
      float v[4];
      load4(row, p, it.len - p, v, vec);
      const int blk = 8 * i + (t >> 5);
#pragma unroll
      for (int j = 0; j < RB; ++j) {
        if (j < r) {
          const uint32_t w = sw[(blk * r + j) * 4 + q] >> sh;
          acc[j] += flip_sign(v[0], w & 1u) + flip_sign(v[1], (w >> 1) & 1u) +
                    (flip_sign(v[2], (w >> 2) & 1u) + flip_sign(v[3], (w >> 3) & 1u));
        }
      }
    }
#pragma unroll
    for (int j = 0; j < RB; ++j) {
      if (j < r) {
        float a = acc[j];
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) a += __shfl_xor(a, m, 64);
        if (lane == 0) red[wv][j] = a;
      }
    }
    __syncthreads();
    if (t < r) part[((int64_t)blockIdx.x * batch + b) * r + t] = (red[0][t] + red[1][t]) + (red[2][t] + red[3][t]);
    __syncthreads();
  }
}

// coef[b][j] = lambda_j / N_tot * sum over items (fp64, fixed order).
__global__ __launch_bounds__(256) void k_hvp_coef(const float *__restrict__ part, int64_t n_items, int64_t batch,
                                                  int r, const float *__restrict__ lambda, double inv_total,
                                                  float *__restrict__ coef) {
  __shared__ double red[256];
  const int bj = blockIdx.x;  // b * r + j
  const int64_t b = bj / r;
  const int j = bj - (int)b * r;
  double a = 0.0;
  for (int64_t i = threadIdx.x; i < n_items; i += 256) a += (double)part[(i * batch + b) * r + j];
  red[threadIdx.x] = a;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) coef[bj] = (float)((double)lambda[j] * red[0] * inv_total);
}

template <int RB>
__global__ __launch_bounds__(256) void k_hvp_combine(const HvpItem *__restrict__ items,
                                                     const HvpLayerPtr *__restrict__ tab, int r, int64_t batch,
                                                     Key key, float shift, const float *__restrict__ coef) {
  __shared__ __align__(16) uint32_t sw[kBlocksPerChunk * RB * 4];
  const HvpItem it = items[blockIdx.x];
  build_sign_table(sw, it, r, key);
  __syncthreads();
  const HvpLayerPtr lp = tab[it.layer];
  const int64_t n = lp.n;
  const int t = threadIdx.x;
  const int q = (t >> 3) & 3, sh = (t & 7) * 4;
  for (int64_t b = 0; b < batch; ++b) {
    const float *row = lp.x + b * n + it.e0;
    float *yrow = lp.y + b * n + it.e0;
    const bool vec = ((reinterpret_cast<uintptr_t>(row) & 15u) == 0) && ((reinterpret_cast<uintptr_t>(yrow) & 15u) == 0);
    float c[RB];
#pragma unroll
    for (int j = 0; j < RB; ++j) c[j] = j < r ? coef[b * r + j] : 0.0f;
    for (int i = 0; i < kChunk / 1024; ++i) {
      const int p = 1024 * i + 4 * t;
      if (p >= it.len) break;
      float v[4];
      load4(row, p, it.len - p, v, vec);
      float o[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) o[k] = shift * v[k];
      const int blk = 8 * i + (t >> 5);
#pragma unroll
      for (int j = 0; j < RB; ++j) {
        if (j < r) {
          const uint32_t w = sw[(blk * r + j) * 4 + q] >> sh;
#pragma unroll
          for (int k = 0; k < 4; ++k) o[k] += flip_sign(c[j], (w >> k) & 1u);
        }
      }
      if (vec && it.len - p >= 4) {
        const f4v ov = {o[0], o[1], o[2], o[3]};
        __builtin_nontemporal_store(ov, reinterpret_cast<f4v *>(yrow + p));
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if (p + k < it.len) yrow[p + k] = o[k];
      }
    }
  }
}

// ---- Arnoldi ---------------------------------------------------------------
// partial[c * ldp + row] = sum over chunk c of Q[row] . w (row < nrows) or w . w (row == nrows).
__global__ __launch_bounds__(256) void k_arn_dots(const float *__restrict__ Q, int64_t D, int nrows,
                                                  const float *__restrict__ w, float *__restrict__ partial, int ldp) {
  __shared__ float red[4][kArnRows];
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int64_t c = blockIdx.x;
  const int row0 = blockIdx.y * kArnRows;
  float wl[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int64_t d = c * kArnChunk + t + 256 * i;
    wl[i] = d < D ? w[d] : 0.0f;
  }
  float acc[kArnRows];
#pragma unroll
  for (int rr = 0; rr < kArnRows; ++rr) {
    const int row = row0 + rr;
    float a = 0.0f;
    if (row < nrows) {
      const float *qr = Q + (int64_t)row * D;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int64_t d = c * kArnChunk + t + 256 * i;
        if (d < D) a += qr[d] * wl[i];
      }
    } else if (row == nrows) {
#pragma unroll
      for (int i = 0; i < 8; ++i) a += wl[i] * wl[i];
    }
    acc[rr] = a;
  }
#pragma unroll
  for (int rr = 0; rr < kArnRows; ++rr) {
    float a = acc[rr];
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) a += __shfl_xor(a, m, 64);
    if (lane == 0) red[wv][rr] = a;
  }
  __syncthreads();
  if (t < kArnRows && row0 + t <= nrows)
    partial[c * ldp + row0 + t] = (red[0][t] + red[1][t]) + (red[2][t] + red[3][t]);
}

// Sums the chunk partials of rows 0..nrows (fp64, fixed order).  pass 0: Hbar[row][j] = c; pass 1:
// Hbar[row][j] += c; rows < nrows go to cvec, row nrows (w . w) to scal[pass].
__global__ __launch_bounds__(256) void k_arn_reduce(const float *__restrict__ partial, int64_t nchunk, int ldp,
                                                    int nrows, int pass, float *__restrict__ Hbar, int k, int j,
                                                    float *__restrict__ cvec, float *__restrict__ scal) {
  for (int row = threadIdx.x; row <= nrows; row += 256) {
    double a = 0.0;
    for (int64_t c = 0; c < nchunk; ++c) a += (double)partial[c * ldp + row];
    if (row < nrows) {
      const float cf = (float)a;
      cvec[row] = cf;
      float *h = Hbar + (int64_t)row * k + j;
      *h = pass == 0 ? cf : *h + cf;
    } else {
      scal[pass] = (float)a;
    }
  }
}

// w[d] -= sum_{row < nrows} cvec[row] Q[row][d]; four waves split the rows, combined in order.
__global__ __launch_bounds__(256) void k_arn_update(const float *__restrict__ Q, int64_t D, int nrows,
                                                    const float *__restrict__ cvec, float *__restrict__ w) {
  __shared__ float red[4][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t d = (int64_t)blockIdx.x * 64 + lane;
  float a0 = 0.0f, a1 = 0.0f;
  if (d < D) {
    int row = wv;
    for (; row + 4 < nrows; row += 8) {
      a0 += cvec[row] * Q[(int64_t)row * D + d];
      a1 += cvec[row + 4] * Q[(int64_t)(row + 4) * D + d];
    }
    if (row < nrows) a0 += cvec[row] * Q[(int64_t)row * D + d];
  }
  red[wv][lane] = a0 + a1;
  __syncthreads();
  if (wv == 0 && d < D) w[d] -= (red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane]);
}

// beta = sqrt(scal[2]); w /= beta or w = 0 on breakdown (beta <= tol sqrt(scal[0])); Hbar column tail.
__global__ __launch_bounds__(256) void k_arn_normalize(float *__restrict__ w, int64_t D, const float *__restrict__ scal,
                                                       int first, float *__restrict__ Hbar, int k, int j, float tol) {
  const float beta = sqrtf(scal[2]);
  const bool ok = first ? beta > 0.0f : beta > tol * sqrtf(scal[0]);
  const float inv = ok ? 1.0f / beta : 0.0f;
  for (int64_t d = (int64_t)blockIdx.x * 256 + threadIdx.x; d < D; d += (int64_t)gridDim.x * 256) w[d] *= inv;
  if (!first && blockIdx.x == 0) {
    for (int i = j + 1 + threadIdx.x; i <= k; i += 256) Hbar[(int64_t)i * k + j] = (i == j + 1 && ok) ? beta : 0.0f;
  }
}

int64_t arn_nchunk(int64_t D) { return (D + kArnChunk - 1) / kArnChunk; }

// Queues one Arnoldi step (see sketch_arnoldi_step); arguments already validated.
void arnoldi_step(float *Q, int64_t D, int j, float *Hbar, int k, float *work, hipStream_t st, sk_hvp *prof) {
  const int64_t nch = arn_nchunk(D);
  const int ldp = k + 2;
  float *partial = work, *cvec = work + nch * ldp, *scal = cvec + ldp;
  float *w = Q + (int64_t)(j + 1) * D;
  const int nrows = j + 1;  // rows 0..j
  const unsigned ngrid = (unsigned)std::min<int64_t>((D + 255) / 256, 4096);
  HvpProf ps(prof, 2, (int64_t)(j + 2) * D * 4 * 5, st);
  if (j >= 0) {
    for (int pass = 0; pass < 2; ++pass) {
      hipLaunchKernelGGL(k_arn_dots, dim3((unsigned)nch, (unsigned)((nrows + 1 + kArnRows - 1) / kArnRows)),
                         dim3(256), 0, st, Q, D, nrows, w, partial, ldp);
      hipLaunchKernelGGL(k_arn_reduce, dim3(1), dim3(256), 0, st, partial, nch, ldp, nrows, pass, Hbar, k, j, cvec,
                         scal);
      hipLaunchKernelGGL(k_arn_update, dim3((unsigned)((D + 63) / 64)), dim3(256), 0, st, Q, D, nrows, cvec, w);
    }
  }
  // |w|^2 after the passes (or of row 0) into scal[2]
  hipLaunchKernelGGL(k_arn_dots, dim3((unsigned)nch, 1u), dim3(256), 0, st, Q, D, 0, w, partial, ldp);
  hipLaunchKernelGGL(k_arn_reduce, dim3(1), dim3(256), 0, st, partial, nch, ldp, 0, 2, Hbar, k, j < 0 ? 0 : j, cvec,
                     scal);
  hipLaunchKernelGGL(k_arn_normalize, dim3(ngrid), dim3(256), 0, st, w, D, scal, j < 0 ? 1 : 0, Hbar, k,
                     j < 0 ? 0 : j, (float)SK_ARNOLDI_BREAKDOWN_TOL);
  (void)hipGetLastError();
}

template <int RB>
void launch_hvp(sk_hvp *h, const HvpLayerPtr *tab, int64_t batch, int pass, hipStream_t st) {
  const unsigned nitems = (unsigned)h->items.size();
  if (pass == 0)
    hipLaunchKernelGGL(k_hvp_dots<RB>, dim3(nitems), dim3(256), 0, st, h->d_items, tab, h->rank, batch, h->key,
                       h->d_part);
  else
    hipLaunchKernelGGL(k_hvp_combine<RB>, dim3(nitems), dim3(256), 0, st, h->d_items, tab, h->rank, batch, h->key,
                       h->shift, h->d_coef);
}

// Queues H x -> y for `batch` vectors (validated); tab: the device table of the layers' x, y, n.
void hvp_run(sk_hvp *h, const HvpLayerPtr *tab, int64_t batch, hipStream_t st) {
  const int64_t bytes = batch * h->total * 4;
  for (int pass = 0; pass < 2; ++pass) {
    HvpProf ps(h, pass, pass == 0 ? bytes : 2 * bytes, st);
    if (h->rank <= 8)
      launch_hvp<8>(h, tab, batch, pass, st);
    else if (h->rank <= 16)
      launch_hvp<16>(h, tab, batch, pass, st);
    else
      launch_hvp<32>(h, tab, batch, pass, st);
    if (pass == 0)
      hipLaunchKernelGGL(k_hvp_coef, dim3((unsigned)(batch * h->rank)), dim3(256), 0, st, h->d_part,
                         (int64_t)h->items.size(), batch, h->rank, h->d_lambda, 1.0 / (double)h->total, h->d_coef);
  }
  (void)hipGetLastError();
}

// ---- intrinsic-dimension search ----------------------------------------------
// Per-item partial inner products x . y over every layer of a table (one vector).
__global__ __launch_bounds__(256) void k_tab_dot(const HvpItem *__restrict__ items, const HvpLayerPtr *__restrict__ tab,
                                                 float *__restrict__ part) {
  __shared__ float red[4];
  const HvpItem it = items[blockIdx.x];
  const HvpLayerPtr lp = tab[it.layer];
  float a = 0.0f;
  for (int i = threadIdx.x; i < it.len; i += 256) a += lp.x[it.e0 + i] * lp.y[it.e0 + i];
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) a += __shfl_xor(a, m, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = a;
  __syncthreads();
  if (threadIdx.x == 0) part[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

// out = scale * sum of n partials (fp64, fixed order; one workgroup).
__global__ __launch_bounds__(256) void k_sum_f64(const float *__restrict__ part, int64_t n, double scale,
                                                 double *__restrict__ out) {
  __shared__ double red[256];
  double a = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += 256) a += (double)part[i];
  red[threadIdx.x] = a;
  __syncthreads();
  for (int st = 128; st > 0; st >>= 1) {
    if ((int)threadIdx.x < st) red[threadIdx.x] += red[threadIdx.x + st];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = scale * red[0];
}

// Block-wide fp64 sum over a 1024-thread workgroup (every thread gets the total).
__device__ __forceinline__ double block_sum_1024(double v, double *red) {
  red[threadIdx.x] = v;
  __syncthreads();
  for (int st = 512; st > 0; st >>= 1) {
    if ((int)threadIdx.x < st) red[threadIdx.x] += red[threadIdx.x + st];
    __syncthreads();
  }
  const double t = red[0];
  __syncthreads();
  return t;
}

enum { kIdL0 = 0, kIdRR = 1, kIdL = 2, kIdTau = 3 };  // slots of the search's fp64 scalars

// Round start: r = (g0 + w) on the free coordinates (i < d), 0 elsewhere; p = -r; rr = r.r.
__global__ __launch_bounds__(1024) void k_cg_start(const float *__restrict__ g0, const float *__restrict__ w,
                                                   float *__restrict__ r, float *__restrict__ p, int64_t d,
                                                   int64_t D, double *__restrict__ scal) {
  __shared__ double red[1024];
  double a = 0.0;
  for (int64_t i = threadIdx.x; i < D; i += 1024) {
    const float ri = i < d ? g0[i] + w[i] : 0.0f;
    r[i] = ri;
    p[i] = -ri;
    a += (double)ri * ri;
  }
  const double rr = block_sum_1024(a, red);
  if (threadIdx.x == 0) scal[kIdRR] = rr;
}

// One conjugate-gradient step on the free coordinates, q = (S H S^T p) given: alpha = rr / p.q,
// omega += alpha p, r += alpha q, beta = r.r / rr, p = -r + beta p.  p.q <= 0 or rr = 0 leaves the
// state unchanged.
__global__ __launch_bounds__(1024) void k_cg_step(float *__restrict__ omega, float *__restrict__ r,
                                                  float *__restrict__ p, const float *__restrict__ q, int64_t d,
                                                  double *__restrict__ scal) {
  __shared__ double red[1024];
  double a = 0.0;
  for (int64_t i = threadIdx.x; i < d; i += 1024) a += (double)p[i] * q[i];
  const double pq = block_sum_1024(a, red);
  const double rr = scal[kIdRR];
  if (!(pq > 0.0) || rr == 0.0) return;  // uniform over the workgroup
  const float alpha = (float)(rr / pq);
  double b = 0.0;
  for (int64_t i = threadIdx.x; i < d; i += 1024) {
    omega[i] += alpha * p[i];
    const float ri = r[i] + alpha * q[i];
    r[i] = ri;
    b += (double)ri * ri;
  }
  const double rr_new = block_sum_1024(b, red);
  const float beta = (float)(rr_new / rr);
  for (int64_t i = threadIdx.x; i < d; i += 1024) p[i] = -r[i] + beta * p[i];
  if (threadIdx.x == 0) scal[kIdRR] = rr_new;
}

// L = L0 + g0 . omega + 1/2 omega . w (w = S H S^T omega; the quadratic's expansion at theta0),
// tau = 1 - L / L0.
__global__ __launch_bounds__(1024) void k_id_eval(const float *__restrict__ g0, const float *__restrict__ w,
                                                  const float *__restrict__ omega, int64_t D,
                                                  double *__restrict__ scal) {
  __shared__ double red[1024];
  double a = 0.0;
  for (int64_t i = threadIdx.x; i < D; i += 1024) a += (double)omega[i] * ((double)g0[i] + 0.5 * (double)w[i]);
  const double t = block_sum_1024(a, red);
  if (threadIdx.x == 0) {
    const double L0 = scal[kIdL0];
    const double L = L0 + t;
    scal[kIdL] = L;
    scal[kIdTau] = 1.0 - L / L0;
  }
}

void free_hvp(sk_hvp *h) {
  auto f = [](void *p) {
    if (p) (void)hipFree(p);
  };
  f(h->d_items);
  f(h->d_lambda);
  f(h->d_part);
  f(h->d_coef);
  f(h->X);
  f(h->Y);
  f(h->d_ws_tab);
  f(h->d_user_tab);
  if (h->h_user_tab) (void)hipHostFree(h->h_user_tab);
  if (h->user_ev) (void)hipEventDestroy(h->user_ev);
  for (hipEvent_t e : h->evpool) (void)hipEventDestroy(e);
  h->evpool.clear();
}

}  // namespace

extern "C" {

int sk_hvp_create(const sk_layer_shape *shapes, int32_t n_layers, int32_t rank, const float *lambdas, float shift,
                  uint64_t seed, int64_t max_batch, int32_t device, sk_hvp **out) {
  if (!out) return fail(SK_EINVAL, "out is NULL");
  *out = nullptr;
  if (!shapes || n_layers < 1) return fail(SK_EINVAL, "need at least one layer shape");
  if (n_layers > (1 << 25)) return fail(SK_EINVAL, "too many layers for the stream counter");
  if (rank < 1 || rank > SK_HVP_MAX_RANK) return fail(SK_EINVAL, "rank must be in [1, 32]");
  if (!lambdas) return fail(SK_EINVAL, "lambdas is NULL");
  if (max_batch < 1) return fail(SK_EINVAL, "max_batch must be >= 1");
  for (int l = 0; l < n_layers; ++l)
    if (shapes[l].rows < 1 || shapes[l].cols < 1)
      return fail(SK_EINVAL, "layer " + std::to_string(l) + ": rows and cols must be >= 1");
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || device < 0 || device >= ndev)
    return fail(SK_EINVAL, "device out of range");
  sk_hvp *h = new (std::nothrow) sk_hvp();
  if (!h) return fail(SK_ENOMEM, "host allocation failed");
  h->device = device;
  h->rank = rank;
  h->shift = shift;
  h->seed = seed;
  h->key = make_key(seed);
  h->max_batch = max_batch;
  h->lambdas.assign(lambdas, lambdas + rank);
  for (int l = 0; l < n_layers; ++l) {
    const int64_t n = shapes[l].rows * shapes[l].cols;
    h->off.push_back(h->total);
    h->n.push_back(n);
    h->total += n;
    for (int64_t e0 = 0; e0 < n; e0 += kChunk)
      h->items.push_back(HvpItem{l, (int32_t)std::min<int64_t>(kChunk, n - e0), e0});
  }
  DeviceGuard guard(device);
  auto alloc = [&](void **p, size_t bytes) -> bool {
    if (hipMalloc(p, bytes) != hipSuccess) {
      (void)hipGetLastError();
      return false;
    }
    return true;
  };
  // workspace regions of the layers start on 256-byte boundaries (the sketch kernels see them as
  // caller buffers)
  std::vector<int64_t> woff;
  for (int l = 0; l < n_layers; ++l) {
    woff.push_back(h->ws_floats);
    h->ws_floats += (max_batch * h->n[l] + 63) / 64 * 64;
  }
  const size_t ws = (size_t)h->ws_floats * 4;
  if (!alloc((void **)&h->d_items, sizeof(HvpItem) * h->items.size()) ||
      !alloc((void **)&h->d_lambda, sizeof(float) * rank) ||
      !alloc((void **)&h->d_part, sizeof(float) * h->items.size() * max_batch * rank) ||
      !alloc((void **)&h->d_coef, sizeof(float) * max_batch * rank) || !alloc((void **)&h->X, ws) ||
      !alloc((void **)&h->Y, ws) || !alloc((void **)&h->d_ws_tab, sizeof(HvpLayerPtr) * n_layers) ||
      !alloc((void **)&h->d_user_tab, sizeof(HvpLayerPtr) * n_layers) ||
      hipHostMalloc((void **)&h->h_user_tab, sizeof(HvpLayerPtr) * n_layers) != hipSuccess ||
      hipEventCreateWithFlags(&h->user_ev, hipEventDisableTiming) != hipSuccess) {
    (void)hipGetLastError();
    free_hvp(h);
    delete h;
    return fail(SK_ENOMEM, "hipMalloc failed (workspace of 2 x " + std::to_string(ws) + " bytes)");
  }
  if (hipMemcpy(h->d_items, h->items.data(), sizeof(HvpItem) * h->items.size(), hipMemcpyHostToDevice) !=
          hipSuccess ||
      hipMemcpy(h->d_lambda, h->lambdas.data(), sizeof(float) * rank, hipMemcpyHostToDevice) != hipSuccess) {
    free_hvp(h);
    delete h;
    return fail(SK_EHIP, "hipMemcpy of the item table failed");
  }
  std::vector<HvpLayerPtr> wtab(n_layers);
  for (int l = 0; l < n_layers; ++l) {
    float *xl = h->X + woff[l], *yl = h->Y + woff[l];
    h->xsk.push_back(xl);
    h->ysk.push_back(yl);
    wtab[l] = HvpLayerPtr{xl, yl, h->n[l]};
  }
  if (hipMemcpy(h->d_ws_tab, wtab.data(), sizeof(HvpLayerPtr) * n_layers, hipMemcpyHostToDevice) != hipSuccess) {
    free_hvp(h);
    delete h;
    return fail(SK_EHIP, "hipMemcpy of the workspace table failed");
  }
  *out = h;
  return SK_OK;
}

int sk_hvp_apply(sk_hvp *h, const float *const *x, int64_t batch, float *const *y, void *stream) {
  if (!h || !x || !y) return fail(SK_EINVAL, "NULL argument");
  if (batch < 1 || batch > h->max_batch) return fail(SK_EINVAL, "batch must be in [1, max_batch]");
  for (size_t l = 0; l < h->n.size(); ++l)
    if (!x[l] || !y[l]) return fail(SK_EINVAL, "NULL layer pointer");
  DeviceGuard guard(h->device);
  hipStream_t st = (hipStream_t)stream;
  if (h->user_ev_pending && hipEventSynchronize(h->user_ev) != hipSuccess)
    return fail(SK_EHIP, "hipEventSynchronize failed");
  for (size_t l = 0; l < h->n.size(); ++l) h->h_user_tab[l] = HvpLayerPtr{x[l], y[l], h->n[l]};
  if (hipMemcpyAsync(h->d_user_tab, h->h_user_tab, sizeof(HvpLayerPtr) * h->n.size(), hipMemcpyHostToDevice, st) !=
          hipSuccess ||
      hipEventRecord(h->user_ev, st) != hipSuccess)
    return fail(SK_EHIP, "upload of the layer table failed");
  h->user_ev_pending = true;
  hvp_run(h, h->d_user_tab, batch, st);
  return SK_OK;
}

void sk_hvp_destroy(sk_hvp *h) {
  if (!h) return;
  {
    DeviceGuard guard(h->device);
    (void)hipDeviceSynchronize();
    free_hvp(h);
  }
  delete h;
}

int sketch_hvp(sk_sketch *s, sk_hvp *h, const float *v, int64_t batch, float *out, void *stream) {
  if (!s || !h || !v || !out) return fail(SK_EINVAL, "NULL argument");
  if (batch < 1) return fail(SK_EINVAL, "batch must be >= 1");
  if (s->device != h->device) return fail(SK_EINVAL, "sketch and Hessian live on different devices");
  if (s->layers.size() != h->n.size()) return fail(SK_EINVAL, "sketch and Hessian have different layer lists");
  for (size_t l = 0; l < h->n.size(); ++l)
    if (s->layers[l].n != h->n[l]) return fail(SK_EINVAL, "layer " + std::to_string(l) + " differs in size");
  const int nl = (int)h->n.size();
  DeviceGuard guard(h->device);
  for (int64_t b0 = 0; b0 < batch; b0 += h->max_batch) {
    const int64_t bc = std::min(h->max_batch, batch - b0);
    int rc = sketch_apply_T(s, v + b0 * s->D, bc, h->xsk.data(), SK_F32, nullptr, 0, nl, stream);
    if (rc != SK_OK) return rc;
    hvp_run(h, h->d_ws_tab, bc, (hipStream_t)stream);
    rc = sketch_apply(s, h->ysk.data(), SK_F32, bc, out + b0 * s->D, 0, nl, 0, stream);
    if (rc != SK_OK) return rc;
  }
  return SK_OK;
}

int64_t sketch_arnoldi_work_floats(int64_t D, int32_t k) {
  if (D < 1 || k < 1) return 0;
  return arn_nchunk(D) * (int64_t)(k + 2) + (k + 2) + 4;
}

int sketch_arnoldi_step(float *Q, int64_t D, int32_t j, float *Hbar, int32_t k, float *work, void *stream) {
  if (!Q || !Hbar || !work) return fail(SK_EINVAL, "NULL argument");
  if (D < 1 || k < 1 || j < -1 || j >= k) return fail(SK_EINVAL, "need D >= 1, k >= 1 and -1 <= j < k");
  if (arn_nchunk(D) > 65535) return fail(SK_EUNSUPPORTED, "D too large for the Arnoldi kernels");
  arnoldi_step(Q, D, j, Hbar, k, work, (hipStream_t)stream, nullptr);
  return SK_OK;
}

int sketch_arnoldi(sk_sketch *s, sk_hvp *h, const float *v0, int32_t k, float *Q, float *Hbar, void *stream) {
  if (!s || !h || !v0 || !Q || !Hbar) return fail(SK_EINVAL, "NULL argument");
  if (k < 1) return fail(SK_EINVAL, "k must be >= 1");
  const int64_t D = s->D;
  if (arn_nchunk(D) > 65535) return fail(SK_EUNSUPPORTED, "D too large for the Arnoldi kernels");
  if (sketch_arnoldi_work_floats(D, k) > h->ws_floats)
    return fail(SK_EUNSUPPORTED, "Krylov dimension too large for the Hessian handle's workspace");
  if (s->device != h->device) return fail(SK_EINVAL, "sketch and Hessian live on different devices");
  DeviceGuard guard(h->device);
  hipStream_t st = (hipStream_t)stream;
  if (hipMemcpyAsync(Q, v0, (size_t)D * 4, hipMemcpyDeviceToDevice, st) != hipSuccess)
    return fail(SK_EHIP, "hipMemcpyAsync of v0 failed");
  // the orthogonalisation scratch lives in the Y workspace: the sketch_apply that reads Y has been
  // queued before it on the same stream, and the next sketch_hvp rewrites Y only after the step
  float *work = h->Y;
  arnoldi_step(Q, D, -1, Hbar, k, work, st, h);
  for (int j = 0; j < k; ++j) {
    const int rc = sketch_hvp(s, h, Q + (int64_t)j * D, 1, Q + (int64_t)(j + 1) * D, stream);
    if (rc != SK_OK) return rc;
    arnoldi_step(Q, D, j, Hbar, k, work, st, h);
  }
  return SK_OK;
}

int64_t sketch_id_search_work_floats(int64_t D) { return D < 1 ? 0 : 6 * D + 32; }

int sketch_id_search(sk_sketch *s, sk_hvp *h, const float *const *theta0, int64_t d_min, float tau_target,
                     float delta, int32_t c, int32_t max_rounds, float *work, double *tau_trace, int64_t *d_trace,
                     sk_id_result *res, void *stream) {
  if (!s || !h || !theta0 || !work || !res) return fail(SK_EINVAL, "NULL argument");
  const int64_t D = s->D;
  if (d_min < 1 || d_min > D) return fail(SK_EINVAL, "need 1 <= d_min <= D");
  if (c < 1 || max_rounds < 1) return fail(SK_EINVAL, "need c >= 1 and max_rounds >= 1");
  if (s->device != h->device) return fail(SK_EINVAL, "sketch and Hessian live on different devices");
  if (s->layers.size() != h->n.size()) return fail(SK_EINVAL, "sketch and Hessian have different layer lists");
  for (size_t l = 0; l < h->n.size(); ++l) {
    if (s->layers[l].n != h->n[l]) return fail(SK_EINVAL, "layer " + std::to_string(l) + " differs in size");
    if (!theta0[l]) return fail(SK_EINVAL, "theta0[" + std::to_string(l) + "] is NULL");
  }
  DeviceGuard guard(h->device);
  hipStream_t st = (hipStream_t)stream;
  const int nl = (int)h->n.size();
  float *omega = work, *r = work + D, *p = work + 2 * D, *q = work + 3 * D, *g0 = work + 4 * D, *w = work + 5 * D;
  double *scal = reinterpret_cast<double *>(work + 6 * D);
  // L0 = 1/2 theta0 . H theta0 and g0 = S H theta0 (H theta0 into the Y workspace)
  if (h->user_ev_pending && hipEventSynchronize(h->user_ev) != hipSuccess)
    return fail(SK_EHIP, "hipEventSynchronize failed");
  for (int l = 0; l < nl; ++l)
    h->h_user_tab[l] = HvpLayerPtr{theta0[l], (float *)h->ysk[l], h->n[l]};
  if (hipMemcpyAsync(h->d_user_tab, h->h_user_tab, sizeof(HvpLayerPtr) * nl, hipMemcpyHostToDevice, st) !=
          hipSuccess ||
      hipEventRecord(h->user_ev, st) != hipSuccess)
    return fail(SK_EHIP, "upload of the layer table failed");
  h->user_ev_pending = true;
  hvp_run(h, h->d_user_tab, 1, st);
  hipLaunchKernelGGL(k_tab_dot, dim3((unsigned)h->items.size()), dim3(256), 0, st, h->d_items, h->d_user_tab,
                     h->d_part);
  hipLaunchKernelGGL(k_sum_f64, dim3(1), dim3(256), 0, st, h->d_part, (int64_t)h->items.size(), 0.5,
                     scal + kIdL0);
  int rc = sketch_apply(s, h->ysk.data(), SK_F32, 1, g0, 0, nl, 0, stream);
  if (rc != SK_OK) return rc;
  launch_fill_zero(omega, D, st);
  launch_fill_zero(w, D, st);  // S H S^T omega at omega = 0
  double tau_old = 0.0;
  int64_t d = d_min;
  res->d = 0;
  res->status = 2;
  res->rounds = 0;
  res->L0 = 0.0;
  for (int k = 0; k < max_rounds; ++k) {
    hipLaunchKernelGGL(k_cg_start, dim3(1), dim3(1024), 0, st, g0, w, r, p, d, D, scal);
    for (int i = 0; i < c; ++i) {
      rc = sketch_hvp(s, h, p, 1, q, stream);
      if (rc != SK_OK) return rc;
      hipLaunchKernelGGL(k_cg_step, dim3(1), dim3(1024), 0, st, omega, r, p, q, d, scal);
    }
    rc = sketch_hvp(s, h, omega, 1, w, stream);
    if (rc != SK_OK) return rc;
    hipLaunchKernelGGL(k_id_eval, dim3(1), dim3(1024), 0, st, g0, w, omega, D, scal);
    double hs[4];
    if (hipMemcpyAsync(hs, scal, sizeof(hs), hipMemcpyDeviceToHost, st) != hipSuccess ||
        hipStreamSynchronize(st) != hipSuccess)
      return fail(SK_EHIP, "reading the metric back failed");
    const double tau = hs[kIdTau];
    res->L0 = hs[kIdL0];
    res->rounds = k + 1;
    if (tau_trace) tau_trace[k] = tau;
    if (d_trace) d_trace[k] = d;
    if (tau >= (double)tau_target) {
      res->d = d;
      res->status = 0;
      return SK_OK;
    }
    if (tau - tau_old < (double)delta) {
      d *= 2;
      if (d > D) {
        res->status = 1;
        return SK_OK;
      }
    }
    tau_old = tau;
  }
  return SK_OK;
}

int sk_hvp_profile(sk_hvp *h, uint32_t classes) {
  if (!h) return fail(SK_EINVAL, "handle is NULL");
  if (classes >> SK_HVP_PROF_CLASSES) return fail(SK_EINVAL, "unknown kernel class in profiling mask");
  DeviceGuard guard(h->device);
  if (classes) {
    if (h->evpool.empty()) {
      h->evpool.resize(2 * 8192);
      for (auto &e : h->evpool)
        if (hipEventCreate(&e) != hipSuccess) return fail(SK_EHIP, "hipEventCreate failed");
    }
    h->evnext = 0;
    h->recs.clear();
  }
  h->prof_mask = classes;
  return SK_OK;
}

int sk_hvp_profile_read(sk_hvp *h, double *ms, int64_t *count, int64_t *bytes) {
  if (!h || !ms || !count || !bytes) return fail(SK_EINVAL, "NULL argument");
  DeviceGuard guard(h->device);
  for (int c = 0; c < SK_HVP_PROF_CLASSES; ++c) {
    ms[c] = 0.0;
    count[c] = 0;
    bytes[c] = 0;
  }
  for (const auto &r : h->recs) {
    if (hipEventSynchronize(h->evpool[r.ev + 1]) != hipSuccess) return fail(SK_EHIP, "hipEventSynchronize failed");
    float t = 0.0f;
    if (hipEventElapsedTime(&t, h->evpool[r.ev], h->evpool[r.ev + 1]) != hipSuccess)
      return fail(SK_EHIP, "hipEventElapsedTime failed");
    ms[r.cls] += t;
    count[r.cls] += 1;
    bytes[r.cls] += r.bytes;
  }
  h->recs.clear();
  h->evnext = 0;
  return SK_OK;
}

}  // extern "C"
