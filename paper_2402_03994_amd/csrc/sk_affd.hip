// sk_affd.hip -- AFFD (eq. bami) for D > 1024 and at most 64 top-digit values.
//
// Index a padded coordinate of a layer as (t, p, l): l the last Kronecker
// digit (L = 1024 columns), p the second-to-last digit (dk1 rows), t the
// remaining top digits (TT values).  H_N' = H_TT (x) H_dk1 (x) H_L, and the
// coordinates kept by R_D Gather_pi2 are (h*, pi2_p(a), pi2_l(b)) for a < R,
// b < L (D = R L), h* the top digits of pi2 at zero.  Hence
//   AFFD(x)[a L + b] = sqrt(N'/D) (H_dk1 (x) H_L F)[pi2_p(a), pi2_l(b)],
//   F[p, l] = sum_t H_TT[h*, t] g[t, p, l] (H_N' w)[t, p, l],
// with w = Scatter_pi1(B x).  Phases (each a kernel, all in fp32):
//   A  rows:  load a source row, sign, pi1 on its columns, H_L  -> W[t,p,:]
//   B  cols:  H_dk1 along p for every live slab t               -> W
//   C  top:   H_TT along t, times g, signed sum onto h*, then H_L -> F
//   D  cols:  H_dk1 along p, keep rows pi2_p(a), a < R          -> G[a,:]
//   E  out:   out[a L + b] (+)= sqrt(N'/D) G[a, pi2_l(b)]
// Rows of W that no source row reaches are never written; B and C treat them
// as zero from the same liveness test (source row < ceil(n / L)).
#include <cstdlib>

#include "sk_kcommon.h"
#include "sk_launch.h"

namespace sk {

namespace {

// Source slab of destination slab t (inverse pi1 over the top digits 0..K-3).
__device__ __forceinline__ int64_t src_slab(const LayerDesc &ld, const uint16_t *ptab, int64_t t) {
  int64_t s = 0, stride = 1;
  for (int k = ld.K - 3; k >= 0; --k) {
    const int64_t dig = (t / stride) & ((1ll << ld.lg[k]) - 1);
    s += (int64_t)ptab[ld.poff[0][1][k] + dig] * stride;
    stride <<= ld.lg[k];
  }
  return s;
}

// Destination row (t, p) of source row h (pi1 over digits 0..K-2).
__device__ __forceinline__ int64_t dst_row(const LayerDesc &ld, const uint16_t *ptab, int64_t h) {
  int64_t r = 0, stride = 1;
  for (int k = ld.K - 2; k >= 0; --k) {
    const int64_t dig = (h / stride) & ((1ll << ld.lg[k]) - 1);
    r += (int64_t)ptab[ld.poff[0][0][k] + dig] * stride;
    stride <<= ld.lg[k];
  }
  return r;
}

}  // namespace

// ---- phase A -------------------------------------------------------------
constexpr int kAffdVB = 8;  // vectors per workgroup in phase A

template <bool BF16>
__global__ __launch_bounds__(256) void k_affd_rows(const LayerDesc *__restrict__ layers,
                                                   const uint16_t *__restrict__ ptab, int layer,
                                                   const void *__restrict__ x, int64_t b_begin, int64_t bc,
                                                   float *__restrict__ w, Key key) {
  __shared__ __align__(16) float s[kAffdVB * 1024];
  const LayerDesc &ld = layers[layer];
  const int64_t h = blockIdx.x;
  const int col0 = threadIdx.x * 4;  // L == 1024 on this path
  const int64_t j0 = h * 1024 + col0;
  const int64_t lim = ld.n - j0;
  const int64_t v0 = (int64_t)blockIdx.y * kAffdVB;
  const int nv = (int)((bc - v0) < kAffdVB ? (bc - v0) : kAffdVB);
  uint32_t bits = 0;
  if (lim > 0) bits = sign_word((uint64_t)j0, (uint32_t)ld.layer_id, key) >> (j0 & 31);
  const uint16_t *fk = ptab + ld.poff[0][0][ld.K - 1];
  int pc[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) pc[q] = fk[col0 + q];
  // load, sign, scatter the columns through pi1 of the last digit
#pragma unroll
  for (int v = 0; v < kAffdVB; ++v) {
    float val[4] = {0.f, 0.f, 0.f, 0.f};
    if (v < nv && lim > 0) load4<BF16, false>(x, (b_begin + v0 + v) * ld.n + j0, lim, val);
#pragma unroll
    for (int q = 0; q < 4; ++q) s[v * 1024 + pc[q]] = flip(val[q], (bits >> q) & 1u);
  }
  __syncthreads();
  float r[kAffdVB][4];
#pragma unroll
  for (int v = 0; v < kAffdVB; ++v) {
    const float4 t = *(const float4 *)(s + v * 1024 + col0);
    r[v][0] = t.x;
    r[v][1] = t.y;
    r[v][2] = t.z;
    r[v][3] = t.w;
  }
  fwht1024_rows<kAffdVB>(r, s);
  const float sc = 1.0f / 32.0f;  // 1024^{-1/2}
  const int64_t drow = dst_row(ld, ptab, h);
#pragma unroll
  for (int v = 0; v < kAffdVB; ++v) {
    if (v < nv) {
      float *dst = w + (v0 + v) * ld.np + drow * 1024 + threadIdx.x;
#pragma unroll
      for (int k = 0; k < 4; ++k) dst[256 * k] = r[v][k] * sc;
    }
  }
}

// ---- phases B and D: transform along p for a 16-column block -------------
// mode 0 (B): W in place; mode 1 (D): F -> G keeping rows pi2_p(a), a < R.
template <int LGD, int MODE>
__global__ __launch_bounds__(256) void k_affd_cols(const LayerDesc *__restrict__ layers,
                                                   const uint16_t *__restrict__ ptab, int layer, float *__restrict__ w,
                                                   int64_t vstride, int R, float *__restrict__ g_out) {
  constexpr int DK = 1 << LGD;
  constexpr int K1 = DK >= 16 ? DK / 16 : 1;  // rows per thread, first layout
  extern __shared__ float s[];                // DK x 16
  const LayerDesc &ld = layers[layer];
  const int L = ld.L;
  const int ncb = L / 16;
  const int64_t blk = blockIdx.x;
  const int cb = (int)(blk % ncb);
  const int64_t t = blk / ncb;       // slab (mode 0) or 0
  const int64_t v = blockIdx.y;
  const int c = threadIdx.x & 15, g = threadIdx.x >> 4;
  float *base = w + v * vstride + (t * DK) * L + cb * 16 + c;
  bool slab_live = true;
  int64_t src0 = 0;
  if (MODE == 0) {
    src0 = src_slab(ld, ptab, t) * DK;
    slab_live = src0 < ld.rows_live;
  }
  if (!slab_live) return;  // all-zero slab: phase C skips it too
  const uint16_t *invp = ptab + ld.poff[0][1][ld.K - 2];
  float r1[K1];
  if (g < DK) {
#pragma unroll
    for (int k = 0; k < K1; ++k) {
      const int r = g + 16 * k;
      bool live = true;
      if (MODE == 0) live = src0 + invp[r] < ld.rows_live;
      r1[k] = live ? base[(int64_t)r * L] : 0.0f;
    }
    fwht_regs_t<K1>(r1);
#pragma unroll
    for (int k = 0; k < K1; ++k) s[(g + 16 * k) * 16 + c] = r1[k];
  }
  __syncthreads();
  // second layout: 16 consecutive rows of one column, DK/16 groups of 16 columns
  constexpr int JR = DK >= 16 ? 16 : DK;
  constexpr int NG = DK / JR * 16;  // (row block, column) groups
  const float sc = rsqrtf((float)DK);
  for (int gi = threadIdx.x; gi < NG; gi += 256) {
    const int cc = gi & 15, rb = gi >> 4;
    float r2[JR];
#pragma unroll
    for (int j = 0; j < JR; ++j) r2[j] = s[(rb * JR + j) * 16 + cc];
    fwht_regs_t<JR>(r2);
    if (MODE == 0) {
      float *o = w + v * vstride + (t * DK) * L + cb * 16 + cc;
#pragma unroll
      for (int j = 0; j < JR; ++j) o[(int64_t)(rb * JR + j) * L] = r2[j] * sc;
    } else {
#pragma unroll
      for (int j = 0; j < JR; ++j) s[(rb * JR + j) * 16 + cc] = r2[j] * sc;
    }
  }
  if (MODE == 1) {
    __syncthreads();
    const uint16_t *p2 = ptab + ld.poff[1][0][ld.K - 2];
    for (int e = threadIdx.x; e < R * 16; e += 256) {
      const int a = e >> 4, cc = e & 15;
      g_out[(v * R + a) * L + cb * 16 + cc] = s[p2[a] * 16 + cc];
    }
  }
}

// ---- phase C -------------------------------------------------------------
// Live-slab mask and fold signs (-1)^{<h*, t>} of the top index t.
__device__ __forceinline__ void top_masks(const LayerDesc &ld, const uint16_t *ptab, int tt, uint64_t &live,
                                          uint64_t &sgn) {
  live = 0;
  sgn = 0;
  for (int t = 0; t < tt; ++t) {
    if (src_slab(ld, ptab, t) * ld.dk1 < ld.rows_live) live |= 1ull << t;
    sgn |= (uint64_t)(__popc((uint32_t)t & ld.hstar) & 1u) << t;
  }
}

// TT <= 16: thread owns 4 consecutive columns (one Philox block per 4
// Gaussians); F rows of CV vectors are transformed by fwht1024_rows.
template <int TT, int CV>
__global__ __launch_bounds__(256) void k_affd_top(const LayerDesc *__restrict__ layers,
                                                  const uint16_t *__restrict__ ptab, int layer,
                                                  const float *__restrict__ w, int64_t bc, float *__restrict__ f,
                                                  Key key) {
  __shared__ __align__(16) float lds[CV * 1024];
  const LayerDesc &ld = layers[layer];
  const int64_t lo_len = (int64_t)ld.dk1 * 1024;
  const int64_t p = blockIdx.x;
  const int64_t v0 = (int64_t)blockIdx.y * CV;
  const int nv = (int)((bc - v0) < CV ? (bc - v0) : CV);
  uint64_t live, sgn;
  top_masks(ld, ptab, TT, live, sgn);
  const int64_t q = p * 1024 + 4 * threadIdx.x;
  float g[TT][4];
#pragma unroll
  for (int t = 0; t < TT; ++t) gauss4((uint64_t)(t * lo_len + q) >> 2, (uint32_t)ld.layer_id, ST_GAUSS, key, g[t]);
#pragma unroll 1
  for (int v = 0; v < CV; ++v) {
    float x[4][TT];
    const float *wv = w + (v0 + (v < nv ? v : 0)) * ld.np + q;
#pragma unroll
    for (int t = 0; t < TT; ++t) {
      float4 val = make_float4(0.f, 0.f, 0.f, 0.f);
      if (v < nv && ((live >> t) & 1ull)) val = *(const float4 *)(wv + (int64_t)t * lo_len);
      x[0][t] = val.x;
      x[1][t] = val.y;
      x[2][t] = val.z;
      x[3][t] = val.w;
    }
    float o[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      fwht_regs_t<TT>(x[c]);
      float acc = 0.0f;
#pragma unroll
      for (int t = 0; t < TT; ++t) acc += flip(g[t][c] * x[c][t], (uint32_t)(sgn >> t) & 1u);
      o[c] = acc;
    }
    *(float4 *)(lds + v * 1024 + 4 * threadIdx.x) = make_float4(o[0], o[1], o[2], o[3]);
  }
  float F[CV][4];
#pragma unroll
  for (int v = 0; v < CV; ++v) {
    const float4 t4 = *(const float4 *)(lds + v * 1024 + 4 * threadIdx.x);
    F[v][0] = t4.x;
    F[v][1] = t4.y;
    F[v][2] = t4.z;
    F[v][3] = t4.w;
  }
  fwht1024_rows<CV>(F, lds);
  const float sc = 1.0f / (32.0f * (float)TT);  // H_TT twice (1/TT) and H_L (1024^{-1/2})
#pragma unroll
  for (int v = 0; v < CV; ++v) {
    if (v < nv) {
      float *dst = f + (v0 + v) * lo_len + p * 1024 + threadIdx.x;
#pragma unroll
      for (int k = 0; k < 4; ++k) dst[256 * k] = F[v][k] * sc;
    }
  }
}

// TT in {32, 64}: thread owns one column per pass (TT Gaussians in registers).
template <int TT, int CV>
__global__ __launch_bounds__(256) void k_affd_top_wide(const LayerDesc *__restrict__ layers,
                                                       const uint16_t *__restrict__ ptab, int layer,
                                                       const float *__restrict__ w, int64_t bc,
                                                       float *__restrict__ f, Key key) {
  __shared__ __align__(16) float lds[CV * 1024];
  const LayerDesc &ld = layers[layer];
  const int64_t lo_len = (int64_t)ld.dk1 * 1024;
  const int64_t p = blockIdx.x;
  const int64_t v0 = (int64_t)blockIdx.y * CV;
  const int nv = (int)((bc - v0) < CV ? (bc - v0) : CV);
  uint64_t live, sgn;
  top_masks(ld, ptab, TT, live, sgn);
  for (int cq = 0; cq < 1024; cq += 256) {
    const int l = cq + threadIdx.x;
    const int64_t q = p * 1024 + l;
    float g[TT];
#pragma clang loop unroll(full)
    for (int t = 0; t < TT; ++t) g[t] = gauss((uint64_t)(t * lo_len + q), (uint32_t)ld.layer_id, ST_GAUSS, key);
#pragma unroll 1
    for (int v = 0; v < CV; ++v) {
      float acc = 0.0f;
      if (v < nv) {
        const float *wv = w + (v0 + v) * ld.np + q;
        float x[TT];
#pragma unroll
        for (int t = 0; t < TT; ++t) x[t] = ((live >> t) & 1ull) ? wv[(int64_t)t * lo_len] : 0.0f;
        fwht_regs_t<TT>(x);
#pragma unroll
        for (int t = 0; t < TT; ++t) acc += flip(g[t] * x[t], (uint32_t)(sgn >> t) & 1u);
      }
      lds[v * 1024 + l] = acc;
    }
  }
  __syncthreads();
  float F[CV][4];
#pragma unroll
  for (int v = 0; v < CV; ++v) {
    const float4 t = *(const float4 *)(lds + v * 1024 + 4 * threadIdx.x);
    F[v][0] = t.x;
    F[v][1] = t.y;
    F[v][2] = t.z;
    F[v][3] = t.w;
  }
  fwht1024_rows<CV>(F, lds);
  const float sc = 1.0f / (32.0f * (float)TT);
#pragma unroll
  for (int v = 0; v < CV; ++v) {
    if (v < nv) {
      float *dst = f + (v0 + v) * lo_len + p * 1024 + threadIdx.x;
#pragma unroll
      for (int k = 0; k < 4; ++k) dst[256 * k] = F[v][k] * sc;
    }
  }
}

// ---- phase E -------------------------------------------------------------
__global__ void k_affd_out(const LayerDesc *__restrict__ layers, const uint16_t *__restrict__ ptab, int layer,
                           const float *__restrict__ g_in, int R, int64_t D, int64_t b_begin,
                           float *__restrict__ out, int accumulate) {
  const LayerDesc &ld = layers[layer];
  const int64_t c = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (c >= D) return;
  const int64_t v = blockIdx.y;
  const int L = ld.L;
  const int64_t a = c / L, b = c - (c / L) * L;
  const float sc = (float)sqrt((double)ld.np / (double)D);
  const float val = sc * g_in[(v * R + a) * L + ptab[ld.poff[1][0][ld.K - 1] + b]];
  float *o = out + (b_begin + v) * D + c;
  *o = accumulate ? *o + val : val;
}

bool affd_fast_path(const sk_sketch *s, int layer) {
  const LayerDesc &ld = s->layers[layer];
  if (s->D <= 1024 || ld.K < 2 || ld.L != 1024) return false;
  const int lgtt = ld.lgnp - ld.lgdk1 - ld.lgL;
  return lgtt >= 0 && lgtt <= 6 && ld.lgdk1 >= 1;
}

int64_t affd_fast_bytes_per_vector(const sk_sketch *s, int layer) {
  const LayerDesc &ld = s->layers[layer];
  const int64_t lo_len = (int64_t)ld.dk1 * ld.L;
  return (ld.np + lo_len + s->D) * 4;
}

// Bytes of intermediate W one vector of the layer touches (live slabs only).
int64_t affd_live_bytes_per_vector(const sk_sketch *s, int layer) {
  const LayerDesc &ld = s->layers[layer];
  const int64_t slab = (int64_t)ld.dk1 * ld.L;
  const int64_t live_rows = ((ld.rows_live + ld.dk1 - 1) / ld.dk1) * ld.dk1;
  return (live_rows * ld.L + slab + s->D) * 4;
}

// Target footprint of one batch tile.  Large tiles amortise the Gaussian
// stream (regenerated once per tile) over many vectors.
int64_t affd_tile_bytes() {
  const char *e = std::getenv("SK_AFFD_TILE_MB");
  const int64_t mb = e ? std::atoll(e) : 4096;
  return (mb < 1 ? 1 : mb) << 20;
}

void run_affd_fast(const sk_sketch *s, int layer, const void *x, int dtype, bool vec, int64_t b_begin, int64_t bc,
                   float *out, bool accumulate, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const int64_t lo_len = (int64_t)ld.dk1 * ld.L;
  float *w = s->ws;
  float *f = w + bc * ld.np;
  float *gbuf = f + bc * lo_len;
  const int R = (int)(s->D / ld.L);
  const int lgtt = ld.lgnp - ld.lgdk1 - ld.lgL;
  const int TT = 1 << lgtt;
  // A
  {
    dim3 grid((unsigned)ld.rows_live, (unsigned)((bc + kAffdVB - 1) / kAffdVB));
    if (dtype == SK_BF16)
      hipLaunchKernelGGL(k_affd_rows<true>, grid, dim3(256), 0, st, s->d_layers, s->d_ptab, layer, x, b_begin, bc, w,
                         s->key);
    else
      hipLaunchKernelGGL(k_affd_rows<false>, grid, dim3(256), 0, st, s->d_layers, s->d_ptab, layer, x, b_begin, bc, w,
                         s->key);
  }
  // B (and D) launch helper
  auto cols = [&](int mode, float *buf, int64_t vstride, int64_t nslab) {
    dim3 grid((unsigned)(nslab * (ld.L / 16)), (unsigned)bc);
    const size_t shm = sizeof(float) * 16 * ld.dk1;
#define SK_COLS(LG)                                                                                          \
  case LG:                                                                                                   \
    if (mode == 0)                                                                                           \
      hipLaunchKernelGGL((k_affd_cols<LG, 0>), grid, dim3(256), shm, st, s->d_layers, s->d_ptab, layer, buf,  \
                         vstride, R, gbuf);                                                                  \
    else                                                                                                     \
      hipLaunchKernelGGL((k_affd_cols<LG, 1>), grid, dim3(256), shm, st, s->d_layers, s->d_ptab, layer, buf,  \
                         vstride, R, gbuf);                                                                  \
    break;
    switch (ld.lgdk1) {
      SK_COLS(1) SK_COLS(2) SK_COLS(3) SK_COLS(4) SK_COLS(5) SK_COLS(6) SK_COLS(7) SK_COLS(8) SK_COLS(9) SK_COLS(10)
      default: break;
    }
#undef SK_COLS
  };
  cols(0, w, ld.np, TT);
  // C
  {
#define SK_TOP(T, CV)                                                                                        \
  case T:                                                                                                    \
    hipLaunchKernelGGL((k_affd_top<T, CV>), dim3((unsigned)ld.dk1, (unsigned)((bc + CV - 1) / CV)), dim3(256), 0, \
                       st, s->d_layers, s->d_ptab, layer, w, bc, f, s->key);                                 \
    break;
#define SK_TOPW(T, CV)                                                                                       \
  case T:                                                                                                    \
    hipLaunchKernelGGL((k_affd_top_wide<T, CV>), dim3((unsigned)ld.dk1, (unsigned)((bc + CV - 1) / CV)),     \
                       dim3(256), 0, st, s->d_layers, s->d_ptab, layer, w, bc, f, s->key);                   \
    break;
    switch (TT) {
      SK_TOP(1, 16) SK_TOP(2, 16) SK_TOP(4, 16) SK_TOP(8, 16) SK_TOP(16, 16) SK_TOPW(32, 16) SK_TOPW(64, 8)
      default: break;
    }
#undef SK_TOP
#undef SK_TOPW
  }
  // D
  cols(1, f, lo_len, 1);
  // E
  {
    dim3 grid((unsigned)((s->D + 255) / 256), (unsigned)bc);
    hipLaunchKernelGGL(k_affd_out, grid, dim3(256), 0, st, s->d_layers, s->d_ptab, layer, gbuf, R, s->D, b_begin,
                       out, (int)accumulate);
  }
  (void)hipGetLastError();
}

}  // namespace sk
