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
constexpr int kAffdVB = 4;  // vectors per workgroup in phase A

template <bool BF16>
__global__ __launch_bounds__(256) void k_affd_rows(const LayerDesc *__restrict__ layers,
                                                   const uint16_t *__restrict__ ptab, int layer,
                                                   const void *__restrict__ x, int64_t b_begin, int64_t bc,
                                                   float *__restrict__ w, Key key) {
  __shared__ float s[kAffdVB][1024];
  const LayerDesc &ld = layers[layer];
  const int64_t h = blockIdx.x;
  const int L = ld.L;
  const int col0 = threadIdx.x * 4;
  const int64_t j0 = h * L + col0;
  const int64_t lim = ld.n - j0;
  const int64_t v0 = (int64_t)blockIdx.y * kAffdVB;
  const int nv = (int)((bc - v0) < kAffdVB ? (bc - v0) : kAffdVB);
  uint32_t bits = 0;
  if (lim > 0) bits = sign_word((uint64_t)j0, (uint32_t)ld.layer_id, key) >> (j0 & 31);
  const uint16_t *fk = ptab + ld.poff[0][0][ld.K - 1];
  if (col0 < L) {
    int pc[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) pc[q] = fk[col0 + q];
#pragma unroll
    for (int v = 0; v < kAffdVB; ++v) {
      float val[4] = {0.f, 0.f, 0.f, 0.f};
      if (v < nv && lim > 0) load4<BF16, false>(x, (b_begin + v0 + v) * ld.n + j0, lim, val);
#pragma unroll
      for (int q = 0; q < 4; ++q) s[v][pc[q]] = flip(val[q], (bits >> q) & 1u);
    }
  }
  const int lgL = ld.lgL;
  for (int v = 0; v < nv; ++v) lds_fwht(&s[v][0], lgL, 0);
  const float sc = rsqrtf((float)L);
  const int64_t drow = dst_row(ld, ptab, h);
  for (int e = threadIdx.x; e < nv * L; e += 256) {
    const int v = e >> lgL, c = e & (L - 1);
    w[(v0 + v) * ld.np + drow * L + c] = s[v][c] * sc;
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
constexpr int kAffdCV = 16;  // vectors per workgroup in phase C

template <int TT>
__global__ __launch_bounds__(256) void k_affd_top(const LayerDesc *__restrict__ layers,
                                                  const uint16_t *__restrict__ ptab, int layer,
                                                  const float *__restrict__ w, int64_t bc,
                                                  float *__restrict__ f, Key key) {
  __shared__ float fs[kAffdCV][1024];
  const LayerDesc &ld = layers[layer];
  const int L = ld.L;
  const int64_t lo_len = (int64_t)ld.dk1 * L;
  const int64_t p = blockIdx.x;
  const int64_t v0 = (int64_t)blockIdx.y * kAffdCV;
  const int nv = (int)((bc - v0) < kAffdCV ? (bc - v0) : kAffdCV);
  // live slabs and the fold signs
  uint32_t live_mask_lo = 0, live_mask_hi = 0, sgn_lo = 0, sgn_hi = 0;
  for (int t = 0; t < TT; ++t) {
    const bool live = src_slab(ld, ptab, t) * ld.dk1 < ld.rows_live;
    const uint32_t sg = __popc((uint32_t)t & ld.hstar) & 1u;
    if (t < 32) {
      live_mask_lo |= (uint32_t)live << t;
      sgn_lo |= sg << t;
    } else {
      live_mask_hi |= (uint32_t)live << (t - 32);
      sgn_hi |= sg << (t - 32);
    }
  }
  const float sc = 1.0f / (float)TT;
  for (int cq = 0; cq < L; cq += 256) {
    const int l = cq + threadIdx.x;
    const int64_t q = p * L + l;
    float g[TT];
#pragma unroll
    for (int t = 0; t < TT; ++t) g[t] = gauss((uint64_t)(t * lo_len + q), (uint32_t)ld.layer_id, ST_GAUSS, key);
    for (int v = 0; v < nv; ++v) {
      const float *wv = w + (v0 + v) * ld.np + q;
      float x[TT];
#pragma unroll
      for (int t = 0; t < TT; ++t) {
        const bool live = t < 32 ? (live_mask_lo >> t) & 1u : (live_mask_hi >> (t - 32)) & 1u;
        x[t] = live ? wv[(int64_t)t * lo_len] : 0.0f;
      }
      fwht_regs_t<TT>(x);
      float acc = 0.0f;
#pragma unroll
      for (int t = 0; t < TT; ++t) {
        const uint32_t sg = t < 32 ? (sgn_lo >> t) & 1u : (sgn_hi >> (t - 32)) & 1u;
        acc += flip(g[t] * x[t], sg);
      }
      fs[v][l] = acc * sc;
    }
  }
  for (int v = 0; v < nv; ++v) lds_fwht(&fs[v][0], ld.lgL, 0);
  const float scl = rsqrtf((float)L);
  for (int e = threadIdx.x; e < nv * L; e += 256) {
    const int v = e / L, l = e - (e / L) * L;
    f[(v0 + v) * lo_len + p * L + l] = fs[v][l] * scl;
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

void run_affd_fast(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc,
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
    dim3 grid((unsigned)ld.dk1, (unsigned)((bc + kAffdCV - 1) / kAffdCV));
#define SK_TOP(T)                                                                                             \
  case T:                                                                                                     \
    hipLaunchKernelGGL((k_affd_top<T>), grid, dim3(256), 0, st, s->d_layers, s->d_ptab, layer, w, bc, f, s->key); \
    break;
    switch (TT) {
      SK_TOP(1) SK_TOP(2) SK_TOP(4) SK_TOP(8) SK_TOP(16) SK_TOP(32) SK_TOP(64)
      default: break;
    }
#undef SK_TOP
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
