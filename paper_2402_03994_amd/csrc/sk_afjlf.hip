// sk_afjlf.hip -- AFJLF: eq. frikadel with the Walsh-Hadamard pre-conditioner
// replaced by the FFT (Sec. 3, "Alternative pre-conditioners"; Table
// tab:gains_design_choices, rows H_N -> FFT):
//
//   y = sqrt(N/D) G R_D F_N B pad(x)
//
// with F_N the real orthonormal Fourier matrix whose rows are 1/sqrt(N),
// (-1)^n/sqrt(N) and then, per frequency k = 1 .. N/2 - 1, the pair
// sqrt(2/N) (cos, -sin)(2 pi k n / N).  R_D keeps the first D rows, i.e. the
// DFT values X_0 .. X_{M-1} (M = D/2) and X_{N/2}:
//   y_0 = g_0 X_0 / sqrt(D),  y_1 = g_1 X_{N/2} / sqrt(D),
//   y_{2k} = sqrt(2/D) g_{2k} Re X_k,  y_{2k+1} = sqrt(2/D) g_{2k+1} Im X_k.
//
// Only M of the N DFT values are needed.  With the layer viewed as P rows of
// R (n = t R + b; R >= M, P = N/R <= 256 so that a row piece is at least 512
// bytes), Q = N/M, J = M/P and k = r + P j (r < P, j < J), b = q + Q s:
//   u_r[b]      = sum_t x[t][b] w_P^{t r}                          (pass 1)
//   X_{r + P j} = sum_q w_N^{q r} w_R^{q j} W_q[j],                 (pass 2)
//   W_q         = FFT_J over s of u_r[q + Q s] w_M^{s r},   q < Q, s < J
// (w_L = exp(-2 pi i / L)).  Pass 1 reads the signed input once and writes u
// for r <= P/2 (u_{P-r} = conj(u_r)); pass 2 gives the residues r and P - r
// from one J-point transform per column q:
//   X_{(P-r) + P (J-1-j)} = sum_q conj(w_N^{q r} w_R^{q j} W_q[j]) w_Q^{q}.
// Layers with N = D and at most 16384 live entries take one kernel instead
// (k = c + (N/L) e: N/L transforms of L >= n points of the twiddled input).
// The transpose runs the same passes backwards.  All transforms are the LDS
// Stockham FFTs of sk_fft.h (their twiddles from a table made in double
// precision at creation); the per-element twiddles of pass 2 run as short
// recurrences from values computed with sincospif.  Every thread issues all
// its global loads of a block before it uses the first (in-order memory
// counters would otherwise serialise them), and the forward residue pass
// loads the next column block during the current block's transform.
#include <algorithm>
#include <cmath>
#include <functional>
#include <vector>

#include "sk_fft.h"
#include "sk_kcommon.h"
#include "sk_launch.h"

namespace sk {

namespace {

// Kernels come in two sizes: 512 threads with an 8192-value transform buffer
// (64 KB of LDS: two workgroups per CU, so one's loads overlap the other's
// transforms) and, for transforms longer than 8192 points, 1024 threads with
// 16384 values.
constexpr int kCap = 16384;      // largest transform buffer (complex values)
constexpr int kLgCap = 14;
constexpr int kLgCapS = 13;      // the default size
constexpr int kLgPMax = 8;       // rows of the pass-1 view: P = N/R <= 256
constexpr int kSlots = 32;       // layers per launch
// Residue-pass transforms of at most 2^kLgTwl points read their twiddles from
// a copy of the table in LDS: they then issue no global loads, so the loads of
// the next column block stay in flight across the transform.
constexpr int kLgTwl = 10;
constexpr int kRAcc = 2;         // residue pass: rows per thread whose sums stay in registers
constexpr int kLgTwSplit = 9;    // two-level twiddle tables of the one-kernel layers: 2 x 512 entries
constexpr int kLgRows = 13;      // forward pass 1: transform buffer of 2^kLgRows values, 2^(kLgRows-4) threads

struct FfLayers {
  int32_t n;                     // layers in this launch
  int32_t layer[kSlots];         // index into the layer table
  int64_t item0[kSlots + 1];     // first work item of each layer (+ total)
  const void *x[kSlots];         // forward: the layer's input; transpose: its output ([batch, n])
  float *u[kSlots];              // pass buffer of the layer, vector 0 of the tile
  int64_t us[kSlots];            // floats per vector of that buffer
  float *y[kSlots];              // forward: the layer's contribution, vector 0 of the tile ([tile][D])
  const float *th[kSlots];       // transpose: theta0 or null
};

__device__ __forceinline__ int find_slot(const FfLayers &g, int64_t item) {
  int s = 0;
  while (s + 1 < g.n && g.item0[s + 1] <= item) ++s;
  return s;
}

// Linear workgroup id -> (item, vector) with every item of vector v on XCD v % 8.
__device__ __forceinline__ bool xcd_decode(int64_t nitems, int64_t bc, int64_t &item, int64_t &v) {
  const int64_t L = blockIdx.x;
  const int64_t rest = L >> 3;
  item = rest % nitems;
  v = (rest / nitems) * 8 + (L & 7);
  return v < bc;
}

__device__ __forceinline__ float load_x(const void *x, int dtype, int64_t j) {
  if (dtype == SK_BF16) return __uint_as_float((uint32_t)((const uint16_t *)x)[j] << 16);
  return ((const float *)x)[j];
}

__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ void store_out(void *o, int dtype, int64_t j, float v) {
  if (dtype == SK_BF16)
    ((uint16_t *)o)[j] = f2bf(v);
  else
    ((float *)o)[j] = v;
}

// Geometry of a two-pass layer (all log2): N = N', M = D/2, P rows of R,
// Q = N/M columns q, J = M/P outputs per residue; pass 1 column blocks of W.
struct FfGeom {
  int lgN, lgM, lgP, lgR, lgQ, lgJ, lgW;
};
__device__ __host__ __forceinline__ FfGeom ff_geom(int lgnp, int lgD, int lgcap = kLgCapS) {
  FfGeom g;
  g.lgN = lgnp;
  g.lgM = lgD - 1;
  g.lgQ = lgnp - g.lgM;
  g.lgP = g.lgQ < kLgPMax ? g.lgQ : kLgPMax;
  g.lgR = lgnp - g.lgP;
  g.lgJ = g.lgM - g.lgP;
  const int w = lgcap + 1 - g.lgP;  // P * W <= 2 * (buffer size) real values
  g.lgW = std::min(std::min(10, w), g.lgR);
  return g;
}

// exp(-2 pi i m / 2^lgL) for 0 <= m < 2^lgL
__device__ __forceinline__ float2 cis_neg(int64_t m, int lgL) {
  float s, c;
  sincospif(ldexpf(-2.0f * (float)m, -lgL), &s, &c);
  return make_float2(c, s);
}

// Sign words of rows t < rows, columns [b0, b0 + 2^lgW) of the P x R view
// into sw[t * nw + w] (nw = W / 32; W >= 128).
// One Philox block holds the sign words of 128 consecutive coordinates: each
// block is generated once and its words of [b0, b0 + W) are written (row
// starts t R are multiples of 128, b0 a multiple of W >= 32).
template <int NT>
__device__ __forceinline__ void build_row_signs(uint32_t *sw, int64_t rows, int lgR, int64_t b0, int lgW,
                                                uint32_t layer, Key key) {
  const int nw = 1 << (lgW - 5);
  const int w0 = (int)((b0 >> 5) & 3);                   // word of b0 in its block
  const int nblk = (w0 + nw + 3) >> 2;                   // blocks per row
  for (int64_t e = threadIdx.x; e < rows * nblk; e += NT) {
    const int64_t t = e / nblk;
    const int bk = (int)(e - t * nblk);
    const W4 q = philox((uint64_t)(((t << lgR) + b0) >> 7) + bk, layer, ST_SIGN, key);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int w = 4 * bk + k - w0;  // word index within the row piece
      if (w >= 0 && w < nw) sw[t * nw + w] = q.w[k];
    }
  }
}

__device__ __forceinline__ uint32_t row_sign_bit(const uint32_t *sw, int64_t t, int nw, int lgR, int64_t b0,
                                                 int64_t j) {
  return (sw[t * nw + ((j - (t << lgR) - b0) >> 5)] >> (j & 31)) & 1u;
}

// ---------------------------------------------------------------------------
// Pass 1, forward: u_r[b] = sum_t B x [t][b] w_P^{t r}, r <= P/2, for one
// column block of W; two real columns per complex transform column.
// ---------------------------------------------------------------------------
template <int LGNT, int LGCAP>
__global__ __launch_bounds__(1 << LGNT) void k_ffr_fwd(const LayerDesc *__restrict__ layers, FfLayers g, int dtype,
                                                 int lgD, int64_t b_begin, int64_t bc,
                                                 const float2 *__restrict__ tw, int lgS, Key key) {
  constexpr int NT = 1 << LGNT, CAP = 1 << LGCAP, MAXE = CAP / NT;
  __shared__ float2 buf[CAP];
  __shared__ uint32_t sw[CAP / 16];  // rows * W / 32 <= CAP / 16
  int64_t item, v;
  if (!xcd_decode(g.item0[g.n], bc, item, v)) return;
  const int slot = find_slot(g, item);
  const LayerDesc &ld = layers[g.layer[slot]];
  const FfGeom fg = ff_geom(ld.lgnp, lgD, LGCAP);
  const int lgR = fg.lgR, lgP = fg.lgP, lgW = fg.lgW, lgWc = lgW - 1;
  const int64_t R = 1ll << lgR, n = ld.n;
  const int64_t b0 = (item - g.item0[slot]) << lgW;
  const int64_t rows = std::min<int64_t>((n + R - 1) >> lgR, 1ll << lgP);
  const int nw = 1 << (lgW - 5);
  const int64_t xo = (b_begin + v) * n;
  // four real columns (two complex ones) per element, at most CAP / (2 NT) elements per thread; every
  // 16-byte (fp32) or 8-byte (bf16) load of the thread is issued before the first one is used
  constexpr int MAXL = CAP / (2 * NT);
  const int lgW4 = lgW - 2;
  const int total = 1 << (lgP + lgW4);
  const bool vec = dtype == SK_BF16 ? !(((uintptr_t)g.x[slot] + 2 * xo) & 7) : !(((uintptr_t)g.x[slot] + 4 * xo) & 15);
  uint4 raw[MAXL];
  uint32_t full = 0;
#pragma unroll
  for (int i = 0; i < MAXL; ++i) {
    const int e = threadIdx.x + i * NT;
    const int64_t t = e >> lgW4;
    const int64_t j = (t << lgR) + b0 + 4 * (e & ((1 << lgW4) - 1));
    raw[i] = make_uint4(0u, 0u, 0u, 0u);
    if (vec && e < total && t < rows && j + 3 < n) full |= 1u << i;
  }
  // one loop per dtype, so that no load result is merged with another before the last load is issued
  if (dtype == SK_BF16) {
    const uint16_t *xb = (const uint16_t *)g.x[slot] + xo + b0;
#pragma unroll
    for (int i = 0; i < MAXL; ++i) {
      const int e = threadIdx.x + i * NT;
      if ((full >> i) & 1u) {
        const uint2 w2 = *(const uint2 *)(xb + ((int64_t)(e >> lgW4) << lgR) + 4 * (e & ((1 << lgW4) - 1)));
        raw[i].x = w2.x;
        raw[i].y = w2.y;
      }
    }
  } else {
    const float *xf = (const float *)g.x[slot] + xo + b0;
#pragma unroll
    for (int i = 0; i < MAXL; ++i) {
      const int e = threadIdx.x + i * NT;
      if ((full >> i) & 1u)
        raw[i] = *(const uint4 *)(xf + ((int64_t)(e >> lgW4) << lgR) + 4 * (e & ((1 << lgW4) - 1)));
    }
  }
  // the block's sign words while the loads are in flight
  build_row_signs<NT>(sw, rows, lgR, b0, lgW, (uint32_t)ld.layer_id, key);
  __syncthreads();
#pragma unroll
  for (int i = 0; i < MAXL; ++i) {
    const int e = threadIdx.x + i * NT;
    if (e >= total) break;
    const int64_t t = e >> lgW4;
    const int c4 = e & ((1 << lgW4) - 1);
    float a[4] = {0.f, 0.f, 0.f, 0.f};
    if (t < rows) {
      if ((full >> i) & 1u) {
        if (dtype == SK_BF16) {
          a[0] = __uint_as_float(raw[i].x << 16);
          a[1] = __uint_as_float(raw[i].x & 0xFFFF0000u);
          a[2] = __uint_as_float(raw[i].y << 16);
          a[3] = __uint_as_float(raw[i].y & 0xFFFF0000u);
        } else {
          a[0] = __uint_as_float(raw[i].x);
          a[1] = __uint_as_float(raw[i].y);
          a[2] = __uint_as_float(raw[i].z);
          a[3] = __uint_as_float(raw[i].w);
        }
      } else {  // the layer's tail, or an input without 16-byte alignment
        const int64_t j = (t << lgR) + b0 + 4 * c4;
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if (j + k < n) a[k] = load_x(g.x[slot], dtype, xo + j + k);
      }
      const uint32_t wd = sw[t * nw + (((b0 + 4 * c4) >> 5) - (b0 >> 5))] >> ((b0 + 4 * c4) & 31);
#pragma unroll
      for (int k = 0; k < 4; ++k) a[k] = flip(a[k], (wd >> k) & 1u);
    }
    buf[(t << lgWc) + 2 * c4] = make_float2(a[0], a[1]);
    buf[(t << lgWc) + 2 * c4 + 1] = make_float2(a[2], a[3]);
  }
  lds_fft<false, NT, MAXE, false, true>(buf, lgP, lgWc, tw, lgS);
  // split the two real columns and write r = 0 .. P/2
  float *u = g.u[slot] + v * g.us[slot];
  const int P = 1 << lgP;
  const int tot2 = (P / 2 + 1) << lgWc;
  for (int e = threadIdx.x; e < tot2; e += NT) {
    const int r = e >> lgWc, c = e & ((1 << lgWc) - 1);
    const float2 zr = buf[(r << lgWc) + c];
    const float2 zm = buf[(((P - r) & (P - 1)) << lgWc) + c];
    const float4 o = make_float4(0.5f * (zr.x + zm.x), 0.5f * (zr.y - zm.y),   // (Z_r + conj Z_{P-r}) / 2
                                 0.5f * (zr.y + zm.y), 0.5f * (zm.x - zr.x));  // -i (Z_r - conj Z_{P-r}) / 2
    *(float4 *)(u + (((int64_t)r << lgR) + b0 + 2 * c) * 2) = o;
  }
}

// ---------------------------------------------------------------------------
// Pass 2, forward: for residue r (and P - r) of one layer and vector, the J
// outputs X_{r + P j} (and X_{(P-r) + P (J-1-j)}), scaled by G into y.
// ---------------------------------------------------------------------------
template <int LGNT, int LGCAP>
__global__ __launch_bounds__(1 << LGNT, 4) void k_ffq_fwd(const LayerDesc *__restrict__ layers, FfLayers g, int lgD,
                                                 int64_t bc, const float *__restrict__ gtab, float c1, float c2,
                                                 const float2 *__restrict__ tw, int lgS) {
  constexpr int NT = 1 << LGNT, CAP = 1 << LGCAP, MAXE = CAP / NT;
  __shared__ float2 buf[CAP];
  __shared__ float2 twl[1 << kLgTwl];
  int64_t item, v;
  if (!xcd_decode(g.item0[g.n], bc, item, v)) return;
  const int slot = find_slot(g, item);
  const LayerDesc &ld = layers[g.layer[slot]];
  const FfGeom fg = ff_geom(ld.lgnp, lgD);
  const int lgM = fg.lgM, lgP = fg.lgP, lgJ = fg.lgJ, lgQ = fg.lgQ, lgR = fg.lgR, lgN = fg.lgN;
  const int P = 1 << lgP, J = 1 << lgJ;
  const int r = (int)(item - g.item0[slot]);
  const bool pair = r > 0 && 2 * r < P;
  const int lgQb = std::min(std::min(lgQ, LGCAP - lgJ), LGNT);
  const int Qb = 1 << lgQb, nqb = 1 << (lgQ - lgQb);
  const bool twlds = lgJ <= kLgTwl;
  if (twlds)
    for (int m = threadIdx.x; m < J; m += NT) twl[m] = tw[(int64_t)m << (lgS - lgJ)];  // w_J^m
  const int lgG = lgJ <= LGNT ? LGNT - lgJ : 0;  // threads per output row
  const int G = 1 << lgG;
  const int rpt = lgJ > LGNT ? 1 << (lgJ - LGNT) : 1;  // rows per thread
  const int j0 = threadIdx.x >> lgG, gi = threadIdx.x & (G - 1);
  const float2 *u = (const float2 *)(g.u[slot] + v * g.us[slot]) + ((int64_t)r << lgR);
  float *y = g.y[slot] + v * ((int64_t)1 << lgD);
  const float *gl = gtab + (int64_t)ld.layer_id * ((int64_t)1 << lgD);
  // load mapping: each thread keeps column qq, rows s = s0 + i * ds
  const int qq_l = threadIdx.x & (Qb - 1), s0 = threadIdx.x >> lgQb, ds = NT >> lgQb;
  const float2 rstep = cis_neg(((int64_t)ds * r) & ((1ll << lgM) - 1), lgM);   // w_M^{ds r}
  const float2 rstart = cis_neg(((int64_t)s0 * r) & ((1ll << lgM) - 1), lgM);  // w_M^{s0 r}
  // the residue's R = J Q values through a buffer resource (8 R bytes < 2^32): lane offset of row s0,
  // column qq_l; uniform step of ds rows
  const __amdgpu_buffer_rsrc_t ur = buf_rsrc(u, (uint32_t)(8ll << lgR));
  const uint32_t vo = (uint32_t)(qq_l + ((int64_t)s0 << lgQ)) * 8u;
  const uint32_t sstep = (uint32_t)(((int64_t)ds << lgQ) * 8);
  const int nr = (J << lgQb) >= NT ? (J << lgQb) >> LGNT : 1;
  const bool act = s0 < J;
  // y (+)= the scaled sums of output row j (sets A and B, X_{N/2} for r = 0)
  auto emit = [&](int j, float2 a, float2 b, float2 nn, bool add) {
    const int64_t ka = r + ((int64_t)j << lgP);
    float2 va, vb = make_float2(0.f, 0.f);
    int64_t ia, ib = 0;
    if (ka == 0) {
      ia = 0;
      va = make_float2(c1 * gl[0] * a.x, c1 * gl[1] * nn.x);
    } else {
      ia = 2 * ka;
      va = make_float2(c2 * gl[ia] * a.x, c2 * gl[ia + 1] * a.y);
    }
    if (pair) {
      ib = 2 * ((P - r) + ((int64_t)(J - 1 - j) << lgP));
      vb = make_float2(c2 * gl[ib] * b.x, c2 * gl[ib + 1] * b.y);
    }
    float2 *pa = (float2 *)(y + ia), *pb = (float2 *)(y + ib);
    if (add) {
      va = cadd(va, *pa);
      if (pair) vb = cadd(vb, *pb);
    }
    *pa = va;
    if (pair) *pb = vb;
  };
  // J Qb <= CAP values per column block: nr <= MAXE rows s = s0 + i ds per thread; the lane's element
  // (s, qq_l) goes to buf[threadIdx.x + i NT].  The next block's loads are issued before this block's
  // transform, so they are in flight during it.
  typedef unsigned int u2v __attribute__((ext_vector_type(2)));
  float2 val[MAXE];
  auto load_block = [&](int64_t q0) {
#pragma unroll
    for (int i = 0; i < MAXE; ++i) {
      if (i < nr && act) {
        const u2v w2 = __builtin_amdgcn_raw_buffer_load_b64(ur, (int)vo, (int)(q0 * 8 + i * sstep), 0);
        val[i] = make_float2(__uint_as_float(w2.x), __uint_as_float(w2.y));
      }
    }
  };
  // this thread's part of row j over the block's columns q = q0 + gi + G m, k = r + P j: set A adds
  // w_N^{q k} W_q[j], set B adds conj(W_q[j]) w_N^{q (M - k)} (= conj(w_N^{q k} W_q[j]) w_Q^q); both
  // twiddles by recurrence over m (at most 16 steps) from values computed directly
  auto row_sums = [&](int j, int64_t q0, float2 &a, float2 &b, float2 &nn) {
    a = b = nn = make_float2(0.f, 0.f);
    const int64_t k = r + ((int64_t)j << lgP), nmask = (1ll << lgN) - 1;
    float2 wa = cis_neg(((q0 + gi) * k) & nmask, lgN);
    const float2 was = cis_neg(((int64_t)G * k) & nmask, lgN);
    float2 wb = cis_neg(((q0 + gi) * (((int64_t)1 << lgM) - k)) & nmask, lgN);
    const float2 wbs = cis_neg(((int64_t)G * (((int64_t)1 << lgM) - k)) & nmask, lgN);
    for (int qq = gi; qq < Qb; qq += G) {
      const float2 w = buf[(j << lgQb) + qq];
      a = cadd(a, cmul(w, wa));
      if (pair) b = cadd(b, cmul(cconj(w), wb));
      if (r == 0 && j == 0) nn = ((q0 + qq) & 1) ? csub(nn, w) : cadd(nn, w);
      wa = cmul(wa, was);
      if (pair) wb = cmul(wb, wbs);
    }
  };
  // rows per thread <= kRAcc: the sums stay in registers across the column blocks and are written once
  const bool racc = rpt <= kRAcc;
  float2 acc_a[kRAcc], acc_b[kRAcc], acc_n = make_float2(0.f, 0.f);
#pragma unroll
  for (int i = 0; i < kRAcc; ++i) acc_a[i] = acc_b[i] = make_float2(0.f, 0.f);
  load_block(0);
  for (int qb = 0; qb < nqb; ++qb) {
    const int64_t q0 = (int64_t)qb << lgQb;
    {
      float2 tr = rstart;
#pragma unroll
      for (int i = 0; i < MAXE; ++i) {
        if (i < nr && act) {
          buf[threadIdx.x + i * NT] = cmul(val[i], tr);
          tr = cmul(tr, rstep);
        }
      }
    }
    if (qb + 1 < nqb) load_block(q0 + Qb);
    if (twlds)
      lds_fft<false, NT, MAXE, true, true>(buf, lgJ, lgQb, twl, lgJ);
    else
      lds_fft<false, NT, MAXE, true, true>(buf, lgJ, lgQb, tw, lgS);
    if (racc) {
#pragma unroll
      for (int i = 0; i < kRAcc; ++i) {
        if (i < rpt) {
          float2 a, b, nn;
          row_sums(j0 + (i << (LGNT - lgG)), q0, a, b, nn);
          acc_a[i] = cadd(acc_a[i], a);
          acc_b[i] = cadd(acc_b[i], b);
          acc_n = cadd(acc_n, nn);
        }
      }
    } else {
      for (int i = 0; i < rpt; ++i) {  // here G = 1
        const int j = j0 + (i << (LGNT - lgG));
        float2 a, b, nn;
        row_sums(j, q0, a, b, nn);
        emit(j, a, b, nn, qb > 0);
      }
    }
    __syncthreads();
  }
  if (racc) {
    if (G == 1) {
#pragma unroll
      for (int i = 0; i < kRAcc; ++i)
        if (i < rpt) emit(j0 + (i << (LGNT - lgG)), acc_a[i], acc_b[i], acc_n, false);
    } else {
      // combine the G partial sums of each row in a fixed order
      buf[threadIdx.x] = acc_a[0];
      buf[NT + threadIdx.x] = acc_b[0];
      buf[2 * NT + threadIdx.x] = acc_n;
      __syncthreads();
      if ((int)threadIdx.x < J) {
        float2 sa = make_float2(0.f, 0.f), sb = sa, sn2 = sa;
        for (int k = 0; k < G; ++k) {
          sa = cadd(sa, buf[(threadIdx.x << lgG) + k]);
          sb = cadd(sb, buf[NT + (threadIdx.x << lgG) + k]);
          sn2 = cadd(sn2, buf[2 * NT + (threadIdx.x << lgG) + k]);
        }
        emit((int)threadIdx.x, sa, sb, sn2, false);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Layers with N = D and n <= 16384: X_{c + (N/L) e} = FFT_L(v_b w_N^{b c})[e].
// The c values go in groups of CAP / L (max(1, D / CAP) groups whatever L is):
// one workgroup per (group, layer, vector), blockIdx.x = group * ipg + the
// (layer, vector) index of xcd_decode (ipg a multiple of 8, so a vector's
// workgroups stay on one XCD).
// ---------------------------------------------------------------------------
template <int LGNT, int LGCAP>
__global__ __launch_bounds__(1 << LGNT) void k_ffs_fwd(const LayerDesc *__restrict__ layers, FfLayers g, int dtype,
                                                 int lgD, int64_t b_begin, int64_t bc, const float *__restrict__ gtab,
                                                 float c1, float c2, const float2 *__restrict__ tw, int lgS, Key key,
                                                 int64_t ipg) {
  constexpr int NT = 1 << LGNT, CAP = 1 << LGCAP, MAXE = CAP / NT;
  __shared__ float2 buf[CAP];
  __shared__ uint32_t sw[CAP / 32];
  __shared__ float2 tlo[1 << kLgTwSplit], thi[1 << kLgTwSplit];
  const int cgrp = (int)(blockIdx.x / ipg);
  int64_t item, v;
  {
    const int64_t L = blockIdx.x - cgrp * ipg, rest = L >> 3;
    item = rest % g.n;
    v = (rest / g.n) * 8 + (L & 7);
    if (v >= bc) return;
  }
  const int slot = (int)item;
  const LayerDesc &ld = layers[g.layer[slot]];
  const int64_t n = ld.n;
  int lgL = 1;
  while ((1ll << lgL) < n) ++lgL;
  const int L = 1 << lgL;
  const int lgcs = lgD - lgL;                       // log2 of the number of c values
  const int lgcg = std::min(lgcs, LGCAP - lgL);    // c values per group
  const int tot = L << lgcg;                        // transform values per group (<= CAP)
  const uint32_t lid = (uint32_t)ld.layer_id;
  // w_N^m = thi[m >> lgLo] tlo[m & (2^lgLo - 1)] from two small LDS tables (D <= 2^(2 kLgTwSplit))
  const int lgLo = lgD >> 1, lgHi = lgD - lgLo;
  const bool split = lgHi <= kLgTwSplit;
  if (split) {
    for (int m = threadIdx.x; m < (1 << lgLo); m += NT) tlo[m] = tw[(int64_t)m << (lgS - lgD)];
    for (int m = threadIdx.x; m < (1 << lgHi); m += NT) thi[m] = tw[(int64_t)m << (lgS - lgHi)];
  }
  for (int w = threadIdx.x; w < (int)((n + 31) >> 5); w += NT) sw[w] = sign_word((uint64_t)w << 5, lid, key);
  // element e = threadIdx.x + i NT of every column group takes input b = e >> lgcg: the thread's inputs
  // are the same in every group, so they are loaded once (all loads issued before the first use)
  const void *x = g.x[slot];
  const int64_t xo = (b_begin + v) * n;
  float xr[MAXE];
#pragma unroll
  for (int i = 0; i < MAXE; ++i) {
    const int e = threadIdx.x + i * NT, b = e >> lgcg;
    xr[i] = (e < tot && b < n) ? load_x(x, dtype, xo + b) : 0.f;
  }
  __syncthreads();  // sign words and twiddle tables
#pragma unroll
  for (int i = 0; i < MAXE; ++i) {
    const int b = (threadIdx.x + i * NT) >> lgcg;
    if (b < n) xr[i] = flip(xr[i], (sw[b >> 5] >> (b & 31)) & 1u);
  }
  float *y = g.y[slot] + v * ((int64_t)1 << lgD);
  const float *gl = gtab + (int64_t)lid * ((int64_t)1 << lgD);
  {
    const int c0 = cgrp << lgcg;  // this workgroup's group of c values (c0 < 2^lgcs: the grid has D / CAP groups)
#pragma unroll
    for (int i = 0; i < MAXE; ++i) {
      const int e = threadIdx.x + i * NT;
      if (e < tot) {
        const int b = e >> lgcg, cc = e & ((1 << lgcg) - 1);
        const uint32_t m = (uint32_t)b * (uint32_t)(c0 + cc);  // < N
        const float2 w = split ? cmul(thi[m >> lgLo], tlo[m & ((1u << lgLo) - 1)]) : twiddle32<false>(tw, lgS, lgD, m);
        buf[e] = cscale(w, xr[i]);
      }
    }
    // outputs k = c + (N / L) ee, ee < L / 2: their G pairs are loaded before the transform, which
    // hides the latency
    const int tot2 = (L / 2) << lgcg;
    float2 gv[MAXE / 2];
#pragma unroll
    for (int i = 0; i < MAXE / 2; ++i) {
      const int e = threadIdx.x + i * NT;
      const int64_t k = (c0 + (e & ((1 << lgcg) - 1))) + ((int64_t)(e >> lgcg) << lgcs);
      if (e < tot2) gv[i] = *(const float2 *)(gl + 2 * k);
    }
    lds_fft<false, NT, MAXE>(buf, lgL, lgcg, tw, lgS);
#pragma unroll
    for (int i = 0; i < MAXE / 2; ++i) {
      const int e = threadIdx.x + i * NT;
      if (e >= tot2) break;
      const int64_t k = (c0 + (e & ((1 << lgcg) - 1))) + ((int64_t)(e >> lgcg) << lgcs);
      const float2 X = buf[e];
      if (k == 0)
        *(float2 *)y = make_float2(c1 * gv[i].x * X.x, c1 * gv[i].y * buf[(L / 2) << lgcg].x);  // X_{N/2}: c = 0, e = L/2
      else
        *(float2 *)(y + 2 * k) = make_float2(c2 * gv[i].x * X.x, c2 * gv[i].y * X.y);
    }
  }
}

// out[v] (+)= sum over the call's layers of y[l][v], in layer order
__global__ void k_ff_tail(const float *__restrict__ y, int nl, int64_t lstride, int64_t D, int64_t b_begin,
                          float *__restrict__ out, int accumulate) {
  const int64_t i = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) * 4;
  const int64_t v = blockIdx.y;
  if (i >= D) return;
  if ((uintptr_t)out & 15) {  // an output view without 16-byte alignment
    for (int k = 0; k < 4; ++k) {
      float a = 0.f;
      for (int l = 0; l < nl; ++l) a += y[l * lstride + v * D + i + k];
      float *o = out + (b_begin + v) * D + i + k;
      *o = accumulate ? *o + a : a;
    }
    return;
  }
  float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int l = 0; l < nl; ++l) {
    const float4 t = *(const float4 *)(y + l * lstride + v * D + i);
    a.x += t.x;
    a.y += t.y;
    a.z += t.z;
    a.w += t.w;
  }
  float4 *o = (float4 *)(out + (b_begin + v) * D + i);
  if (accumulate) {
    const float4 p = *o;
    a.x += p.x;
    a.y += p.y;
    a.z += p.z;
    a.w += p.w;
  }
  *o = a;
}

// coefficient c_k of the transpose (k < M): c_0 = g_0 z_0 / sqrt(D),
// c_k = sqrt(2/D) (g_{2k} z_{2k} + i g_{2k+1} z_{2k+1})
__device__ __forceinline__ float2 coef(const float *z, const float *gl, int64_t k, float c1, float c2) {
  if (k == 0) return make_float2(c1 * gl[0] * z[0], 0.f);
  return make_float2(c2 * gl[2 * k] * z[2 * k], c2 * gl[2 * k + 1] * z[2 * k + 1]);
}

// ---------------------------------------------------------------------------
// Pass 2, transpose: E~_r[q + Q s] (r <= P/2) from the coefficients of
// residues r and P - r (one inverse J-point transform per column q):
//   a_q[m] = c_{r+Pm} w_R^{-q m} + conj(c_{P-r+P(J-1-m)}) w_R^{q (J-m)},
//   E~_r[q + Q s] = w_N^{-q r} w_M^{-s r} IFFT_J(a_q)[s]  (+ (-1)^q c_{N/2}, r = 0).
// ---------------------------------------------------------------------------
template <int LGNT, int LGCAP>
__global__ __launch_bounds__(1 << LGNT) void k_ffq_T(const LayerDesc *__restrict__ layers, FfLayers g, int lgD,
                                               const float *__restrict__ z, int64_t b_begin, int64_t bc,
                                               const float *__restrict__ gtab, float c1, float c2,
                                               const float2 *__restrict__ tw, int lgS) {
  constexpr int NT = 1 << LGNT, CAP = 1 << LGCAP, MAXE = CAP / NT;
  __shared__ float2 buf[CAP];
  int64_t item, v;
  if (!xcd_decode(g.item0[g.n], bc, item, v)) return;
  const int slot = find_slot(g, item);
  const LayerDesc &ld = layers[g.layer[slot]];
  const FfGeom fg = ff_geom(ld.lgnp, lgD);
  const int lgM = fg.lgM, lgP = fg.lgP, lgJ = fg.lgJ, lgQ = fg.lgQ, lgR = fg.lgR, lgN = fg.lgN;
  const int P = 1 << lgP, J = 1 << lgJ;
  const int r = (int)(item - g.item0[slot]);
  const bool pair = r > 0 && 2 * r < P;
  const int lgQb = std::min(std::min(lgQ, LGCAP - lgJ), LGNT);
  const int Qb = 1 << lgQb, nqb = 1 << (lgQ - lgQb);
  const float *zv = z + (b_begin + v) * ((int64_t)1 << lgD);
  const float *gl = gtab + (int64_t)ld.layer_id * ((int64_t)1 << lgD);
  const float cN2 = c1 * gl[1] * zv[1];
  float2 *u = (float2 *)(g.u[slot] + v * g.us[slot]) + ((int64_t)r << lgR);
  const int qq_l = threadIdx.x & (Qb - 1), s0 = threadIdx.x >> lgQb, ds = NT >> lgQb;
  const float2 rstep = cis_neg(((int64_t)ds * r) & ((1ll << lgM) - 1), lgM);   // w_M^{ds r}
  const float2 rstart = cis_neg(((int64_t)s0 * r) & ((1ll << lgM) - 1), lgM);  // w_M^{s0 r}
  for (int qb = 0; qb < nqb; ++qb) {
    const int64_t q = ((int64_t)qb << lgQb) + qq_l;
    // rows m = s0 + i ds: w_R^{q m} by recurrence; w_R^{q (J - m)} = w_Q^{q} conj(w_R^{q m})
    {
      float2 wm = cis_neg((q * s0) & ((1ll << lgR) - 1), lgR);
      const float2 wst = cis_neg((q * ds) & ((1ll << lgR) - 1), lgR);
      const float2 wqq = cis_neg(q & ((1ll << lgQ) - 1), lgQ);
      // coefficient loads four rows at a time, issued before they are used
      for (int m0 = s0; m0 < J; m0 += 4 * ds) {
        float2 ca[4], cp[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int m = m0 + k * ds;
          if (m < J) {
            ca[k] = coef(zv, gl, r + ((int64_t)m << lgP), c1, c2);
            if (pair) cp[k] = coef(zv, gl, (P - r) + ((int64_t)(J - m - 1) << lgP), c1, c2);
          }
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int m = m0 + k * ds;
          if (m < J) {
            float2 a = cmulc(ca[k], wm);
            if (pair) a = cadd(a, cmul(cconj(cp[k]), cmulc(wqq, wm)));
            buf[(m << lgQb) + qq_l] = a;
            wm = cmul(wm, wst);
          }
        }
      }
    }
    lds_fft<true, NT, MAXE>(buf, lgJ, lgQb, tw, lgS);
    {
      const float2 tq = cis_neg((q * r) & ((1ll << lgN) - 1), lgN);  // w_N^{q r}
      float2 tr = rstart;
      for (int s = s0; s < J; s += ds) {
        float2 E = cmulc(cmulc(buf[(s << lgQb) + qq_l], tq), tr);
        if (r == 0) E.x += (q & 1) ? -cN2 : cN2;
        u[q + ((int64_t)s << lgQ)] = E;
        tr = cmul(tr, rstep);
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Pass 1, transpose: x[t][b] = Re sum_{r <= P/2} w_P^{-t r} E~_r[b] for one
// column block (a complex-to-real inverse transform of two columns at a
// time), signed, plus theta0, truncated to the layer.
// ---------------------------------------------------------------------------
template <int LGNT, int LGCAP>
__global__ __launch_bounds__(1 << LGNT) void k_ffr_T(const LayerDesc *__restrict__ layers, FfLayers g, int out_dtype,
                                               int lgD, int64_t b_begin, int64_t bc,
                                               const float2 *__restrict__ tw, int lgS, Key key) {
  constexpr int NT = 1 << LGNT, CAP = 1 << LGCAP, MAXE = CAP / NT;
  __shared__ float2 buf[CAP];
  __shared__ uint32_t sw[1024];
  int64_t item, v;
  if (!xcd_decode(g.item0[g.n], bc, item, v)) return;
  const int slot = find_slot(g, item);
  const LayerDesc &ld = layers[g.layer[slot]];
  const FfGeom fg = ff_geom(ld.lgnp, lgD);
  const int lgR = fg.lgR, lgP = fg.lgP, lgW = fg.lgW, lgWc = lgW - 1;
  const int64_t R = 1ll << lgR, n = ld.n;
  const int P = 1 << lgP;
  const int64_t b0 = (item - g.item0[slot]) << lgW;
  const int64_t rows = std::min<int64_t>((n + R - 1) >> lgR, (int64_t)P);
  const int nw = 1 << (lgW - 5);
  build_row_signs<NT>(sw, rows, lgR, b0, lgW, (uint32_t)ld.layer_id, key);
  const float *u = g.u[slot] + v * g.us[slot];
  // (P/2 + 1) Wc <= CAP/2 + Wc values: at most MAXL per thread, loaded before use
  constexpr int MAXL = CAP / (2 * NT) + 1;
  const int tot = (P / 2 + 1) << lgWc;
  float4 Ev[MAXL];
#pragma unroll
  for (int i = 0; i < MAXL; ++i) {
    const int e = threadIdx.x + i * NT;
    if (e < tot) {
      const int r = e >> lgWc, c = e & ((1 << lgWc) - 1);
      Ev[i] = *(const float4 *)(u + (((int64_t)r << lgR) + b0 + 2 * c) * 2);
    }
  }
#pragma unroll
  for (int i = 0; i < MAXL; ++i) {
    const int e = threadIdx.x + i * NT;
    if (e >= tot) break;
    const int r = e >> lgWc, c = e & ((1 << lgWc) - 1);
    const float4 E = Ev[i];
    const bool edge = r == 0 || 2 * r == P;
    const float2 ha = edge ? make_float2(E.x, 0.f) : make_float2(0.5f * E.x, 0.5f * E.y);
    const float2 hb = edge ? make_float2(E.z, 0.f) : make_float2(0.5f * E.z, 0.5f * E.w);
    buf[(r << lgWc) + c] = make_float2(ha.x - hb.y, ha.y + hb.x);          // H_a + i H_b
    if (!edge) buf[((P - r) << lgWc) + c] = make_float2(ha.x + hb.y, hb.x - ha.y);  // conj H_a + i conj H_b
  }
  lds_fft<true, NT, MAXE, false, true>(buf, lgP, lgWc, tw, lgS);
  void *o = (void *)g.x[slot];
  const float *th = g.th[slot];
  const int64_t oo = (b_begin + v) * n;
  // rows * Wc <= CAP values: at most MAXE per thread; the theta0 loads go out before the sums
  const int tot1 = (int)(rows << lgWc);
  float2 thv[MAXE];
  if (th) {
#pragma unroll
    for (int i = 0; i < MAXE; ++i) {
      const int e = threadIdx.x + i * NT;
      const int64_t j = ((int64_t)(e >> lgWc) << lgR) + b0 + 2 * (e & ((1 << lgWc) - 1));
      thv[i] = make_float2(0.f, 0.f);
      if (e < tot1 && j < n) thv[i].x = th[j];
      if (e < tot1 && j + 1 < n) thv[i].y = th[j + 1];
    }
  }
#pragma unroll
  for (int i = 0; i < MAXE; ++i) {
    const int e = threadIdx.x + i * NT;
    if (e >= tot1) break;
    const int64_t t = e >> lgWc;
    const int c = e & ((1 << lgWc) - 1);
    const float2 zt = buf[e];
    const int64_t j = (t << lgR) + b0 + 2 * c;
    if (j < n) {
      float a = flip(zt.x, row_sign_bit(sw, t, nw, lgR, b0, j));
      if (th) a += thv[i].x;
      store_out(o, out_dtype, oo + j, a);
    }
    if (j + 1 < n) {
      float b = flip(zt.y, row_sign_bit(sw, t, nw, lgR, b0, j + 1));
      if (th) b += thv[i].y;
      store_out(o, out_dtype, oo + j + 1, b);
    }
  }
}

// ---------------------------------------------------------------------------
// Small layers, transpose: x_b = Re sum_c w_N^{-b c} IFFT_L(coef_c)[b].
// ---------------------------------------------------------------------------
template <int LGNT, int LGCAP>
__global__ __launch_bounds__(1 << LGNT) void k_ffs_T(const LayerDesc *__restrict__ layers, FfLayers g, int out_dtype,
                                               int lgD, const float *__restrict__ z, int64_t b_begin, int64_t bc,
                                               const float *__restrict__ gtab, float c1, float c2,
                                               const float2 *__restrict__ tw, int lgS, Key key) {
  constexpr int NT = 1 << LGNT, CAP = 1 << LGCAP, MAXE = CAP / NT;
  __shared__ float2 buf[CAP];
  __shared__ uint32_t sw[CAP / 32];
  int64_t item, v;
  if (!xcd_decode(g.n, bc, item, v)) return;
  const int slot = (int)item;
  const LayerDesc &ld = layers[g.layer[slot]];
  const int64_t n = ld.n;
  int lgL = 1;
  while ((1ll << lgL) < n) ++lgL;
  const int L = 1 << lgL;
  const int lgcs = lgD - lgL;
  const int lgcg = std::min(lgcs, LGCAP - lgL);
  const uint32_t lid = (uint32_t)ld.layer_id;
  for (int w = threadIdx.x; w < (int)((n + 31) >> 5); w += NT) sw[w] = sign_word((uint64_t)w << 5, lid, key);
  const float *zv = z + (b_begin + v) * ((int64_t)1 << lgD);
  const float *gl = gtab + (int64_t)lid * ((int64_t)1 << lgD);
  float acc[MAXE];
#pragma unroll
  for (int i = 0; i < MAXE; ++i) acc[i] = 0.f;
  for (int c0 = 0; c0 < (1 << lgcs); c0 += 1 << lgcg) {
    __syncthreads();
    for (int e = threadIdx.x; e < (L << lgcg); e += NT) {
      const int ee = e >> lgcg, cc = e & ((1 << lgcg) - 1);
      const int c = c0 + cc;
      float2 a = make_float2(0.f, 0.f);
      if (2 * ee < L) {
        a = coef(zv, gl, c + ((int64_t)ee << lgcs), c1, c2);
      } else if (2 * ee == L && c == 0) {
        a = make_float2(c1 * gl[1] * zv[1], 0.f);  // the (-1)^b row
      }
      buf[e] = a;
    }
    lds_fft<true, NT, MAXE>(buf, lgL, lgcg, tw, lgS);
    for (int cc = 0; cc < (1 << lgcg); ++cc) {
#pragma unroll
      for (int i = 0; i < MAXE; ++i) {
        const int b = threadIdx.x + i * NT;
        if (b < L) {
          const float2 w = buf[(b << lgcg) + cc];
          const float2 t = twiddle<false>(tw, lgS, lgD, (int64_t)b * (c0 + cc));
          acc[i] += w.x * t.x + w.y * t.y;  // Re(w conj(t))
        }
      }
    }
  }
  void *o = (void *)g.x[slot];
  const float *th = g.th[slot];
  const int64_t oo = (b_begin + v) * n;
#pragma unroll
  for (int i = 0; i < MAXE; ++i) {
    const int b = threadIdx.x + i * NT;
    if (b < n) {
      float a = flip(acc[i], (sw[b >> 5] >> (b & 31)) & 1u);
      if (th) a += th[b];
      store_out(o, out_dtype, oo + b, a);
    }
  }
}

}  // namespace

// ------------------------------- host side ---------------------------------

namespace {
int lg2(int64_t v) {
  int l = 0;
  while ((1ll << l) < v) ++l;
  return l;
}
int64_t ceil8(int64_t v) { return (v + 7) / 8 * 8; }
}  // namespace

bool afjlf_small_layer(const sk_sketch *s, int layer) {
  const LayerDesc &ld = s->layers[layer];
  return ld.np == s->D && ld.n <= kCap;
}

// floats per vector of a layer's pass buffer: (P/2 + 1) R complex
int64_t afjlf_u_floats(const sk_sketch *s, int layer) {
  if (afjlf_small_layer(s, layer)) return 0;
  const FfGeom fg = ff_geom(s->layers[layer].lgnp, lg2(s->D));
  return s->layers[layer].np + (2ll << fg.lgR);
}

bool afjlf_two_pass_ok(int lgnp, int lgD) {
  const FfGeom fg = ff_geom(lgnp, lgD);
  // (the residue buffers are addressed with 32-bit byte offsets: 8 R <= 2^30)
  return fg.lgQ >= 1 && fg.lgJ >= 0 && fg.lgJ <= kLgCap && fg.lgR <= 27;
}

int64_t afjlf_bytes_per_vector(const sk_sketch *s, int l0, int l1, bool transpose) {
  int64_t u = 0;
  for (int l = l0; l < l1; ++l) u = std::max(u, afjlf_u_floats(s, l));
  return (u + (transpose ? 0 : (int64_t)(l1 - l0) * s->D)) * 4;
}

void afjlf_twiddles(int64_t D, std::vector<float> &host, int &lgS) {
  const int64_t S = std::max<int64_t>(D, 4096);
  lgS = lg2(S);
  host.resize(2 * S);
  for (int64_t m = 0; m < S; ++m) {
    const double a = -2.0 * M_PI * (double)m / (double)S;
    host[2 * m] = (float)std::cos(a);
    host[2 * m + 1] = (float)std::sin(a);
  }
}

namespace {

// whether a two-pass layer's residue pass needs the 16384-value kernels
bool big_residue(const sk_sketch *s, int layer) {
  return ff_geom(s->layers[layer].lgnp, lg2(s->D)).lgJ > kLgCapS;
}
// whether a one-kernel layer needs the 16384-value kernels
bool big_small(const sk_sketch *s, int layer) { return s->layers[layer].n > (1 << kLgCapS); }

// The call's general (two-pass) layers in groups: a group holds up to kSlots
// layers of one residue-kernel size whose pass buffers for `tile` vectors fit
// in ufl floats; a layer too large for the whole chunk is a group of its own,
// run in vector tiles.
template <class F>
void for_groups(const sk_sketch *s, int l0, int l1, int64_t bc, int64_t ufl, F &&f) {
  for (int big = 0; big < 2; ++big) {
    int l = l0;
    while (l < l1) {
      if (afjlf_small_layer(s, l) || (int)big_residue(s, l) != big) {
        ++l;
        continue;
      }
      std::vector<int> grp{l};
      int64_t used = afjlf_u_floats(s, l) * bc;
      int64_t tile = bc;
      int lend = l + 1;
      if (used > ufl) {
        tile = std::max<int64_t>(1, ufl / afjlf_u_floats(s, l));
        if (tile > 8) tile &= ~7ll;  // whole XCD rounds (a vector's items run on XCD v mod 8)
      } else {
        while (lend < l1 && (int)grp.size() < kSlots) {
          if (afjlf_small_layer(s, lend) || (int)big_residue(s, lend) != big) {
            ++lend;
            continue;
          }
          const int64_t nd = afjlf_u_floats(s, lend) * bc;
          if (used + nd > ufl) break;
          used += nd;
          grp.push_back(lend++);
        }
      }
      f(grp, tile, big != 0);
      l = lend;
    }
  }
}

void small_groups(const sk_sketch *s, int l0, int l1, const std::function<void(FfLayers &, bool)> &f) {
  for (int big = 0; big < 2; ++big) {
    FfLayers g{};
    for (int l = l0; l < l1; ++l) {
      if (!afjlf_small_layer(s, l) || (int)big_small(s, l) != big) continue;
      g.layer[g.n++] = l;
      if (g.n == kSlots) {
        f(g, big != 0);
        g = FfLayers{};
      }
    }
    if (g.n) f(g, big != 0);
  }
}

}  // namespace

// Forward of layers [l0, l1) for vectors b_begin .. b_begin + bc - 1.  ws
// holds (l1 - l0) bc D floats of per-layer contributions, then pass buffers.
void run_afjlf_fwd(sk_sketch *s, int l0, int l1, const void *const *grads, int dtype, int64_t b_begin,
                   int64_t bc, float *ws, int64_t ws_floats, float *out, bool accumulate, hipStream_t st) {
  const int esz = dtype == SK_BF16 ? 2 : 4;
  const int64_t D = s->D;
  const int lgD = lg2(D);
  const float c1 = (float)(1.0 / std::sqrt((double)D)), c2 = (float)std::sqrt(2.0 / (double)D);
  const int nl = l1 - l0;
  const int64_t lstride = bc * D;
  float *ybase = ws, *ubase = ws + (int64_t)nl * lstride;
  const int64_t ufl = ws_floats - (int64_t)nl * lstride;
  const float2 *tw = (const float2 *)s->d_ftw;
  small_groups(s, l0, l1, [&](FfLayers &g, bool big) {
    int64_t gb = 0;
    for (int i = 0; i < g.n; ++i) {
      g.x[i] = grads[g.layer[i] - l0];
      g.y[i] = ybase + (int64_t)(g.layer[i] - l0) * lstride;
      gb += bc * s->layers[g.layer[i]].n * esz;
    }
    // one workgroup per group of c values: max(1, D / CAP) groups for every layer
    const int64_t ipg = (int64_t)g.n * ceil8(bc);
    const int64_t ncg = std::max<int64_t>(1, D >> (big ? 14 : 13));
    const dim3 grid((unsigned)(ipg * ncg));
    SK_PROF(SK_PROF_FF_SMALL, gb, {
      if (big)
        hipLaunchKernelGGL((k_ffs_fwd<10, 14>), grid, dim3(1024), 0, st, s->d_layers, g, dtype, lgD, b_begin, bc,
                           s->d_gtab, c1, c2, tw, s->ftw_lg, s->key, ipg);
      else
        hipLaunchKernelGGL((k_ffs_fwd<9, 13>), grid, dim3(512), 0, st, s->d_layers, g, dtype, lgD, b_begin, bc,
                           s->d_gtab, c1, c2, tw, s->ftw_lg, s->key, ipg);
    });
  });
  for_groups(s, l0, l1, bc, ufl, [&](const std::vector<int> &grp, int64_t tile, bool big) {
    for (int64_t t0 = 0; t0 < bc; t0 += tile) {
      const int64_t tb = std::min(tile, bc - t0);
      FfLayers g1{}, g2{};
      int64_t off = 0, gb = 0;
      for (int l : grp) {
        const int i = g1.n;
        const LayerDesc &ld = s->layers[l];
        const FfGeom fg = ff_geom(ld.lgnp, lgD);
        const FfGeom fg1 = ff_geom(ld.lgnp, lgD, kLgRows);  // pass 1 column blocks
        gb += tb * ld.n * esz;
        g1.layer[i] = g2.layer[i] = l;
        g1.x[i] = grads[l - l0];
        g1.u[i] = g2.u[i] = ubase + off;
        g1.us[i] = g2.us[i] = afjlf_u_floats(s, l);
        g2.y[i] = ybase + (int64_t)(l - l0) * lstride + t0 * D;
        g1.item0[i + 1] = g1.item0[i] + ((int64_t)1 << (fg1.lgR - fg1.lgW));
        g2.item0[i + 1] = g2.item0[i] + ((int64_t)1 << (fg.lgP - 1)) + 1;
        off += g1.us[i] * tb;
        ++g1.n;
        ++g2.n;
      }
      SK_PROF(SK_PROF_FF_ROWS, gb,
              hipLaunchKernelGGL((k_ffr_fwd<kLgRows - 4, kLgRows>), dim3((unsigned)(g1.item0[g1.n] * ceil8(tb))),
                                 dim3(1 << (kLgRows - 4)), 0,
                                 st, s->d_layers, g1, dtype, lgD, b_begin + t0, tb, tw, s->ftw_lg, s->key));
      const dim3 grid2((unsigned)(g2.item0[g2.n] * ceil8(tb)));
      SK_PROF(SK_PROF_FF_RES, 0, {
        if (big)
          hipLaunchKernelGGL((k_ffq_fwd<10, 14>), grid2, dim3(1024), 0, st, s->d_layers, g2, lgD, tb, s->d_gtab, c1,
                             c2, tw, s->ftw_lg);
        else
          hipLaunchKernelGGL((k_ffq_fwd<9, 13>), grid2, dim3(512), 0, st, s->d_layers, g2, lgD, tb, s->d_gtab, c1,
                             c2, tw, s->ftw_lg);
      });
    }
  });
  const dim3 gt((unsigned)((D / 4 + 255) / 256), (unsigned)bc);
  SK_PROF(SK_PROF_GATHER, bc * D * 4,
          hipLaunchKernelGGL(k_ff_tail, gt, dim3(256), 0, st, ybase, nl, lstride, D, b_begin, out, (int)accumulate));
}

// Transpose of layers [l0, l1) for vectors b_begin .. b_begin + bc - 1; ws holds the pass buffers.
void run_afjlf_T(sk_sketch *s, int l0, int l1, const float *z, int64_t b_begin, int64_t bc, float *ws,
                 int64_t ws_floats, void *const *outs, int out_dtype, const void *const *theta0, hipStream_t st) {
  const int osz = out_dtype == SK_BF16 ? 2 : 4;
  const int64_t D = s->D;
  const int lgD = lg2(D);
  const float c1 = (float)(1.0 / std::sqrt((double)D)), c2 = (float)std::sqrt(2.0 / (double)D);
  const float2 *tw = (const float2 *)s->d_ftw;
  small_groups(s, l0, l1, [&](FfLayers &g, bool big) {
    int64_t ob = 0;
    for (int i = 0; i < g.n; ++i) {
      const int64_t n = s->layers[g.layer[i]].n;
      g.x[i] = outs[g.layer[i] - l0];
      g.th[i] = theta0 ? (const float *)theta0[g.layer[i] - l0] : nullptr;
      ob += bc * n * osz + (g.th[i] ? n * 4 : 0);
    }
    const dim3 grid((unsigned)(g.n * ceil8(bc)));
    SK_PROF(SK_PROF_GATHER, ob, {
      if (big)
        hipLaunchKernelGGL((k_ffs_T<10, 14>), grid, dim3(1024), 0, st, s->d_layers, g, out_dtype, lgD, z, b_begin,
                           bc, s->d_gtab, c1, c2, tw, s->ftw_lg, s->key);
      else
        hipLaunchKernelGGL((k_ffs_T<9, 13>), grid, dim3(512), 0, st, s->d_layers, g, out_dtype, lgD, z, b_begin, bc,
                           s->d_gtab, c1, c2, tw, s->ftw_lg, s->key);
    });
  });
  for_groups(s, l0, l1, bc, ws_floats, [&](const std::vector<int> &grp, int64_t tile, bool big) {
    for (int64_t t0 = 0; t0 < bc; t0 += tile) {
      const int64_t tb = std::min(tile, bc - t0);
      FfLayers g1{}, g2{};
      int64_t off = 0, ob = 0;
      for (int l : grp) {
        const int i = g1.n;
        const LayerDesc &ld = s->layers[l];
        const FfGeom fg = ff_geom(ld.lgnp, lgD);
        g1.layer[i] = g2.layer[i] = l;
        g1.x[i] = outs[l - l0];
        g1.th[i] = theta0 ? (const float *)theta0[l - l0] : nullptr;
        ob += tb * ld.n * osz + (g1.th[i] ? ld.n * 4 : 0);
        g1.u[i] = g2.u[i] = ws + off;
        g1.us[i] = g2.us[i] = afjlf_u_floats(s, l);
        g1.item0[i + 1] = g1.item0[i] + ((int64_t)1 << (fg.lgR - fg.lgW));
        g2.item0[i + 1] = g2.item0[i] + ((int64_t)1 << (fg.lgP - 1)) + 1;
        off += g1.us[i] * tb;
        ++g1.n;
        ++g2.n;
      }
      const dim3 grid2((unsigned)(g2.item0[g2.n] * ceil8(tb)));
      SK_PROF(SK_PROF_FF_RES, tb * D * 4, {
        if (big)
          hipLaunchKernelGGL((k_ffq_T<10, 14>), grid2, dim3(1024), 0, st, s->d_layers, g2, lgD, z, b_begin + t0, tb,
                             s->d_gtab, c1, c2, tw, s->ftw_lg);
        else
          hipLaunchKernelGGL((k_ffq_T<9, 13>), grid2, dim3(512), 0, st, s->d_layers, g2, lgD, z, b_begin + t0, tb,
                             s->d_gtab, c1, c2, tw, s->ftw_lg);
      });
      SK_PROF(SK_PROF_GATHER, ob,
              hipLaunchKernelGGL((k_ffr_T<9, 13>), dim3((unsigned)(g1.item0[g1.n] * ceil8(tb))), dim3(512), 0, st,
                                 s->d_layers, g1, out_dtype, lgD, b_begin + t0, tb, tw, s->ftw_lg, s->key));
    }
  });
}

}  // namespace sk
