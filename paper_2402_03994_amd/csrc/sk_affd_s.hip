// sk_affd_s.hip -- AFFD (eq. bami) for groups of small layers.
//
// A layer is small here when it pads to N' = D (two Kronecker digits: p with
// dk1 = D / 1024 values and l with 1024) and has at most kSmallRows source
// rows of 1024 elements (biases and norm weights of a transformer).  With no
// top digits the method reduces to
//   W  = Scatter_pi1(B x) (rows pi1_p(h) for the live source rows h)
//   F  = (I (x) H_l) (g . ((H_p (x) I) (I (x) H_l) W))
//   AFFD(x)[a 1024 + b] = ((H_p (x) I) F)[pi2_p(a), pi2_l(b)]   (N' = D).
// Since W has at most kSmallRows non-zero rows, (H_p (x) I) W is formed row by
// row as a signed sum of those rows, inside the kernel that applies g; that
// kernel stores F with its columns already gathered through pi2_l, so the last
// kernel transforms columns b of F and writes output columns b directly.  Up
// to 64 layers run in one launch per phase (grid z = slot), each with its own
// region of the workspace; the last kernel adds the slots in slot order, so the
// result does not depend on the schedule.
#include <algorithm>

#include "sk_kcommon.h"
#include "sk_launch.h"

namespace sk {

// A: workgroup per (slot, live source row h, 8 vectors): sign, pi1 on the
// columns, H_l, write row pi1_p(h) of W.
template <bool BF16>
__global__ __launch_bounds__(256) void k_affdS_rows(const LayerDesc *__restrict__ layers,
                                                    const uint16_t *__restrict__ ptab, SmallGroup g,
                                                    int64_t b_begin, int64_t bc, float *__restrict__ w,
                                                    int64_t wslot, Key key) {
  using L = Lds1024<8>;
  __shared__ __align__(16) float s[L::kFloats];
  const int z = blockIdx.z;
  const LayerDesc &ld = layers[g.layer[z]];
  const int64_t h = blockIdx.x;
  if (h >= ld.rows_live) return;
  const void *x = g.x[z];
  const int col0 = threadIdx.x * 4;
  const int64_t j0 = h * 1024 + col0;
  const int64_t lim = ld.n - j0;
  const int64_t v0 = (int64_t)blockIdx.y * 8;
  const int nv = (int)((bc - v0) < 8 ? (bc - v0) : 8);
  uint32_t bits = 0;
  if (lim > 0) bits = sign_word((uint64_t)j0, (uint32_t)ld.layer_id, key) >> (j0 & 31);
  const uint16_t *fk = ptab + ld.poff[0][0][1];
#pragma unroll
  for (int v = 0; v < 8; ++v) {
    float val[4] = {0.f, 0.f, 0.f, 0.f};
    if (v < nv && lim > 0) load4<BF16, false>(x, (b_begin + v0 + v) * ld.n + j0, lim, val);
#pragma unroll
    for (int q = 0; q < 4; ++q) s[L::idx(v, fk[col0 + q])] = flip(val[q], (bits >> q) & 1u);
  }
  __syncthreads();
  fwht1024_lds<8>(s);
  const int64_t row = ptab[ld.poff[0][0][0] + h];
  float *wz = w + z * wslot + row * 1024;
  for (int v = 0; v < nv; ++v)
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int l = threadIdx.x + 256 * k;
      wz[(v0 + v) * ld.np + l] = s[L::idx(v, l)] * (1.0f / 32.0f);
    }
}

// B + C: workgroup per (slot, row p, 8 vectors): row p of (H_p (x) I) W as a
// signed sum of the live rows, times g, H_l -> row p of F.
__global__ __launch_bounds__(256) void k_affdS_top(const LayerDesc *__restrict__ layers,
                                                   const uint16_t *__restrict__ ptab, SmallGroup g, int64_t bc,
                                                   const float *__restrict__ w, int64_t wslot,
                                                   float *__restrict__ f, Key key) {
  using L = Lds1024<8>;
  __shared__ __align__(16) float s[L::kFloats];
  const int z = blockIdx.z;
  const LayerDesc &ld = layers[g.layer[z]];
  const int p = blockIdx.x;
  const int64_t v0 = (int64_t)blockIdx.y * 8;
  const int nv = (int)((bc - v0) < 8 ? (bc - v0) : 8);
  const int nh = (int)ld.rows_live;
  const float rs = rsqrtf((float)ld.dk1);
  float gk[4];
#pragma unroll
  for (int k = 0; k < 4; ++k)
    gk[k] = gauss((uint64_t)p * 1024 + threadIdx.x + 256 * k, (uint32_t)ld.layer_id, ST_GAUSS, key) * rs;
  // one pass per live row: the 64 loads of a pass are independent
  float acc[8][4];
#pragma unroll
  for (int v = 0; v < 8; ++v)
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[v][k] = 0.0f;
  const float *wz = w + z * wslot + v0 * ld.np + threadIdx.x;
  for (int h = 0; h < nh; ++h) {
    const int q = ptab[ld.poff[0][0][0] + h];
    const uint32_t sg = (uint32_t)__popc((uint32_t)(p & q)) & 1u;
    const float *wr = wz + (int64_t)q * 1024;
#pragma unroll
    for (int v = 0; v < 8; ++v)
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (v < nv) acc[v][k] += flip(wr[v * ld.np + 256 * k], sg);
  }
#pragma unroll
  for (int v = 0; v < 8; ++v)
#pragma unroll
    for (int k = 0; k < 4; ++k) s[L::idx(v, threadIdx.x + 256 * k)] = acc[v][k] * gk[k];
  __syncthreads();
  fwht1024_lds<8>(s);
  // F'[p][b] = F[p][pi2_l(b)]
  const uint16_t *p2l = ptab + ld.poff[1][0][1];
  int src[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) src[k] = p2l[threadIdx.x + 256 * k];
  float *fz = f + z * wslot;
  for (int v = 0; v < nv; ++v)
#pragma unroll
    for (int k = 0; k < 4; ++k)
      fz[(v0 + v) * ld.np + (int64_t)p * 1024 + threadIdx.x + 256 * k] = s[L::idx(v, src[k])] * (1.0f / 32.0f);
}

// B + C with the stored G (dk1 a multiple of 8): workgroup per (slot, 8 rows
// p, vector); the vector's live W rows are loaded once for the 8 rows, each
// row of (H_p (x) I) W is their signed sum, times g, H_l -> rows of F'.  Same
// arithmetic, in the same order, as k_affdS_top.
__global__ __launch_bounds__(256) void k_affdS_top8(const LayerDesc *__restrict__ layers,
                                                    const uint16_t *__restrict__ ptab, SmallGroup g,
                                                    const float *__restrict__ w, int64_t wslot, float *__restrict__ f) {
  using L = Lds1024<8>;
  __shared__ __align__(16) float s[L::kFloats];
  const int z = blockIdx.z;
  const LayerDesc &ld = layers[g.layer[z]];
  const int p0 = blockIdx.x * 8;
  const int64_t v = blockIdx.y;
  const int nh = (int)ld.rows_live;  // <= kSmallRows
  const float rs = rsqrtf((float)ld.dk1);
  const float *wz = w + z * wslot + v * ld.np + threadIdx.x;
  // every load is issued before the first use: the row ids, the 8 rows' G,
  // then the live rows (rows h >= nh read row q[0] and are not used)
  int q[kSmallRows];
#pragma unroll
  for (int h = 0; h < kSmallRows; ++h) q[h] = ptab[ld.poff[0][0][0] + (h < nh ? h : 0)];
  const float *gz = g.gt[z] + threadIdx.x;
  float gv[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int k = 0; k < 4; ++k) gv[i][k] = gz[(int64_t)(p0 + i) * 1024 + 256 * k];
  float wv[kSmallRows][4];
#pragma unroll
  for (int h = 0; h < kSmallRows; ++h)
#pragma unroll
    for (int k = 0; k < 4; ++k) wv[h][k] = wz[(int64_t)q[h] * 1024 + 256 * k];
  // rows past nh add zero (a select, not a branch per row, which would hold
  // each row's load back until its test)
#pragma unroll
  for (int h = 0; h < kSmallRows; ++h)
#pragma unroll
    for (int k = 0; k < 4; ++k) wv[h][k] = h < nh ? wv[h][k] : 0.0f;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int p = p0 + i;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      float acc = 0.0f;
#pragma unroll
      for (int h = 0; h < kSmallRows; ++h) acc += flip(wv[h][k], (uint32_t)__popc((uint32_t)(p & q[h])) & 1u);
      s[L::idx(i, threadIdx.x + 256 * k)] = acc * (gv[i][k] * rs);
    }
  }
  __syncthreads();
  fwht1024_lds<8>(s);
  // F'[p][b] = F[p][pi2_l(b)]
  const uint16_t *p2l = ptab + ld.poff[1][0][1];
  int src[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) src[k] = p2l[threadIdx.x + 256 * k];
  float *fz = f + z * wslot + v * ld.np + (int64_t)p0 * 1024 + threadIdx.x;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int k = 0; k < 4; ++k) fz[i * 1024 + 256 * k] = s[L::idx(i, src[k])] * (1.0f / 32.0f);
}

// D + E for dk1 = 64: workgroup per (32 output columns b, vector); thread
// (cc = tid % 32, rg = tid / 32) loads rows rg + 8 m (m < 8) of column cc of
// each slot's F' (128-byte row pieces), H_8 over m in registers, one LDS
// exchange, H_8 over the low three row bits, then adds rows pi2_p(a) for
// a = rg + 8 m.  Slots in order; the next slot's loads go out first.
__global__ __launch_bounds__(256) void k_affdS_cols64(const LayerDesc *__restrict__ layers,
                                                      const uint16_t *__restrict__ ptab, SmallGroup g, int nslots,
                                                      const float *__restrict__ f, int64_t wslot, int64_t b_begin,
                                                      float *__restrict__ out, int accumulate) {
  __shared__ float s[64 * 33];
  const int cb = blockIdx.x;
  const int64_t v = blockIdx.y;
  const int cc = threadIdx.x & 31, rg = threadIdx.x >> 5;
  const int64_t np = layers[g.layer[0]].np;  // = D for every slot
  float acc[8], nx[8];
#pragma unroll
  for (int m = 0; m < 8; ++m) acc[m] = 0.0f;
  auto fetch = [&](int z) {
    const float *fz = f + z * wslot + v * np + cb * 32 + cc;
#pragma unroll
    for (int m = 0; m < 8; ++m) nx[m] = fz[(int64_t)(rg + 8 * m) * 1024];
  };
  fetch(0);
  for (int z = 0; z < nslots; ++z) {
    float x[8];
#pragma unroll
    for (int m = 0; m < 8; ++m) x[m] = nx[m];
    if (z + 1 < nslots) fetch(z + 1);
    fwht_regs_t<8>(x);  // row bits 3..5
    __syncthreads();    // the previous slot's gathers from s are done
#pragma unroll
    for (int m = 0; m < 8; ++m) s[(rg + 8 * m) * 33 + cc] = x[m];
    __syncthreads();
#pragma unroll
    for (int m = 0; m < 8; ++m) x[m] = s[(8 * rg + m) * 33 + cc];
    fwht_regs_t<8>(x);  // row bits 0..2
#pragma unroll
    for (int m = 0; m < 8; ++m) s[(8 * rg + m) * 33 + cc] = x[m];
    __syncthreads();
    const uint16_t *p2 = ptab + layers[g.layer[z]].poff[1][0][0];
#pragma unroll
    for (int m = 0; m < 8; ++m) acc[m] += s[p2[rg + 8 * m] * 33 + cc];
  }
  float *o = out + (b_begin + v) * np + cb * 32 + cc;
#pragma unroll
  for (int m = 0; m < 8; ++m) {
    float *d = o + (int64_t)(rg + 8 * m) * 1024;
    const float val = acc[m] * 0.125f;  // 1 / sqrt(dk1)
    *d = accumulate ? *d + val : val;
  }
}

__global__ void k_affdS_gtab(const LayerDesc *__restrict__ layers, int layer, int64_t D, float *__restrict__ gt,
                             Key key) {
  const int64_t t = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) * 4;
  if (t >= D) return;
  float gq[4];
  gauss4((uint64_t)t >> 2, (uint32_t)layers[layer].layer_id, ST_GAUSS, key, gq);
#pragma unroll
  for (int q = 0; q < 4; ++q) gt[t + q] = gq[q];
}

void launch_affd_small_gtab(const sk_sketch *s, int layer, float *g, hipStream_t st) {
  hipLaunchKernelGGL(k_affdS_gtab, dim3((unsigned)((s->D / 4 + 255) / 256)), dim3(256), 0, st, s->d_layers, layer, s->D,
                     g, s->key);
  (void)hipGetLastError();
}

// D + E: workgroup per (16 output columns b, vector); for every slot in order:
// H_p along the dk1 rows of F'[.][b], add rows pi2_p(a), a < R, to out[a][b].
// The next slot's tile and row indices are loaded during the current
// transform.  Element e = tid + 256 i of a tile is (row e / 16, column e % 16).
template <int kMaxE>  // tile elements per thread: max(1, dk1 / 16)
__global__ __launch_bounds__(256) void k_affdS_cols(const LayerDesc *__restrict__ layers,
                                                    const uint16_t *__restrict__ ptab, SmallGroup g, int nslots,
                                                    const float *__restrict__ f, int64_t wslot, int R,
                                                    int64_t b_begin, float *__restrict__ out, int accumulate) {
  __shared__ float s[kMaxE * 256];
  const int cb = blockIdx.x;
  const int64_t v = blockIdx.y;
  const LayerDesc &l0 = layers[g.layer[0]];  // dk1 = R for every slot (N' = D)
  const int ne = (l0.dk1 * 16 + 255) / 256;
  const int nel = l0.dk1 * 16;
  const float rs = rsqrtf((float)l0.dk1);
  float nx[kMaxE], acc[kMaxE];
  int nidx[kMaxE];
  auto fetch = [&](int z) {
    const LayerDesc &ld = layers[g.layer[z]];
    const float *fz = f + z * wslot + v * ld.np + cb * 16;
    const uint16_t *p2 = ptab + ld.poff[1][0][0];
#pragma unroll
    for (int i = 0; i < kMaxE; ++i) {
      const int e = threadIdx.x + 256 * i;
      if (i < ne && e < nel) {
        nx[i] = fz[(int64_t)(e >> 4) * 1024 + (e & 15)];
        nidx[i] = p2[e >> 4] * 16 + (e & 15);
      }
    }
  };
#pragma unroll
  for (int i = 0; i < kMaxE; ++i) acc[i] = 0.0f;
  fetch(0);
  for (int z = 0; z < nslots; ++z) {
    __syncthreads();  // the previous slot's reads of s are done
    int idx[kMaxE];
#pragma unroll
    for (int i = 0; i < kMaxE; ++i) {
      const int e = threadIdx.x + 256 * i;
      idx[i] = nidx[i];
      if (i < ne && e < nel) s[e] = nx[i];
    }
    if (z + 1 < nslots) fetch(z + 1);
    lds_fwht(s, l0.lgdk1, 4);
#pragma unroll
    for (int i = 0; i < kMaxE; ++i) {
      const int e = threadIdx.x + 256 * i;
      if (i < ne && e < nel) acc[i] += s[idx[i]];
    }
  }
  float *o = out + (b_begin + v) * (int64_t)R * 1024 + cb * 16;
#pragma unroll
  for (int i = 0; i < kMaxE; ++i) {
    const int e = threadIdx.x + 256 * i;
    if (i < ne && e < nel) {
      float *d = o + (int64_t)(e >> 4) * 1024 + (e & 15);
      *d = accumulate ? *d + acc[i] * rs : acc[i] * rs;
    }
  }
}

bool affd_small_path(const sk_sketch *s, int layer) {
  const LayerDesc &ld = s->layers[layer];
  return s->D > 1024 && ld.K == 2 && ld.L == 1024 && ld.np == s->D && ld.dk1 >= 2 && ld.dk1 <= kSmallMaxDk1 &&
         ld.rows_live <= kSmallRows;
}

int64_t affd_small_bytes_per_vector(const sk_sketch *s) { return 2 * s->D * 4; }

void run_affd_small(const sk_sketch *s, const SmallGroup &g, int nslots, int dtype, int64_t b_begin, int64_t bc,
                    int phases, float *out, bool accumulate, hipStream_t st) {
  if (nslots <= 0 || bc <= 0) return;
  const int64_t D = s->D;
  const int R = (int)(D / 1024);
  const int64_t wslot = bc * D;  // floats of W (and of F) per slot
  float *w = s->ws;
  float *f = w + nslots * wslot;
  const unsigned zs = (unsigned)nslots;
  if (phases & 1) {
    if (dtype == SK_BF16)
      hipLaunchKernelGGL(k_affdS_rows<true>, dim3(kSmallRows, (unsigned)((bc + 7) / 8), zs), dim3(256), 0, st,
                         s->d_layers, s->d_ptab, g, b_begin, bc, w, wslot, s->key);
    else
      hipLaunchKernelGGL(k_affdS_rows<false>, dim3(kSmallRows, (unsigned)((bc + 7) / 8), zs), dim3(256), 0, st,
                         s->d_layers, s->d_ptab, g, b_begin, bc, w, wslot, s->key);
  }
  if (!(phases & 2)) return;
  const int dk1 = s->layers[g.layer[0]].dk1;  // = R for every slot (N' = D)
  if (s->d_gsmall && dk1 % 8 == 0)
    hipLaunchKernelGGL(k_affdS_top8, dim3((unsigned)(R / 8), (unsigned)bc, zs), dim3(256), 0, st, s->d_layers,
                       s->d_ptab, g, w, wslot, f);
  else
    hipLaunchKernelGGL(k_affdS_top, dim3((unsigned)R, (unsigned)((bc + 7) / 8), zs), dim3(256), 0, st, s->d_layers,
                       s->d_ptab, g, bc, w, wslot, f, s->key);
  if (dk1 == 64) {
    hipLaunchKernelGGL(k_affdS_cols64, dim3(32u, (unsigned)bc), dim3(256), 0, st, s->d_layers, s->d_ptab, g, nslots, f,
                       wslot, b_begin, out, (int)accumulate);
    (void)hipGetLastError();
    return;
  }
#define SK_SCOLS(E)                                                                                           \
  hipLaunchKernelGGL(k_affdS_cols<E>, dim3(64u, (unsigned)bc), dim3(256), 0, st, s->d_layers, s->d_ptab, g, nslots, f, \
                     wslot, R, b_begin, out, (int)accumulate)
  switch (R <= 16 ? 1 : R / 16) {
    case 1: SK_SCOLS(1); break;
    case 2: SK_SCOLS(2); break;
    case 4: SK_SCOLS(4); break;
    case 8: SK_SCOLS(8); break;
    case 16: SK_SCOLS(16); break;
    default: SK_SCOLS(32); break;
  }
#undef SK_SCOLS
  (void)hipGetLastError();
}

}  // namespace sk
