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
  hipLaunchKernelGGL(k_affdS_top, dim3((unsigned)R, (unsigned)((bc + 7) / 8), zs), dim3(256), 0, st, s->d_layers,
                     s->d_ptab, g, bc, w, wslot, f, s->key);
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
