// sk_affd_t.hip -- AFFD (eq. bami) for layers whose second-to-last Kronecker
// digit has 1024 values (padded length N' = TT 2^20, TT <= 64) and D > 1024.
//
// Coordinates of a layer are (t, p, l): top digits t (TT values), digit p
// (1024), last digit l (1024).  With w = Scatter_pi1(B x) and h* the top
// digits of pi2(0),
//   AFFD(x)[a 1024 + b] = sqrt(N'/D) (H_p (x) H_l F)[pi2_p(a), pi2_l(b)],
//   F[p, l] = sum_t H_TT[h*, t] g[t, p, l] ((H_TT (x) H_p (x) H_l) w)[t, p, l].
// Each slab t of w is written transposed, W^T[t][l][p], so that every
// transform along p runs over contiguous memory:
//   A  16 destination rows per workgroup: load, sign, pi1 on the columns,
//      H_l, write 16 consecutive p of every column l            -> W^T
//   B  (TT > 8 only) H_p along each W^T row                    -> W^T
//   C  per column l: H_p (TT <= 8), H_TT in registers, x g, signed sum onto
//      h*, H_p again, keep the rows pi2_p(a), a < R             -> G^T[l][a]
//   E  H_l along each row a of G, gather pi2_l(b), scale, add  -> out
// Three passes over the data (read x, write W^T, read W^T) for TT <= 8.
#include <algorithm>
#include <cstdlib>

#include "sk_kcommon.h"
#include "sk_launch.h"

namespace sk {

namespace {

__device__ __forceinline__ int64_t src_slab_t(const LayerDesc &ld, const uint16_t *ptab, int64_t t) {
  int64_t s = 0, stride = 1;
  for (int k = ld.K - 3; k >= 0; --k) {
    const int64_t dig = (t / stride) & ((1ll << ld.lg[k]) - 1);
    s += (int64_t)ptab[ld.poff[0][1][k] + dig] * stride;
    stride <<= ld.lg[k];
  }
  return s;
}

__device__ __forceinline__ void masks_t(const LayerDesc &ld, const uint16_t *ptab, int tt, uint64_t &live,
                                        uint64_t &sgn) {
  live = 0;
  sgn = 0;
  for (int t = 0; t < tt; ++t) {
    if (src_slab_t(ld, ptab, t) * 1024 < ld.rows_live) live |= 1ull << t;
    sgn |= (uint64_t)(__popc((uint32_t)t & ld.hstar) & 1u) << t;
  }
}

}  // namespace

// ---- A ---------------------------------------------------------------------
// Persistent: gridDim.x (a multiple of 8) workgroups walk the live tiles
// (vector, slab t, 16 destination rows p0..p0+15).  Workgroup b runs on XCD
// b mod 8; the tile map gives each XCD a contiguous range per sweep, so one
// XCD writes all 64 tiles of a slab and its W^T lines are completed in one L2.
// The 16 row loads of the next tile are issued before the transform of the
// current one; the row tables live in LDS so no load waits on another.
namespace {
struct RowTile {
  int64_t v, t, p0;
};

__device__ __forceinline__ RowTile decode_tile(int64_t tile, int64_t per_v, uint64_t live) {
  RowTile r;
  r.v = tile / per_v;
  const int64_t rem = tile - r.v * per_v;
  const int sl = (int)(rem >> 6);
  r.p0 = (rem & 63) * 16;
  uint64_t m = live;
  for (int i = 0; i < sl; ++i) m &= m - 1;
  r.t = __builtin_ctzll(m);
  return r;
}

template <bool BF16, bool VEC>
__device__ __forceinline__ void load_rows16(const LayerDesc &ld, const uint16_t *s_invp, int64_t sslab, int64_t p0,
                                            const void *x, int64_t xrow, int col0, float (&val)[16][4]) {
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int64_t h = sslab * 1024 + s_invp[p0 + i];
    const int64_t j0 = h * 1024 + col0;
    const int64_t lim = ld.n - j0;
#pragma unroll
    for (int q = 0; q < 4; ++q) val[i][q] = 0.0f;
    if (h < ld.rows_live && lim > 0) load4<BF16, VEC>(x, xrow * ld.n + j0, lim, val[i]);
  }
}

}  // namespace

template <bool BF16, bool VEC>
__global__ __launch_bounds__(256) void k_affdT_rows(const LayerDesc *__restrict__ layers,
                                                    const uint16_t *__restrict__ ptab, int layer,
                                                    const void *__restrict__ x, int64_t b_begin, int64_t bc,
                                                    float *__restrict__ w, Key key) {
  using L = Lds1024R;
  __shared__ __align__(16) float s[L::kFloats];
  __shared__ __align__(16) uint32_t sg[16 * 32];
  __shared__ uint16_t s_invp[1024];
  __shared__ int32_t s_slab[64];
  const LayerDesc &ld = layers[layer];
  const int TT = 1 << (ld.lgnp - 20);
  const uint16_t *invp = ptab + ld.poff[0][1][ld.K - 2];
  for (int e = threadIdx.x; e < 1024; e += 256) s_invp[e] = invp[e];
  if (threadIdx.x < TT) s_slab[threadIdx.x] = (int32_t)src_slab_t(ld, ptab, threadIdx.x);
  __syncthreads();
  uint64_t live = 0;
  for (int t = 0; t < TT; ++t)
    if ((int64_t)s_slab[t] * 1024 < ld.rows_live) live |= 1ull << t;
  const int64_t per_v = (int64_t)__popcll(live) * 64;
  const int64_t ntiles = bc * per_v;
  const int64_t G = gridDim.x;
  int64_t tile = (int64_t)(blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3);
  if (tile >= ntiles) return;  // uniform over the workgroup
  const int64_t lo_len = 1ll << 20;
  const uint16_t *fk = ptab + ld.poff[0][0][ld.K - 1];
  const int col0 = threadIdx.x * 4;
  int pc[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) pc[q] = fk[col0 + q];
  RowTile cur = decode_tile(tile, per_v, live);
  int64_t sslab = s_slab[cur.t];
  float val[16][4];
  load_rows16<BF16, VEC>(ld, s_invp, sslab, cur.p0, x, b_begin + cur.v, col0, val);
  const int ri = threadIdx.x & 15, rc = threadIdx.x >> 4;  // transform: row ri, column group rc
  for (;;) {
    __syncthreads();  // the previous tile's reads of s and sg are done
    // sign words of the 16 rows: 8 Philox blocks of 128 signs per row, one per
    // thread of the first half, shared through LDS (word index = col0 / 32)
    if (threadIdx.x < 128) {
      const int i = threadIdx.x >> 3;
      const int64_t h = sslab * 1024 + s_invp[cur.p0 + i];
      const W4 q = philox((uint64_t)(h * 8 + (threadIdx.x & 7)), (uint32_t)ld.layer_id, ST_SIGN, key);
      *(uint4 *)(sg + 4 * threadIdx.x) = make_uint4(q.w[0], q.w[1], q.w[2], q.w[3]);
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const uint32_t bits = sg[i * 32 + (threadIdx.x >> 3)] >> (col0 & 31);
#pragma unroll
      for (int q = 0; q < 4; ++q) s[L::idx(i, pc[q])] = flip(val[i][q], (bits >> q) & 1u);
    }
    // prefetch the next tile into the registers just consumed
    const int64_t ntile = tile + G;
    const bool more = ntile < ntiles;
    RowTile nxt = cur;
    int64_t nslab = sslab;
    if (more) {
      nxt = decode_tile(ntile, per_v, live);
      nslab = s_slab[nxt.t];
      load_rows16<BF16, VEC>(ld, s_invp, nslab, nxt.p0, x, b_begin + nxt.v, col0, val);
    }
    __syncthreads();
    // H_l (unnormalised; the 1/32 is applied by the readers of W^T)
    float e[64];
    fwht1024_rows16_r(s, e);
    float *dst = w + cur.v * ld.np + cur.t * lo_len + (int64_t)(64 * rc) * 1024 + cur.p0 + ri;
#pragma unroll
    for (int m = 0; m < 64; ++m) dst[(int64_t)m * 1024] = e[m];
    if (!more) break;
    tile = ntile;
    cur = nxt;
    sslab = nslab;
  }
}

// ---- B (TT > 8) --------------------------------------------------------------
__global__ __launch_bounds__(256) void k_affdT_prow(const LayerDesc *__restrict__ layers,
                                                    const uint16_t *__restrict__ ptab, int layer,
                                                    float *__restrict__ w) {
  using L = Lds1024<16>;
  __shared__ __align__(16) float s[L::kFloats];
  const LayerDesc &ld = layers[layer];
  const int64_t row0 = (int64_t)blockIdx.x * 16;  // rows (t, l) of W^T
  const int64_t t = row0 >> 10;
  const int64_t v = blockIdx.y;
  if (src_slab_t(ld, ptab, t) * 1024 >= ld.rows_live) return;
  float *base = w + v * ld.np + row0 * 1024;
  // row i = tid / 16 holds columns c + 16 k
  float e[64];
  {
    const float *src = base + (threadIdx.x >> 4) * 1024 + (threadIdx.x & 15);
#pragma unroll
    for (int k = 0; k < 64; ++k) e[k] = src[16 * k];
  }
  fwht1024_lds_regs<16>(s, e);
  const float sc = 1.0f / 1024.0f;  // H_p here and H_l of phase A
#pragma unroll
  for (int i = 0; i < 16; ++i)
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int p = threadIdx.x + 256 * k;
      base[i * 1024 + p] = s[L::idx(i, p)] * sc;
    }
}

// ---- C ---------------------------------------------------------------------
// Shared ending: F rows (one per vector, p = tid + 256 k in f[v][k]) -> H_p ->
// G^T[v][l][a] = value at p = pi2_p(a), a < R (R consecutive floats per l).
template <int VB>
__device__ __forceinline__ void affdT_finish(const LayerDesc &ld, const uint16_t *ptab, float (&f)[VB][4],
                                             float *lds, int64_t l, int64_t v0, int nv, int R, float sc,
                                             float *__restrict__ gout) {
  using L = Lds1024<VB>;
  __syncthreads();
#pragma unroll
  for (int v = 0; v < VB; ++v)
#pragma unroll
    for (int k = 0; k < 4; ++k) lds[L::idx(v, threadIdx.x + 256 * k)] = f[v][k];
  __syncthreads();
  fwht1024_lds<VB>(lds);
  const uint16_t *p2 = ptab + ld.poff[1][0][ld.K - 2];
  for (int e = threadIdx.x; e < VB * R; e += 256) {
    const int v = e / R, a = e - (e / R) * R;
    if (v < nv) gout[((v0 + v) * 1024 + l) * R + a] = lds[L::idx(v, p2[a])] * sc;
  }
}

// TT <= 8: with M = H_TT (s . g) (formed once per column from the Gaussians),
// sum_t s(t) g[t] (H_TT x)[t] = sum_t' M[t'] x[t'], so the TT slab rows of a
// vector are taken one at a time: H_p of row t' for VB vectors at once, then
// acc += M[t'] x.  The Gaussians of a column are generated once per VB vectors.
template <int TT, int VB>
__global__ __launch_bounds__(256) void k_affdT_top(const LayerDesc *__restrict__ layers,
                                                   const uint16_t *__restrict__ ptab, int layer,
                                                   const float *__restrict__ w, int64_t bc, int R,
                                                   float *__restrict__ gout, Key key) {
  using L = Lds1024<VB>;
  __shared__ __align__(16) float lds[L::kFloats];
  const LayerDesc &ld = layers[layer];
  const int64_t lo_len = 1ll << 20;
  const int64_t l = blockIdx.x;
  const int64_t v0 = (int64_t)blockIdx.y * VB;
  const int nv = (int)((bc - v0) < VB ? (bc - v0) : VB);
  uint64_t live, sgn;
  masks_t(ld, ptab, TT, live, sgn);
  float m[4][TT];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int64_t p = threadIdx.x + 256 * k;
#pragma clang loop unroll(full)
    for (int t = 0; t < TT; ++t)
      m[k][t] = flip(gauss((uint64_t)(t * lo_len + p * 1024 + l), (uint32_t)ld.layer_id, ST_GAUSS, key),
                     (uint32_t)(sgn >> t) & 1u);
    fwht_regs_t<TT>(m[k]);
  }
  float f[VB][4];
#pragma unroll
  for (int v = 0; v < VB; ++v)
#pragma unroll
    for (int k = 0; k < 4; ++k) f[v][k] = 0.0f;
#pragma unroll
  for (int t = 0; t < TT; ++t) {
    if (!((live >> t) & 1ull)) continue;  // uniform: all-zero slab
    // row v = tid / C of the block holds columns c + C k (C = 256 / VB)
    constexpr int C = 256 / VB, E = 4 * VB;
    float e[E];
    {
      const int v = threadIdx.x / C;
      const float *src = w + (v0 + v) * ld.np + t * lo_len + l * 1024 + (threadIdx.x % C);
#pragma unroll
      for (int k = 0; k < E; ++k) e[k] = v < nv ? src[C * k] : 0.0f;
    }
    __syncthreads();  // the previous slab row's reads of lds are done
    fwht1024_lds_regs<VB>(lds, e);
#pragma unroll
    for (int v = 0; v < VB; ++v)
#pragma unroll
      for (int k = 0; k < 4; ++k) f[v][k] += m[k][t] * lds[L::idx(v, threadIdx.x + 256 * k)];
  }
  // H_l of phase A, H_p twice (1/32 each) and H_TT (1/TT)
  affdT_finish<VB>(ld, ptab, f, lds, l, v0, nv, R, 1.0f / (32768.0f * (float)TT), gout);
}

// TT in {16, 32, 64}: W^T rows already carry H_p (phase B); one p per thread and
// pass, TT Gaussians in registers.
template <int TT, int VB>
__global__ __launch_bounds__(256, 1) void k_affdT_top_wide(const LayerDesc *__restrict__ layers,
                                                        const uint16_t *__restrict__ ptab, int layer,
                                                        const float *__restrict__ w, int64_t bc, int R,
                                                        float *__restrict__ gout, Key key) {
  using L = Lds1024<VB>;
  __shared__ __align__(16) float lds[L::kFloats];
  const LayerDesc &ld = layers[layer];
  const int64_t lo_len = 1ll << 20;
  const int64_t l = blockIdx.x;
  const int64_t v0 = (int64_t)blockIdx.y * VB;
  const int nv = (int)((bc - v0) < VB ? (bc - v0) : VB);
  uint64_t live, sgn;
  masks_t(ld, ptab, TT, live, sgn);
  float f[VB][4];
#pragma unroll 1
  for (int k = 0; k < 4; ++k) {
    const int64_t p = threadIdx.x + 256 * k;
    // M = H_TT (s . g) once per column (see k_affdT_top)
    float m[TT];
#pragma clang loop unroll(full)
    for (int t = 0; t < TT; ++t)
      m[t] = flip(gauss((uint64_t)(t * lo_len + p * 1024 + l), (uint32_t)ld.layer_id, ST_GAUSS, key),
                  (uint32_t)(sgn >> t) & 1u);
    fwht_regs_t<TT>(m);
#pragma unroll 1
    for (int v = 0; v < VB; ++v) {
      float acc = 0.0f;
      if (v < nv) {
        const float *wv = w + (v0 + v) * ld.np + l * 1024 + p;
        // 16 loads in flight at a time keeps the address registers bounded
#pragma clang loop unroll(full)
        for (int t0 = 0; t0 < TT; t0 += 16) {
          float xv[16];
#pragma unroll
          for (int t = 0; t < 16; ++t) xv[t] = ((live >> (t0 + t)) & 1ull) ? wv[(t0 + t) * lo_len] : 0.0f;
#pragma unroll
          for (int t = 0; t < 16; ++t) acc += m[t0 + t] * xv[t];
        }
      }
      lds[L::idx(v, (int)p)] = acc;
    }
  }
  __syncthreads();
#pragma unroll
  for (int v = 0; v < VB; ++v)
#pragma unroll
    for (int k = 0; k < 4; ++k) f[v][k] = lds[L::idx(v, threadIdx.x + 256 * k)];
  // H_p was applied by phase B; H_TT (1/TT) and H_p (1/32) here
  affdT_finish<VB>(ld, ptab, f, lds, l, v0, nv, R, 1.0f / (32.0f * (float)TT), gout);
}

// ---- C with a stored M --------------------------------------------------------
// M[t'][l][p] = (H_TT (c . g[., p, l]))[t'], c_t = (-1)^<h*, t>, written once
// per sketch: thread per (p, l) with p fastest so the TT rows are coalesced.
template <int TT>
__global__ __launch_bounds__(256) void k_affd_mtab(const LayerDesc *__restrict__ layers, int layer,
                                                   float *__restrict__ m, Key key) {
  const LayerDesc &ld = layers[layer];
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;  // < 2^20
  const int64_t p = q & 1023, l = q >> 10;
  const int64_t lo_len = 1ll << 20;
  float v[TT];
#pragma clang loop unroll(full)
  for (int t = 0; t < TT; ++t)
    v[t] = flip(gauss((uint64_t)(t * lo_len + p * 1024 + l), (uint32_t)ld.layer_id, ST_GAUSS, key),
                (uint32_t)__popc((uint32_t)t & ld.hstar) & 1u);
  fwht_regs_t<TT>(v);
#pragma clang loop unroll(full)
  for (int t = 0; t < TT; ++t) m[t * lo_len + l * 1024 + p] = v[t];
}

// Any TT <= 64 with M stored: per live slab row t of the column l, H_p of the
// VB vectors' rows (fed from global memory in the first pass's layout), then
// acc += M[t][l][p] x.  No Gaussians are generated and W^T is read once.
template <int VB>
__global__ __launch_bounds__(256) void k_affdT_topM(const LayerDesc *__restrict__ layers,
                                                    const uint16_t *__restrict__ ptab, int layer,
                                                    const float *__restrict__ w, int64_t bc, int R,
                                                    const float *__restrict__ mt, float *__restrict__ gout) {
  using L = Lds1024<VB>;
  __shared__ __align__(16) float lds[L::kFloats];
  const LayerDesc &ld = layers[layer];
  const int TT = 1 << (ld.lgnp - 20);
  const int64_t lo_len = 1ll << 20;
  const int64_t l = blockIdx.x;
  const int64_t v0 = (int64_t)blockIdx.y * VB;
  const int nv = (int)((bc - v0) < VB ? (bc - v0) : VB);
  uint64_t live, sgn;
  masks_t(ld, ptab, TT, live, sgn);
  constexpr int C = 256 / VB, E = 4 * VB;
  const int vr = threadIdx.x / C;
  const float *src = w + (v0 + vr) * ld.np + l * 1024 + (threadIdx.x % C);
  const float *mcol = mt + l * 1024 + threadIdx.x;
  float f[VB][4];
#pragma unroll
  for (int v = 0; v < VB; ++v)
#pragma unroll
    for (int k = 0; k < 4; ++k) f[v][k] = 0.0f;
  // the loads of the next live slab row are issued before the transform of
  // the current one
  float e[E], mm[4];
  auto fetch = [&](int t) {
#pragma unroll
    for (int k = 0; k < E; ++k) e[k] = vr < nv ? src[t * lo_len + C * k] : 0.0f;
#pragma unroll
    for (int k = 0; k < 4; ++k) mm[k] = mcol[t * lo_len + 256 * k];
  };
  uint64_t rest = live;  // never empty: slab 0 holds source row 0
  int t = __builtin_ctzll(rest);
  rest &= rest - 1;
  fetch(t);
#pragma unroll 1
  for (;;) {
    float ec[E], mc[4];
#pragma unroll
    for (int k = 0; k < E; ++k) ec[k] = e[k];
#pragma unroll
    for (int k = 0; k < 4; ++k) mc[k] = mm[k];
    const bool more = rest != 0;
    if (more) {
      t = __builtin_ctzll(rest);
      rest &= rest - 1;
      fetch(t);
    }
    __syncthreads();  // the previous slab row's reads of lds are done
    fwht1024_lds_regs<VB>(lds, ec);
#pragma unroll
    for (int v = 0; v < VB; ++v)
#pragma unroll
      for (int k = 0; k < 4; ++k) f[v][k] += mc[k] * lds[L::idx(v, threadIdx.x + 256 * k)];
    if (!more) break;
  }
  // H_l of phase A, H_p twice (1/32 each) and H_TT (1/TT)
  affdT_finish<VB>(ld, ptab, f, lds, l, v0, nv, R, 1.0f / (32768.0f * (float)TT), gout);
}

void launch_affd_mtab(const sk_sketch *s, int layer, float *m, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const dim3 grid(1u << 12);  // 2^20 (p, l) pairs
  switch (ld.lgnp - 20) {
    case 0: hipLaunchKernelGGL(k_affd_mtab<1>, grid, dim3(256), 0, st, s->d_layers, layer, m, s->key); break;
    case 1: hipLaunchKernelGGL(k_affd_mtab<2>, grid, dim3(256), 0, st, s->d_layers, layer, m, s->key); break;
    case 2: hipLaunchKernelGGL(k_affd_mtab<4>, grid, dim3(256), 0, st, s->d_layers, layer, m, s->key); break;
    case 3: hipLaunchKernelGGL(k_affd_mtab<8>, grid, dim3(256), 0, st, s->d_layers, layer, m, s->key); break;
    case 4: hipLaunchKernelGGL(k_affd_mtab<16>, grid, dim3(256), 0, st, s->d_layers, layer, m, s->key); break;
    case 5: hipLaunchKernelGGL(k_affd_mtab<32>, grid, dim3(256), 0, st, s->d_layers, layer, m, s->key); break;
    case 6: hipLaunchKernelGGL(k_affd_mtab<64>, grid, dim3(256), 0, st, s->d_layers, layer, m, s->key); break;
    default: break;
  }
  (void)hipGetLastError();
}

// ---- E ---------------------------------------------------------------------
// One workgroup per (vector, block of 16 values of a): reads G^T[v][l][a0..a0+15]
// for every l (64-byte pieces), transposes through LDS, H_l, gathers pi2_l.
__global__ __launch_bounds__(256) void k_affdT_out(const LayerDesc *__restrict__ layers,
                                                   const uint16_t *__restrict__ ptab, int layer,
                                                   const float *__restrict__ gin, int R, int64_t D, int64_t b_begin,
                                                   float *__restrict__ out, int accumulate) {
  using L = Lds1024<16>;
  __shared__ __align__(16) float s[L::kFloats];
  const LayerDesc &ld = layers[layer];
  const int a0 = blockIdx.x * 16;
  const int na = (R - a0) < 16 ? (R - a0) : 16;
  const int64_t v = blockIdx.y;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int l = threadIdx.x + 256 * k;
    const float *src = gin + (v * 1024 + l) * R + a0;
#pragma unroll
    for (int i = 0; i < 16; ++i) s[L::idx(i, l)] = i < na ? src[i] : 0.0f;
  }
  __syncthreads();
  fwht1024_lds<16>(s);
  const uint16_t *p2l = ptab + ld.poff[1][0][ld.K - 1];
  const float sc = (float)(sqrt((double)ld.np / (double)D) / 32.0);
  for (int i = 0; i < na; ++i) {
    float *o = out + (b_begin + v) * D + (int64_t)(a0 + i) * 1024;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int b = threadIdx.x + 256 * k;
      const float val = s[L::idx(i, p2l[b])] * sc;
      o[b] = accumulate ? o[b] + val : val;
    }
  }
}

constexpr unsigned kRowsGrid = 512;

// Vectors per call for TT <= 8: a multiple of 8 (the vectors of one phase-C
// workgroup) whose W^T (live slabs x 4 MB per vector) stays within the 256 MB
// memory-side cache between phases A and C, so that the W^T round trip rarely
// reaches HBM.  0 = no preference (TT > 8: W^T is far larger).
int64_t affd_transposed_tile(const sk_sketch *s, int layer) {
  const LayerDesc &ld = s->layers[layer];
  if (!affd_transposed_path(s, layer) || ld.lgnp - 20 > 3) return 0;
  const char *e = std::getenv("SK_AFFD_MALL_MB");
  const int64_t budget = (e ? std::atoll(e) : 192) << 20;
  const int64_t wbytes = ((ld.rows_live + 1023) / 1024) * (4ll << 20);
  return 8 * std::max<int64_t>(1, budget / (8 * wbytes));
}

bool affd_transposed_path(const sk_sketch *s, int layer) {
  const LayerDesc &ld = s->layers[layer];
  if (s->D <= 1024 || ld.K < 2 || ld.L != 1024 || ld.dk1 != 1024) return false;
  const int lgtt = ld.lgnp - 20;
  return lgtt >= 0 && lgtt <= 6;
}

void run_affd_transposed(const sk_sketch *s, int layer, const void *x, int dtype, bool vec, int64_t b_begin,
                         int64_t bc, float *gbuf, int phases, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const int TT = 1 << (ld.lgnp - 20);
  const int R = (int)(s->D / 1024);
  float *w = s->ws;
  if (phases & 1) {  // A
    // two resident workgroups per CU (64 KB of LDS each); a multiple of 8
    const dim3 grid(kRowsGrid);
#define SK_AROWS(BF, VE)                                                                                  \
  hipLaunchKernelGGL((k_affdT_rows<BF, VE>), grid, dim3(256), 0, st, s->d_layers, s->d_ptab, layer, x, b_begin, \
                     bc, w, s->key)
    if (dtype == SK_BF16) {
      if (vec) SK_AROWS(true, true); else SK_AROWS(true, false);
    } else {
      if (vec) SK_AROWS(false, true); else SK_AROWS(false, false);
    }
#undef SK_AROWS
  }
  if (!(phases & 2)) return;
  if (s->d_mtab && s->mtab_off[layer] >= 0) {
    hipLaunchKernelGGL(k_affdT_topM<8>, dim3(1024u, (unsigned)((bc + 7) / 8)), dim3(256), 0, st, s->d_layers,
                       s->d_ptab, layer, w, bc, R, s->d_mtab + s->mtab_off[layer], gbuf);
    (void)hipGetLastError();
    return;
  }
  // B, C
  if (TT > 8) {
    dim3 gb((unsigned)((int64_t)TT * 1024 / 16), (unsigned)bc);
    hipLaunchKernelGGL(k_affdT_prow, gb, dim3(256), 0, st, s->d_layers, s->d_ptab, layer, w);
  }
  {
#define SK_CT(T, VB)                                                                                          \
  case T:                                                                                                     \
    hipLaunchKernelGGL((k_affdT_top<T, VB>), dim3(1024u, (unsigned)((bc + VB - 1) / VB)), dim3(256), 0, st,   \
                       s->d_layers, s->d_ptab, layer, w, bc, R, gbuf, s->key);                                \
    break;
#define SK_CTW(T, VB)                                                                                         \
  case T:                                                                                                     \
    hipLaunchKernelGGL((k_affdT_top_wide<T, VB>), dim3(1024u, (unsigned)((bc + VB - 1) / VB)), dim3(256), 0,  \
                       st, s->d_layers, s->d_ptab, layer, w, bc, R, gbuf, s->key);                            \
    break;
    switch (TT) {
      SK_CT(1, 16) SK_CT(2, 16) SK_CT(4, 16) SK_CT(8, 16) SK_CTW(16, 8) SK_CTW(32, 8) SK_CTW(64, 8)
      default: break;
    }
#undef SK_CT
#undef SK_CTW
  }
  (void)hipGetLastError();
}

void run_affd_transposed_out(const sk_sketch *s, int layer, const float *gbuf, int64_t b_begin, int64_t gb,
                             float *out, bool accumulate, hipStream_t st) {
  const int R = (int)(s->D / 1024);
  hipLaunchKernelGGL(k_affdT_out, dim3((unsigned)((R + 15) / 16), (unsigned)gb), dim3(256), 0, st, s->d_layers,
                     s->d_ptab, layer, gbuf, R, s->D, b_begin, out, (int)accumulate);
  (void)hipGetLastError();
}

}  // namespace sk
