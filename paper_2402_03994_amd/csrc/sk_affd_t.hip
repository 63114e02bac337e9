// sk_affd_t.hip -- AFFD (eq. bami) for layers whose second-to-last Kronecker
// digit has 1024 values (padded length N' = TT 2^20, TT <= 64) and D > 1024.
//
// Coordinates of a layer are (t, p, l): top digits t (TT values), digit p
// (1024), last digit l (1024).  With w = Scatter_pi1(B x) and h* the top
// digits of pi2(0),
//   AFFD(x)[a 1024 + b] = sqrt(N'/D) (H_p (x) H_l F)[pi2_p(a), pi2_l(b)],
//   F[p, l] = sum_t H_TT[h*, t] g[t, p, l] ((H_TT (x) H_p (x) H_l) w)[t, p, l].
// Each slab t of w is written transposed, so that every transform along p
// runs over contiguous memory: W^T[t][l][p] (slab after slab) or, with the
// stored M tables, W^T[l][t][p] over the live slabs only (a column's slabs
// one after the other, which C reads in that order):
//   A  16 destination rows per workgroup: load, sign, pi1 on the columns,
//      H_l, write 16 consecutive p of every column l            -> W^T
//   C  per column l, with the stored M = H_TT (s . g): for each live slab
//      H_p and F += M[t] x; then H_p again, keep the rows pi2_p(a), a < R
//                                                               -> G^T[l][a]
//   E  for all the layers of a call at once: H_l along each row a of G,
//      gather pi2_l(b), scale, sum, write                     -> out
// Three passes over the data: read x, write W^T, read W^T.  Without the
// stored tables C regenerates g (TT <= 8: H_TT in registers; TT > 8: phase B
// applies H_p along each W^T row first).
#include <algorithm>
#include <cstdlib>
#include <cmath>

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
// The row loads of the next tile are issued before the transform of the
// current one; the row tables live in LDS so no load waits on another.
namespace {
struct RowTile {
  int64_t v, t, p0;
  int sl;  // index of slab t among the group's live slabs
};

// Tiles of one vector: 32 per live slab of the group (live slabs s_first ..
// s_first + nsl - 1 in increasing t).
__device__ __forceinline__ RowTile decode_tile(int64_t tile, int64_t per_v, uint64_t live, int s_first) {
  RowTile r;
  r.v = tile / per_v;
  const int64_t rem = tile - r.v * per_v;
  r.sl = (int)(rem >> 5);
  r.p0 = (rem & 31) * 32;
  uint64_t m = live;
  for (int i = 0; i < s_first + r.sl; ++i) m &= m - 1;
  r.t = __builtin_ctzll(m);
  return r;
}

// Rows 4k + quarter (k < 8) of a tile: thread column col0..col0+3.  General
// form: any alignment and length.
template <bool BF16>
__device__ __forceinline__ void load_rows8(const LayerDesc &ld, const uint16_t *s_invp, int64_t sslab, int64_t p0,
                                           int quarter, const void *x, int64_t xrow, int col0, float (&val)[8][4]) {
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int64_t h = sslab * 1024 + s_invp[p0 + 4 * k + quarter];
    const int64_t j0 = h * 1024 + col0;
    const int64_t lim = ld.n - j0;
#pragma unroll
    for (int q = 0; q < 4; ++q) val[k][q] = 0.0f;
    if (h < ld.rows_live && lim > 0) load4<BF16, false>(x, xrow * ld.n + j0, lim, val[k]);
  }
}

// Same rows through a buffer resource over the vector's n elements (n a
// multiple of 4, n elt < 2^31): the row index is uniform over the wave, so
// rows without data are skipped by a scalar branch and the end of the last
// row is zero-filled by the hardware range check (the whole byte offset is in
// the vector operand, which the check covers).  The loads carry the non-temporal
// hint: the input is read once, and keeping it out of the caches leaves more
// of the memory-side cache to the transposed slabs the next kernel reads
// (measured 3% faster on this kernel).
template <bool BF16>
__device__ __forceinline__ void load_rows8_buf(const LayerDesc &ld, const uint16_t *s_invp, int sslab, int p0,
                                               int quarter, __amdgpu_buffer_rsrc_t rs, int voff, float (&val)[8][4]) {
  typedef unsigned int u4 __attribute__((ext_vector_type(4)));
  typedef unsigned int u2 __attribute__((ext_vector_type(2)));
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int h = __builtin_amdgcn_readfirstlane(sslab * 1024 + (int)s_invp[p0 + 4 * k + quarter]);
    if (h < ld.rows_live) {
      if (BF16) {
        const u2 u = __builtin_amdgcn_raw_buffer_load_b64(rs, voff + h * 2048, 0, kNt);
        val[k][0] = __uint_as_float(u.x << 16);
        val[k][1] = __uint_as_float(u.x & 0xFFFF0000u);
        val[k][2] = __uint_as_float(u.y << 16);
        val[k][3] = __uint_as_float(u.y & 0xFFFF0000u);
      } else {
        const u4 u = __builtin_amdgcn_raw_buffer_load_b128(rs, voff + h * 4096, 0, kNt);
        val[k][0] = __uint_as_float(u.x);
        val[k][1] = __uint_as_float(u.y);
        val[k][2] = __uint_as_float(u.z);
        val[k][3] = __uint_as_float(u.w);
      }
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) val[k][q] = 0.0f;
    }
  }
}

}  // namespace

// 1024 threads per workgroup (one per CU), tiles of 32 destination rows:
// thread tid loads columns col0 = 4 (tid % 256) .. col0 + 3 of tile rows
// 4k + tid / 256 and ends holding 32 columns of one row after the transform;
// W^T is written through a buffer resource whose offsets are scalar
// constants, 32 threads x 4 bytes = one 128-byte line per column (64-byte
// pieces write at about two thirds of the rate).
// W^T of the tile's slab with group index sl (slab t) of vector v starts at
// w + v vstride + (compact ? sl : t) 2^20.
template <bool BF16, bool VEC>
__global__ __launch_bounds__(1024) void k_affdT_rows(const LayerDesc *__restrict__ layers,
                                                    const uint16_t *__restrict__ ptab, int layer,
                                                    const void *__restrict__ x, int64_t b_begin, int64_t bc,
                                                    float *__restrict__ w, int s_first, int nsl, int64_t vstride,
                                                    int compact, Key key) {
  using L = Lds1024R32;
  __shared__ __align__(16) float s[L::kFloats];
  __shared__ __align__(16) uint32_t sg[32 * 32];
  __shared__ uint16_t s_invp[1024];
  __shared__ int32_t s_slab[64];
  const LayerDesc &ld = layers[layer];
  const int TT = 1 << (ld.lgnp - 20);
  const uint16_t *invp = ptab + ld.poff[0][1][ld.K - 2];
  s_invp[threadIdx.x] = invp[threadIdx.x];
  if (threadIdx.x < TT) s_slab[threadIdx.x] = (int32_t)src_slab_t(ld, ptab, threadIdx.x);
  __syncthreads();
  uint64_t live = 0;
  for (int t = 0; t < TT; ++t)
    if ((int64_t)s_slab[t] * 1024 < ld.rows_live) live |= 1ull << t;
  const int64_t per_v = (int64_t)nsl * 32;
  const int64_t ntiles = bc * per_v;
  const int64_t G = gridDim.x;
  int64_t tile = (int64_t)(blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3);
  if (tile >= ntiles) return;  // uniform over the workgroup
  const int64_t lo_len = 1ll << 20;
  const uint16_t *fk = ptab + ld.poff[0][0][ld.K - 1];
  const int quarter = threadIdx.x >> 8;  // uniform over each wave
  const int col0 = (threadIdx.x & 255) * 4;
  const int elt = BF16 ? 2 : 4;
  int pc[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) pc[q] = fk[col0 + q];
  RowTile cur = decode_tile(tile, per_v, live, s_first);
  int64_t sslab = s_slab[cur.t];
  float val[8][4];
  auto load = [&](const RowTile &rt, int64_t slab) {
    const int64_t xrow = b_begin + rt.v;
    if (VEC)
      load_rows8_buf<BF16>(ld, s_invp, (int)slab, (int)rt.p0, quarter,
                           buf_rsrc((const char *)x + xrow * ld.n * elt, (uint32_t)(ld.n * elt)), col0 * elt, val);
    else
      load_rows8<BF16>(ld, s_invp, slab, rt.p0, quarter, x, xrow, col0, val);
  };
  load(cur, sslab);
  const int ri = threadIdx.x & 31, rc = threadIdx.x >> 5;  // transform: row ri, columns 32 rc ..
  for (;;) {
    __syncthreads();  // the previous tile's reads of s and sg are done
    // sign words of the 32 rows: 8 Philox blocks of 128 signs per row, one per
    // thread of the first 256, shared through LDS (word index = col0 / 32)
    if (threadIdx.x < 256) {
      const int i = threadIdx.x >> 3;
      const int64_t h = sslab * 1024 + s_invp[cur.p0 + i];
      const W4 q = philox((uint64_t)(h * 8 + (threadIdx.x & 7)), (uint32_t)ld.layer_id, ST_SIGN, key);
      *(uint4 *)(sg + 4 * threadIdx.x) = make_uint4(q.w[0], q.w[1], q.w[2], q.w[3]);
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int i = 4 * k + quarter;
      const uint32_t bits = sg[i * 32 + (col0 >> 5)] >> (col0 & 31);
#pragma unroll
      for (int q = 0; q < 4; ++q) s[L::idx(i, pc[q])] = flip(val[k][q], (bits >> q) & 1u);
    }
    // prefetch the next tile into the registers just consumed
    const int64_t ntile = tile + G;
    const bool more = ntile < ntiles;
    RowTile nxt = cur;
    int64_t nslab = sslab;
    if (more) {
      nxt = decode_tile(ntile, per_v, live, s_first);
      nslab = s_slab[nxt.t];
      load(nxt, nslab);
    }
    __syncthreads();
    // H_l (unnormalised; the 1/32 is applied by the readers of W^T)
    float e[32];
    fwht1024_rows32(s, e);
    // column 32 rc + m, row p0 + ri of the slab: byte (32 rc + m) cstride + 4 (p0 + ri), cstride = 4096
    // bytes ([slab][l][p], one slab after the other) or, compact, vslabs 4096 ([l][slab][p]: a column's
    // slabs contiguous, so the top kernel reads one region per column and vector)
    const __amdgpu_buffer_rsrc_t ws =
        compact ? buf_rsrc(w + cur.v * vstride + cur.sl * 1024 + cur.p0, (uint32_t)((vstride - cur.sl * 1024 - cur.p0) * 4))
                : buf_rsrc(w + cur.v * vstride + cur.t * lo_len + cur.p0, (uint32_t)((lo_len - cur.p0) * 4));
    const uint32_t cstride = compact ? (uint32_t)((vstride >> 20) * 4096) : 4096u;
    const uint32_t soffc = 32u * (uint32_t)rc * cstride + 4u * (uint32_t)ri;
#pragma unroll
    for (int m = 0; m < 32; ++m)
      __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(e[m]), ws, soffc, m * cstride, 0);
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
// Stored-M top kernel, 8 vectors per workgroup.  Thread (i = tid / 32,
// c = tid % 32) loads column c + 32 k (k < 32) of the slab row of vector i
// straight into registers (pass-1 order), and after the LDS exchange holds the
// 32 consecutive columns 32 c .. 32 c + 31, where it applies M (staged in LDS
// once per slab) and accumulates F.  Two register sets alternate between the
// slab being transformed and the next live slab being loaded.
// The slabs are the group's live slabs s_first .. s_first + nsl - 1, stored
// compactly (W^T of group slab j of vector v, column l at w + v vstride + (l vslabs + j) 1024).  A
// layer whose slabs come in several groups carries F between launches in
// facc[v][l][p] (fmode bit 0: start from facc, bit 1: last group, finish).
namespace {
constexpr int kMPad(int p) { return p + 4 * (p >> 5); }  // 16-byte reads of 8 lanes hit 32 banks

// F of vector i at p = 32 c + m in f[m]: second H_p (bits 0..4 in registers,
// bits 5..9 after one LDS exchange), keep the rows pi2_p(a), a < R.
__device__ __forceinline__ void affdT_finish8(const LayerDesc &ld, const uint16_t *ptab, float (&f)[32], float *lds,
                                              int64_t l, int64_t v0, int nv, int R, float sc,
                                              float *__restrict__ gout) {
  using L = Lds1024<8>;
  const int i = threadIdx.x >> 5, c = threadIdx.x & 31;
  fwht_regs_t<32>(f);
  __syncthreads();  // the last slab's readers of lds are done
  float *b2 = lds + i * L::kStride + 33 * c;  // column 32 c + m
#pragma unroll
  for (int m = 0; m < 32; ++m) b2[m] = f[m];
  __syncthreads();
  float *b1 = lds + i * L::kStride + c;  // column c + 32 k
#pragma unroll
  for (int k = 0; k < 32; ++k) f[k] = b1[33 * k];
  fwht_regs_t<32>(f);
#pragma unroll
  for (int k = 0; k < 32; ++k) b1[33 * k] = f[k];
  __syncthreads();
  const uint16_t *p2 = ptab + ld.poff[1][0][ld.K - 2];
  for (int e = threadIdx.x; e < 8 * R; e += 256) {
    const int v = e / R, a = e - (e / R) * R;
    if (v < nv) gout[((v0 + v) * 1024 + l) * R + a] = lds[L::idx(v, p2[a])] * sc;
  }
  __syncthreads();  // the block is free for the workgroup's next item
}
}  // namespace

// Persistent: gridDim.x workgroups walk the items (column l, 8 vectors),
// item = vector group * 1024 + l, workgroup b taking items b, b + G, ...; the
// slab sequence runs on across items, so the first slab of the next item
// loads during the last slab (and the final transform) of the current one.
template <int VB>
__global__ __launch_bounds__(256, 3) void k_affdT_topM(const LayerDesc *__restrict__ layers,
                                                    const uint16_t *__restrict__ ptab, int layer,
                                                    const float *__restrict__ w, int64_t bc, int R,
                                                    const float *__restrict__ mt, int s_first, int nsl,
                                                    int64_t vstride, float *__restrict__ facc, int fmode,
                                                    float *__restrict__ gout) {
  static_assert(VB == 8, "8 vectors per workgroup");
  using L = Lds1024<8>;
  __shared__ __align__(16) float lds[L::kFloats];
  __shared__ __align__(16) float sm[kMPad(1024)];
  __shared__ int32_t s_t[64];  // slab id of group slab j
  const LayerDesc &ld = layers[layer];
  const int TT = 1 << (ld.lgnp - 20);
  const int64_t lo_len = 1ll << 20;
  const int64_t nitems = 1024 * ((bc + 7) / 8);
  const int64_t G = gridDim.x;
  int64_t item = blockIdx.x;
  if (item >= nitems) return;  // uniform over the workgroup
  if (threadIdx.x == 0) {
    uint64_t live, sgn;
    masks_t(ld, ptab, TT, live, sgn);
    uint64_t rest = live;  // never empty: slab 0 holds source row 0
    for (int q = 0; q < s_first; ++q) rest &= rest - 1;
    for (int q = 0; q < nsl; ++q) {
      s_t[q] = __builtin_ctzll(rest);
      rest &= rest - 1;
    }
  }
  __syncthreads();
  const int i = threadIdx.x >> 5, c = threadIdx.x & 31;
  float4 *mst = (float4 *)(sm + kMPad(4 * threadIdx.x));
  const float4 *mld = (const float4 *)(sm + kMPad(32 * c));
  float *b1 = lds + i * L::kStride + c;       // column c + 32 k at 33 k
  float *b2 = lds + i * L::kStride + 33 * c;  // column 32 c + m at m
  // an item's scalars; its pointers are formed where they are used
  struct Item {
    int64_t l, v0;
    int nv;
  };
  // item -> (column l, vector group): it = ((l / 8) ngroups + group) 8 + l % 8, so the vector groups of
  // a column fall on workgroups 8 apart, i.e. on one XCD (workgroups are dealt to the 8 XCDs in turn and
  // the grid is a multiple of 8), and read that column's M rows from the XCD's L2
  const int64_t ngroups = (bc + 7) / 8;
  auto open = [&](int64_t it) {
    Item r;
    const int64_t q = it >> 3;
    const int64_t grp = q % ngroups;
    r.l = ((q / ngroups) << 3) | (it & 7);
    r.v0 = grp * 8;
    r.nv = (int)((bc - r.v0) < 8 ? (bc - r.v0) : 8);
    return r;
  };
  // rows of absent vectors (i >= nv) load vector v0's data and are discarded
  auto vrow = [&](const Item &it) { return it.v0 + (i < it.nv ? i : 0); };
  auto fvp = [&](const Item &it) { return facc + (vrow(it) * 1024 + it.l) * 1024 + 32 * c; };  // F at p = 32 c + m
  float f[32];
  auto init_f = [&](const Item &it) {
    if (fmode & 1) {
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const float4 u = ((const float4 *)fvp(it))[q];
        f[4 * q] = u.x;
        f[4 * q + 1] = u.y;
        f[4 * q + 2] = u.z;
        f[4 * q + 3] = u.w;
      }
    } else {
#pragma unroll
      for (int m = 0; m < 32; ++m) f[m] = 0.0f;
    }
  };
  auto fetch = [&](const Item &it, int j, float(&e)[32], float4 &mv) {
    // W^T of group slab j ([l][slab][p] per vector), M of slab s_t[j]
    const float *src = w + vrow(it) * vstride + (it.l * (vstride >> 20) + j) * 1024 + c;
#pragma unroll
    for (int k = 0; k < 32; ++k) e[k] = src[32 * k];
    mv = *(const float4 *)(mt + (int64_t)s_t[j] * lo_len + it.l * 1024 + 4 * threadIdx.x);
  };
  auto step = [&](float(&e)[32], const float4 &mv) {
    fwht_regs_t<32>(e);
#pragma unroll
    for (int k = 0; k < 32; ++k) b1[33 * k] = e[k];
    *mst = mv;
    __syncthreads();
#pragma unroll
    for (int m = 0; m < 32; ++m) e[m] = b2[m];
    fwht_regs_t<32>(e);
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const float4 mm = mld[q];
      f[4 * q] += mm.x * e[4 * q];
      f[4 * q + 1] += mm.y * e[4 * q + 1];
      f[4 * q + 2] += mm.z * e[4 * q + 2];
      f[4 * q + 3] += mm.w * e[4 * q + 3];
    }
    __syncthreads();  // before the next slab's writes of lds and sm
  };
  auto end_item = [&](const Item &it) {
    if (!(fmode & 2)) {
      if (i < it.nv) {
#pragma unroll
        for (int q = 0; q < 8; ++q)
          ((float4 *)fvp(it))[q] = make_float4(f[4 * q], f[4 * q + 1], f[4 * q + 2], f[4 * q + 3]);
      }
      return;
    }
    // H_l of phase A, H_p twice (1/32 each) and H_TT (1/TT)
    affdT_finish8(ld, ptab, f, lds, it.l, it.v0, it.nv, R, 1.0f / (32768.0f * (float)TT), gout);
  };
  Item cur = open(item), nx = cur;
  init_f(cur);
  int j = 0;
  // one slab: prefetch the next (item, slab) into the other register set,
  // transform this one; false at the end of the workgroup's items
  auto iter = [&](float(&ec)[32], float4 &mc, float(&en)[32], float4 &mn) {
    int jn = j + 1;
    int64_t itn = item;
    if (jn == nsl) {
      jn = 0;
      itn = item + G;
    }
    const bool more = itn < nitems;
    if (more) {
      if (jn == 0) nx = open(itn);
      fetch(jn == 0 ? nx : cur, jn, en, mn);
    }
    step(ec, mc);
    if (j == nsl - 1) {
      end_item(cur);
      if (more) {
        cur = nx;
        init_f(cur);
      }
    }
    item = itn;
    j = jn;
    return more;
  };
  float ea[32], eb[32];
  float4 ma, mb;
  fetch(cur, 0, ea, ma);
#pragma unroll 1
  for (;;) {
    if (!iter(ea, ma, eb, mb)) break;
    if (!iter(eb, mb, ea, ma)) break;
  }
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

// Phase E for several layers at once: workgroup per (16 rows a, vector);
// for each listed layer in order, H_l along the 16 rows of its G, gather
// pi2_l(b) and add (times the layer's scale) into registers; out is written
// once.  The next layer's G rows are loaded during the current transform.
__global__ __launch_bounds__(256) void k_affdT_outm(const LayerDesc *__restrict__ layers,
                                                    const uint16_t *__restrict__ ptab, OutLayers ol, int R,
                                                    int64_t D, int64_t b_begin, int64_t gstride,
                                                    float *__restrict__ out, int accumulate) {
  using L = Lds1024<16>;
  __shared__ __align__(16) float s[L::kFloats];
  const int a0 = blockIdx.x * 16;
  const int na = (R - a0) < 16 ? (R - a0) : 16;
  const int64_t v = blockIdx.y;
  float acc[16][4];
#pragma unroll
  for (int i = 0; i < 16; ++i)
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[i][k] = 0.0f;
  // thread: columns l = tid + 256 k, rows a0 .. a0 + 15 (four 16-byte pieces)
  float4 g[4][4];
  auto fetch = [&](int j) {
    const float *src = ol.g[j] + v * gstride + (int64_t)threadIdx.x * R + a0;
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float *p = src + (int64_t)256 * k * R + 4 * q;
        if (4 * q + 4 <= na) {  // R is a power of two: whole pieces when R >= 4
          g[k][q] = *(const float4 *)p;
        } else {
          g[k][q].x = 4 * q < na ? p[0] : 0.0f;
          g[k][q].y = 4 * q + 1 < na ? p[1] : 0.0f;
          g[k][q].z = 4 * q + 2 < na ? p[2] : 0.0f;
          g[k][q].w = 4 * q + 3 < na ? p[3] : 0.0f;
        }
      }
  };
  fetch(0);
  for (int j = 0; j < ol.n; ++j) {
    __syncthreads();  // the previous layer's gathers from s are done
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int l = threadIdx.x + 256 * k;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        s[L::idx(4 * q, l)] = g[k][q].x;
        s[L::idx(4 * q + 1, l)] = g[k][q].y;
        s[L::idx(4 * q + 2, l)] = g[k][q].z;
        s[L::idx(4 * q + 3, l)] = g[k][q].w;
      }
    }
    if (j + 1 < ol.n) fetch(j + 1);
    __syncthreads();
    fwht1024_lds<16>(s);
    const LayerDesc &ld = layers[ol.layer[j]];
    const uint16_t *p2l = ptab + ld.poff[1][0][ld.K - 1];
    const float sc = ol.scale[j];
    int src[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) src[k] = p2l[threadIdx.x + 256 * k];
#pragma unroll
    for (int i = 0; i < 16; ++i)
#pragma unroll
      for (int k = 0; k < 4; ++k) acc[i][k] += s[L::idx(i, src[k])] * sc;
  }
  for (int i = 0; i < na; ++i) {
    float *o = out + (b_begin + v) * D + (int64_t)(a0 + i) * 1024;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int b = threadIdx.x + 256 * k;
      o[b] = accumulate ? o[b] + acc[i][k] : acc[i][k];
    }
  }
}

constexpr unsigned kRowsGrid = 256;

// Live slabs of a transposed-path layer: the images of the source slabs
// that hold data (the top-digit permutation is a bijection).
int affd_transposed_nlive(const sk_sketch *s, int layer) {
  return (int)((s->layers[layer].rows_live + 1023) / 1024);
}

// Vectors per call and live slabs per group.  A layer whose live slabs for 8
// vectors (the vectors of one top workgroup) fit the budget takes a multiple
// of 8 vectors that keeps one call's W^T (4 MB per vector and live slab)
// within the size of the 256 MB memory-side cache between the row and top
// kernels (measured on the GPT-2-small workload: 256 MB 31.0 ms per step,
// 192 MB 31.5, 128 MB 33.7, 512 MB 32.3: larger calls amortise the ramp of
// each launch, W^T beyond the cache slows the top kernel).  A
// larger layer takes 16 vectors (W^T then goes through HBM), and with the
// stored M tables, if the workspace cannot hold all their live slabs, as many
// slabs per group as fit, F being carried between the groups.  Without the
// tables (top kernels that regenerate G) TT > 8 has no preferred tile.
AffdTPlan affd_transposed_plan(const sk_sketch *s, int layer) {
  const LayerDesc &ld = s->layers[layer];
  const int nlive = affd_transposed_nlive(s, layer);
  AffdTPlan pl{0, nlive, false};
  if (!affd_transposed_path(s, layer)) return pl;
  const char *e = std::getenv("SK_AFFD_MALL_MB");
  const int64_t budget = std::max<int64_t>(1, e ? std::atoll(e) : 256) << 20;
  const int64_t wbytes = (int64_t)nlive * (4ll << 20);
  pl.compact = s->d_mtab && s->mtab_off[layer] >= 0;
  if (!pl.compact && ld.lgnp - 20 > 3) return pl;
  if (8 * wbytes <= budget || !pl.compact) {
    pl.tile = 8 * std::max<int64_t>(1, budget / (8 * wbytes));
    return pl;
  }
  pl.tile = 16;
  const int64_t avail = s->ws_bytes / 4 / pl.tile - s->D;  // floats per vector for W^T (and F)
  if (((int64_t)nlive << 20) > avail) pl.gsl = (int)std::max<int64_t>(1, (avail >> 20) - 1);
  return pl;
}

// Input elements of the source slabs behind live slabs s_first .. s_first +
// nsl - 1 (in increasing t) of a transposed-path layer.
int64_t affd_transposed_group_elems(const sk_sketch *s, int layer, int s_first, int nsl) {
  const LayerDesc &ld = s->layers[layer];
  const int TT = 1 << (ld.lgnp - 20);
  int64_t n = 0;
  int li = 0;
  for (int t = 0; t < TT; ++t) {
    int64_t src = 0, stride = 1;
    for (int k = ld.K - 3; k >= 0; --k) {
      const int64_t dig = (t / stride) & ((1ll << ld.lg[k]) - 1);
      src += (int64_t)s->h_ptab[ld.poff[0][1][k] + dig] * stride;
      stride <<= ld.lg[k];
    }
    if (src * 1024 >= ld.rows_live) continue;
    if (li >= s_first && li < s_first + nsl) n += std::min<int64_t>(ld.n, (src + 1) << 20) - (src << 20);
    ++li;
  }
  return n;
}

bool affd_transposed_path(const sk_sketch *s, int layer) {
  const LayerDesc &ld = s->layers[layer];
  if (s->D <= 1024 || ld.K < 2 || ld.L != 1024 || ld.dk1 != 1024) return false;
  const int lgtt = ld.lgnp - 20;
  return lgtt >= 0 && lgtt <= 6;
}

void run_affd_transposed(const sk_sketch *s, int layer, const void *x, int dtype, bool vec, int64_t b_begin,
                         int64_t bc, float *gbuf, int phases, const AffdTGroup &grp, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const int TT = 1 << (ld.lgnp - 20);
  const int R = (int)(s->D / 1024);
  float *w = s->ws;
  const int64_t vstride = grp.compact ? ((int64_t)grp.vslabs << 20) : ld.np;
  if (phases & 1) {  // A
    // one resident workgroup per CU (141 KB of LDS); a multiple of 8
    const dim3 grid(kRowsGrid);
    // buffer loads take 32-bit byte offsets
    if (ld.n * (dtype == SK_BF16 ? 2 : 4) >= (1ll << 31)) vec = false;
#define SK_AROWS(BF, VE)                                                                                  \
  hipLaunchKernelGGL((k_affdT_rows<BF, VE>), grid, dim3(1024), 0, st, s->d_layers, s->d_ptab, layer, x, b_begin, \
                     bc, w, grp.s_first, grp.nsl, vstride, (int)grp.compact, s->key)
    if (dtype == SK_BF16) {
      if (vec) SK_AROWS(true, true); else SK_AROWS(true, false);
    } else {
      if (vec) SK_AROWS(false, true); else SK_AROWS(false, false);
    }
#undef SK_AROWS
  }
  if (!(phases & 2)) return;
  if (grp.compact) {
    static int resident = 0;  // workgroups of the top kernel resident on the device at once
    if (!resident) {
      int per_cu = 0, cus = 0;
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_affdT_topM<8>, 256, 0) != hipSuccess || per_cu < 1)
        per_cu = 1;
      if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, s->device) != hipSuccess || cus < 1)
        cus = 1;
      resident = per_cu * cus;
    }
    const int64_t nitems = 1024 * ((bc + 7) / 8);
    hipLaunchKernelGGL(k_affdT_topM<8>, dim3((unsigned)std::min<int64_t>(nitems, resident)), dim3(256), 0, st, s->d_layers,
                       s->d_ptab, layer, w, bc, R, s->d_mtab + s->mtab_off[layer], grp.s_first, grp.nsl, vstride,
                       grp.facc, grp.fmode, gbuf);
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

void run_affd_transposed_outm(const sk_sketch *s, const OutLayers &ol, int64_t gstride, int64_t b_begin,
                              int64_t gb, float *out, bool accumulate, hipStream_t st) {
  const int R = (int)(s->D / 1024);
  hipLaunchKernelGGL(k_affdT_outm, dim3((unsigned)((R + 15) / 16), (unsigned)gb), dim3(256), 0, st, s->d_layers,
                     s->d_ptab, ol, R, s->D, b_begin, gstride, out, (int)accumulate);
  (void)hipGetLastError();
}

float affd_transposed_out_scale(const sk_sketch *s, int layer) {
  return (float)(std::sqrt((double)s->layers[layer].np / (double)s->D) / 32.0);
}

}  // namespace sk
