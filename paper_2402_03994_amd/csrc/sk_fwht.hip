// sk_fwht.hip -- Walsh-Hadamard based sketch kernels for gfx950 (wave64).
//
// Kinds: FJL (eq. ailon_chazelle), FFD (eq. fastfood, transposed), AFFD
// (eq. bami) and AFJL (eq. frikadel).  Conventions shared by every kernel:
//  - 256 threads per workgroup (four wave64 wavefronts);
//  - H is the normalised Walsh-Hadamard matrix; a full transform of length
//    2^m is a chain of LDS-tiled radix-2 passes whose per-pass scales multiply
//    to 2^{-m/2};
//  - random signs, Gaussians, sample positions and block permutations are
//    regenerated from (seed, layer, stream, index) (sk_device.h); digit
//    permutations of at most 1024 entries are small tables built at creation
//    (the O(A+B) lookups of Sec. 3, "Removing the lookup bottleneck");
//  - no floating-point atomics: every output element has one writer and a
//    fixed summation order.
#include <algorithm>

#include "sk_kcommon.h"
#include "sk_launch.h"

namespace sk {

#define SK_CHECK_LAUNCH() (void)hipGetLastError()

// log2 of a power of two held in 64 bits.
static int log2_exact(int64_t v) {
  int l = 0;
  while ((1ll << l) < v) ++l;
  return l;
}

// ---------------------------------------------------------------------------
// Generic pass: transform along index bits [lo, lo + w) of each vector.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_fwht_pass(float *data, int lgn, int lo, int w, int lgcs, float scale) {
  extern __shared__ float s[];
  const int64_t n = 1ll << lgn;
  const int64_t tiles_per_vec = n >> (w + lgcs);
  const int64_t v = blockIdx.x / tiles_per_vec;
  const int64_t tv = blockIdx.x - v * tiles_per_vec;
  const int lgcb = lo - lgcs;  // column blocks per high index
  const int64_t a = tv >> lgcb;
  const int64_t cb = tv & ((1ll << lgcb) - 1);
  float *base = data + v * n + (a << (lo + w)) + (cb << lgcs);
  const int total = 1 << (w + lgcs);
  const int cmask = (1 << lgcs) - 1;
  for (int e = threadIdx.x; e < total; e += 256) s[p16(e)] = base[((int64_t)(e >> lgcs) << lo) + (e & cmask)];
  lds_fwht_regs(s, w + lgcs, lgcs);
  for (int e = threadIdx.x; e < total; e += 256) base[((int64_t)(e >> lgcs) << lo) + (e & cmask)] = s[p16(e)] * scale;
}

void fwht_inplace(float *data, int64_t V, int lgn, hipStream_t st) { fwht_inplace_from(data, V, lgn, 0, st); }

int fwht_pass_plan(int lgn, int lo0, int *los, int *ws, int *lgcss) {
  int np = 0, lo = lo0;
  while (lo < lgn) {
    int w, lgcs;
    if (lo == 0) {
      w = lgn < 13 ? lgn : 13;
      lgcs = 0;
    } else {
      w = (lgn - lo) < 8 ? (lgn - lo) : 8;
      lgcs = 13 - w;
      if (lgcs > lo) lgcs = lo;
    }
    los[np] = lo;
    ws[np] = w;
    lgcss[np] = lgcs;
    ++np;
    lo += w;
  }
  return np;
}

// Passes [first, end) of the plan of fwht_pass_plan(lgn, lo0).
static void fwht_passes(float *data, int64_t V, int lgn, int lo0, int first, int end, hipStream_t st) {
  int los[64], ws[64], lgcss[64];
  const int np = fwht_pass_plan(lgn, lo0, los, ws, lgcss);
  for (int k = first; k < std::min(end, np); ++k) {
    const int lo = los[k], w = ws[k], lgcs = lgcss[k];
    const int64_t tiles = V * ((1ll << lgn) >> (w + lgcs));
    const float scale = (float)(1.0 / sqrt((double)(1ll << w)));
    const size_t shm = sizeof(float) * p16_floats(1 << (w + lgcs));
    hipLaunchKernelGGL(k_fwht_pass, dim3((unsigned)tiles), dim3(256), shm, st, data, lgn, lo, w, lgcs, scale);
    SK_CHECK_LAUNCH();
  }
}

// The passes of fwht_inplace from index bit lo0 on (bits below lo0 already transformed).
void fwht_inplace_from(float *data, int64_t V, int lgn, int lo0, hipStream_t st) {
  if (lgn == 0 || V == 0) return;
  fwht_passes(data, V, lgn, lo0, 0, 64, st);
}

void fwht_inplace_from_but_last(float *data, int64_t V, int lgn, int lo0, hipStream_t st) {
  if (lgn == 0 || V == 0) return;
  int los[64], ws[64], lgcss[64];
  const int np = fwht_pass_plan(lgn, lo0, los, ws, lgcss);
  fwht_passes(data, V, lgn, lo0, 0, np - 1, st);
}

__global__ void k_fill_zero(float *p, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0.0f;
}

void launch_fill_zero(float *p, int64_t n, hipStream_t st) {
  if (n <= 0) return;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_fill_zero, dim3((unsigned)blocks), dim3(256), 0, st, p, n);
  SK_CHECK_LAUNCH();
}

// ===========================================================================
// AFJL.  With w = Scatter_pi1(B x), the restriction to the first D rows of a
// normalised Hadamard transform of length N' is sqrt(D/N') H_D fold_D(w)
// (fold_D sums the N'/D consecutive length-D chunks; this follows from the
// Hadamard definition), so AFJL(x) = g_{<D} . H_D fold_D(Scatter_pi1 B x).
// The digit structure of pi1 makes fold_D a row routing: row h (the L = 1024
// consecutive coordinates sharing all digits but the last) lands in
// destination row r = pi1_{K-2}(h mod dk1) mod R of an R x L accumulator
// (D = R L), its columns permuted by pi1_{K-1}.  H_D = H_R (x) H_L: the fold
// kernel applies H_L to each destination row, the tail kernel H_R, G and the
// sum over layers.  For D < L the row is folded once more to D columns.
// ===========================================================================
// Up to CPT consecutive input elements starting at element e (missing -> 0).
template <int CPT, bool BF16, bool VEC>
__device__ __forceinline__ void load_cols(const void *x, int64_t e, int64_t lim, float v[CPT]) {
  if (CPT == 8 && BF16 && VEC && lim >= 8) {
    const uint4 u = *(const uint4 *)((const uint16_t *)x + e);
    v[0] = __uint_as_float(u.x << 16);
    v[1] = __uint_as_float(u.x & 0xFFFF0000u);
    v[2] = __uint_as_float(u.y << 16);
    v[3] = __uint_as_float(u.y & 0xFFFF0000u);
    v[4] = __uint_as_float(u.z << 16);
    v[5] = __uint_as_float(u.z & 0xFFFF0000u);
    v[6] = __uint_as_float(u.w << 16);
    v[7] = __uint_as_float(u.w & 0xFFFF0000u);
    return;
  }
#pragma unroll
  for (int q = 0; q < CPT; q += 4) load4<BF16, VEC>(x, e + q, lim - q, v + q);
}

// CPT (4 fp32 or up to 8 bf16) consecutive elements from element e as their raw
// bit patterns in 16 bytes; elements at or past lim read as zero.
template <int CPT, bool BF16, bool VEC>
__device__ __forceinline__ uint4 load_raw16(const void *x, int64_t e, int64_t lim) {
  if (VEC && lim >= CPT && (BF16 ? CPT == 8 : CPT == 4)) {
    // each input element is read once
    return ld_nt16(BF16 ? (const void *)((const uint16_t *)x + e) : (const void *)((const float *)x + e));
  }
  uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int q = 0; q < CPT; ++q) {
    if (q < lim) {
      if (BF16)
        w[q >> 1] |= (uint32_t)((const uint16_t *)x)[e + q] << (16 * (q & 1));
      else
        w[q] = ((const uint32_t *)x)[e + q];
    }
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

template <bool BF16>
__device__ __forceinline__ float raw16_value(const uint4 &r, int q) {
  const uint32_t w = (q >> (BF16 ? 1 : 0)) == 0 ? r.x : (q >> (BF16 ? 1 : 0)) == 1 ? r.y
                   : (q >> (BF16 ? 1 : 0)) == 2 ? r.z : r.w;
  return BF16 ? __uint_as_float((q & 1) ? (w & 0xFFFF0000u) : (w << 16)) : __uint_as_float(w);
}

// Fold kernel.  Each thread owns CPT consecutive columns of a row; when a row
// needs fewer than 256 threads, NGR = 256 / (L / CPT) row groups take
// interleaved rows and their sums are combined in LDS in group order.  The
// item's source rows are resolved into LDS first, and the loads of a group's
// next row are issued before the current one is added.
template <int BT, int CPT, bool BF16, bool VEC>
__global__ __launch_bounds__(256) void k_afjl_fold(const FoldItem *__restrict__ items,
                                                   const LayerDesc *__restrict__ layers,
                                                   const uint16_t *__restrict__ ptab, PtrPack ptrs, int first_layer,
                                                   int64_t batch, int64_t b_begin, int64_t bc, int item_begin, int R,
                                                   int Lw, float *__restrict__ part, Key key) {
  using LF = Lds1024<BT>;
  __shared__ __align__(16) float s_raw[LF::kFloats > BT * 1024 ? LF::kFloats : BT * 1024];
  static_assert(kFoldRowsPerItem <= 256, "one thread per source row of an item");
  __shared__ int32_t srow[kFoldRowsPerItem];
  float(*s)[1024] = reinterpret_cast<float(*)[1024]>(s_raw);
  const FoldItem it = items[item_begin + blockIdx.x];
  const LayerDesc &ld = layers[it.layer];
  const int64_t n = ld.n;
  const int L = ld.L;
  const int tid = threadIdx.x;
  const int tpr = L / CPT < 1 ? 1 : L / CPT;  // threads per row
  const int ngr = 256 / tpr;                  // row groups
  const int grp = tid / tpr;
  const int col0 = (tid - grp * tpr) * CPT;
  const bool active = grp < ngr && col0 < L;
  const int bt0 = blockIdx.y * BT;
  const void *xp = ptrs.p[it.layer - first_layer];
  const int nb = (int)((batch - b_begin - bt0) < BT ? (batch - b_begin - bt0) : BT);  // rows of this tile
  const int nt = it.t1 - it.t0;  // <= kFoldRowsPerItem
  // source row of each fold step (-1 past the data)
  {
    const int nk = R > 1 ? ld.dk1 / R : 1;
    const uint16_t *inv_k1 = ptab + ld.poff[0][1][ld.K >= 2 ? ld.K - 2 : 0];
    if (tid < nt) {
      const int t = it.t0 + tid;
      int64_t h;
      if (R == 1) {
        h = t;
      } else {
        const int htop = t / nk;
        const int k = t - htop * nk;
        h = (int64_t)htop * ld.dk1 + inv_k1[it.r + k * R];
      }
      srow[tid] = h < ld.rows_live ? (int32_t)h : -1;
    }
    __syncthreads();
  }
  float acc[BT][CPT];
#pragma unroll
  for (int b = 0; b < BT; ++b)
#pragma unroll
    for (int q = 0; q < CPT; ++q) acc[b][q] = 0.0f;
  if (active) {
    // raw 16-byte pieces (CPT fp32 or bf16 values) of the next row, per vector
    uint4 v[BT];
    int64_t jn = -1;
    auto fetch = [&](int i) {
      const int32_t h = i < nt ? srow[i] : -1;
      jn = h >= 0 ? (int64_t)h * L + col0 : -1;
      if (jn >= n) jn = -1;
#pragma unroll
      for (int b = 0; b < BT; ++b) {
        v[b] = make_uint4(0u, 0u, 0u, 0u);
        if (jn >= 0 && b < nb) v[b] = load_raw16<CPT, BF16, VEC>(xp, (b_begin + bt0 + b) * n + jn, n - jn);
      }
    };
    fetch(grp);
    for (int i = grp; i < nt; i += ngr) {
      uint4 cur[BT];
#pragma unroll
      for (int b = 0; b < BT; ++b) cur[b] = v[b];
      const int64_t j = jn;
      fetch(i + ngr);
      if (j >= 0) {
        const uint32_t bits = sign_word((uint64_t)j, (uint32_t)ld.layer_id, key) >> (j & 31);
#pragma unroll
        for (int b = 0; b < BT; ++b)
#pragma unroll
          for (int q = 0; q < CPT; ++q) acc[b][q] += flip(raw16_value<BF16>(cur[b], q), (bits >> q) & 1u);
      }
    }
  }
  // route the columns through pi1 of the last digit
  const uint16_t *fwd_k = ptab + ld.poff[0][0][ld.K - 1];
  int pc[CPT];
  if (active) {
#pragma unroll
    for (int q = 0; q < CPT; ++q) pc[q] = fwd_k[col0 + q];
  }
  const int64_t slot = blockIdx.x;
  if (L == 1024 && Lw == 1024) {
    // row groups add in order, then H_L of the BT rows in a conflict-free LDS block
    for (int gi = 0; gi < ngr; ++gi) {
      if (active && grp == gi) {
#pragma unroll
        for (int q = 0; q < CPT; ++q)
#pragma unroll
          for (int b = 0; b < BT; ++b) {
            float *d = s_raw + LF::idx(b, pc[q]);
            *d = gi == 0 ? acc[b][q] : *d + acc[b][q];
          }
      }
      __syncthreads();
    }
    fwht1024_lds<BT>(s_raw);
    for (int b = 0; b < nb; ++b)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int c = tid + 256 * k;
        part[(slot * bc + bt0 + b) * 1024 + c] = s_raw[LF::idx(b, c)] * (1.0f / 32.0f);
      }
    return;
  }
  // row groups add in order
  for (int gi = 0; gi < ngr; ++gi) {
    if (active && grp == gi) {
#pragma unroll
      for (int q = 0; q < CPT; ++q)
#pragma unroll
        for (int b = 0; b < BT; ++b) s[b][pc[q]] = gi == 0 ? acc[b][q] : s[b][pc[q]] + acc[b][q];
    }
    __syncthreads();
  }
  int lgw;
  if (Lw < L) {
    // fold the permuted row to Lw = D columns
    float tmp[BT * 2];
    const int tot = BT * Lw;
    int cnt = 0;
    for (int e = tid; e < tot; e += 256, ++cnt) {
      const int b = e / Lw, c = e - (e / Lw) * Lw;
      float v = 0.0f;
      for (int k = 0; k < L; k += Lw) v += s[b][k + c];
      tmp[cnt] = v;
    }
    __syncthreads();
    cnt = 0;
    for (int e = tid; e < tot; e += 256, ++cnt) s[e / Lw][e - (e / Lw) * Lw] = tmp[cnt];
    __syncthreads();
  }
  lgw = 31 - __clz(Lw);
  for (int b = 0; b < BT; ++b) {
    // each row is a separate transform: reuse the tile routine with one column
    lds_fwht(&s[b][0], lgw, 0);
  }
  const float sc = rsqrtf((float)Lw);
  for (int e = tid; e < nb * Lw; e += 256) {
    const int b = e / Lw, c = e - (e / Lw) * Lw;
    part[(slot * bc + bt0 + b) * Lw + c] = s[b][c] * sc;
  }
}

// Fold kernel for a single vector (batch tiles of one row) of layers with
// L = Lw = 1024.  With one vector the per-thread sign block of the tiled
// kernel is not shared by any other vector, so here the item's sign words are
// built first, one Philox block per 128 coordinates (8 per source row) into
// LDS, and each row group keeps PF rows of 16-byte loads in flight (one
// vector gives a workgroup too little work to hide the latency otherwise).
template <int CPT, bool BF16, bool VEC>
__global__ __launch_bounds__(256) void k_afjl_fold1(const FoldItem *__restrict__ items,
                                                    const LayerDesc *__restrict__ layers,
                                                    const uint16_t *__restrict__ ptab, PtrPack ptrs, int first_layer,
                                                    int64_t b_row, int64_t bc, int64_t slot_row, int item_begin, int R,
                                                    float *__restrict__ part, Key key) {
  constexpr int PF = 4;
  constexpr int TPR = 1024 / CPT;  // threads per row
  constexpr int NGR = 256 / TPR;   // row groups
  __shared__ float s[1024];
  __shared__ int32_t srow[kFoldRowsPerItem];
  __shared__ __align__(16) uint32_t sgn[kFoldRowsPerItem * 32];
  const FoldItem it = items[item_begin + blockIdx.x];
  const LayerDesc &ld = layers[it.layer];
  const int64_t n = ld.n;
  const int tid = threadIdx.x;
  const int grp = tid / TPR;
  const int col0 = (tid - grp * TPR) * CPT;
  const void *xp = ptrs.p[it.layer - first_layer];
  const int nt = it.t1 - it.t0;  // <= kFoldRowsPerItem
  {
    const int nk = R > 1 ? ld.dk1 / R : 1;
    const uint16_t *inv_k1 = ptab + ld.poff[0][1][ld.K >= 2 ? ld.K - 2 : 0];
    if (tid < nt) {
      const int t = it.t0 + tid;
      int64_t h;
      if (R == 1) {
        h = t;
      } else {
        const int htop = t / nk;
        const int k = t - htop * nk;
        h = (int64_t)htop * ld.dk1 + inv_k1[it.r + k * R];
      }
      srow[tid] = h < ld.rows_live ? (int32_t)h : -1;
    }
    __syncthreads();
  }
  // sign words of the item's rows: 8 Philox blocks of 128 coordinates per row
  for (int u = tid; u < nt * 8; u += 256) {
    const int32_t h = srow[u >> 3];
    if (h >= 0) {
      const W4 w = philox((uint64_t)h * 8u + (uint64_t)(u & 7), (uint32_t)ld.layer_id, ST_SIGN, key);
      *reinterpret_cast<uint4 *>(&sgn[4 * u]) = make_uint4(w.w[0], w.w[1], w.w[2], w.w[3]);
    }
  }
  __syncthreads();
  float acc[CPT];
#pragma unroll
  for (int q = 0; q < CPT; ++q) acc[q] = 0.0f;
  const int64_t xrow = b_row * n;
  uint4 ring[PF];
  int64_t jr[PF];
  auto fetch = [&](int i, uint4 &v, int64_t &jn) {
    const int32_t h = i < nt ? srow[i] : -1;
    jn = h >= 0 ? (int64_t)h * 1024 + col0 : -1;
    if (jn >= n) jn = -1;
    v = make_uint4(0u, 0u, 0u, 0u);
    if (jn >= 0) v = load_raw16<CPT, BF16, VEC>(xp, xrow + jn, n - jn);
  };
#pragma unroll
  for (int p = 0; p < PF; ++p) fetch(grp + p * NGR, ring[p], jr[p]);
  for (int i0 = grp; i0 < nt; i0 += PF * NGR) {
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      const int i = i0 + p * NGR;
      const uint4 cur = ring[p];
      const int64_t j = jr[p];
      fetch(i + PF * NGR, ring[p], jr[p]);
      if (j >= 0) {
        const uint32_t bits = sgn[i * 32 + (col0 >> 5)] >> (col0 & 31);
#pragma unroll
        for (int q = 0; q < CPT; ++q) acc[q] += flip(raw16_value<BF16>(cur, q), (bits >> q) & 1u);
      }
    }
  }
  // route the columns through pi1 of the last digit; row groups add in order
  const uint16_t *fwd_k = ptab + ld.poff[0][0][ld.K - 1];
  int pc[CPT];
#pragma unroll
  for (int q = 0; q < CPT; ++q) pc[q] = fwd_k[col0 + q];
  for (int gi = 0; gi < NGR; ++gi) {
    if (grp == gi) {
#pragma unroll
      for (int q = 0; q < CPT; ++q) s[pc[q]] = gi == 0 ? acc[q] : s[pc[q]] + acc[q];
    }
    __syncthreads();
  }
  lds_fwht(s, 10, 0);
  const int64_t slot = blockIdx.x;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int c = tid + 256 * k;
    part[(slot * bc + slot_row) * 1024 + c] = s[c] * (1.0f / 32.0f);
  }
}

void launch_afjl_fold(const sk_sketch *s, const PtrPack &ptrs, int first_layer, int dtype, bool vec, int64_t batch,
                      int64_t b_begin, int64_t bc, int item_begin, int item_end, float *part, hipStream_t st) {
  constexpr int BT = 8;
  const int nitems = item_end - item_begin;
  if (nitems <= 0) return;
  const int64_t rows = (batch - b_begin) < bc ? (batch - b_begin) : bc;
  bool one = rows == 1 && s->Lw == 1024;
  for (int i = item_begin; i < item_end && one; ++i) one = s->layers[s->items[i].layer].L == 1024;
  if (one) {
#define SK_FOLD1(CPT, BF, VE)                                                                                        \
  hipLaunchKernelGGL((k_afjl_fold1<CPT, BF, VE>), dim3((unsigned)nitems), dim3(256), 0, st, s->d_items, s->d_layers, \
                     s->d_ptab, ptrs, first_layer, b_begin, bc, (int64_t)0, item_begin, s->R, part, s->key)
    if (dtype == SK_BF16) {
      if (vec) SK_FOLD1(8, true, true); else SK_FOLD1(4, true, false);
    } else {
      if (vec) SK_FOLD1(4, false, true); else SK_FOLD1(4, false, false);
    }
#undef SK_FOLD1
    SK_CHECK_LAUNCH();
    return;
  }
  dim3 grid((unsigned)nitems, (unsigned)((rows + BT - 1) / BT));
#define SK_FOLD(CPT, BF, VE)                                                                                       \
  hipLaunchKernelGGL((k_afjl_fold<BT, CPT, BF, VE>), grid, dim3(256), 0, st, s->d_items, s->d_layers, s->d_ptab,   \
                     ptrs, first_layer, batch, b_begin, bc, item_begin, s->R, s->Lw, part, s->key)
  if (dtype == SK_BF16) {
    if (vec) SK_FOLD(8, true, true); else SK_FOLD(4, true, false);
  } else {
    if (vec) SK_FOLD(4, false, true); else SK_FOLD(4, false, false);
  }
#undef SK_FOLD
  SK_CHECK_LAUNCH();
}

// Tail: out[b, r' Lw + c] = sum_l g_l[r' Lw + c] * (H_R T_l[b, :, c])[r'],
// T_l the sum of a layer's fold partials.
template <int PER>
__global__ __launch_bounds__(256) void k_afjl_tail(const LayerDesc *__restrict__ layers, const int2 *__restrict__ rslot,
                                                   const float *__restrict__ part, const float *__restrict__ gtab,
                                                   int l_begin, int l_end, int item_begin, int lgR, int Lw,
                                                   int lgcs, int64_t D, int64_t bc, int64_t b_begin,
                                                   int64_t batch, float *__restrict__ out, int accumulate) {
  extern __shared__ float s[];
  const int CS = 1 << lgcs;
  const int R = 1 << lgR;
  const int c0 = blockIdx.x * CS;
  const int bl = blockIdx.y;
  const int64_t b = b_begin + bl;
  if (b >= batch) return;
  const int tot = R * CS;
  float acc[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) acc[i] = 0.0f;
  const float sc = rsqrtf((float)R);
  for (int l = l_begin; l < l_end; ++l) {
    const LayerDesc &ld = layers[l];
    const int2 *rs = rslot + ld.rslot_off;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = threadIdx.x + i * 256;
      if (e < tot) {
        const int r = e >> lgcs, c = e & (CS - 1);
        const int2 q = rs[r];
        float v = 0.0f;
        for (int k = 0; k < q.y; ++k) v += part[((int64_t)(q.x - item_begin + k) * bc + bl) * Lw + c0 + c];
        s[e] = v;
      }
    }
    if (R > 1)
      lds_fwht(s, lgR, lgcs);
    else
      __syncthreads();
    const float *g = gtab + (int64_t)l * D;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = threadIdx.x + i * 256;
      if (e < tot) {
        const int r = e >> lgcs, c = e & (CS - 1);
        acc[i] += g[(int64_t)r * Lw + c0 + c] * (s[e] * sc);
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int e = threadIdx.x + i * 256;
    if (e < tot) {
      const int r = e >> lgcs, c = e & (CS - 1);
      const int64_t o = b * D + (int64_t)r * Lw + c0 + c;
      out[o] = accumulate ? out[o] + acc[i] : acc[i];
    }
  }
}

// v[j] = sum of the fold partials of destination row j (rs[j] = first item,
// item count; rf[j] = first item or -1) at one column of one vector.  The
// layer's partials are read through the buffer resource pr: item item0 + i at
// byte i stride + voff0 (missing rows read past the end, i.e. zero).  With at
// most one item per row the J loads go out together; otherwise chunk k of
// every row is added in turn, the row records being re-read for each chunk
// rather than held in registers.
template <int J>
__device__ __forceinline__ void tail_gather(int maxch, const int2 *rs, const int32_t *rf, __amdgpu_buffer_rsrc_t pr,
                                            uint32_t stride, uint32_t voff0, int item0, float (&v)[J]) {
  constexpr uint32_t kNone = 0x80000000u;  // beyond the resource (< 2^31 bytes)
  if (maxch <= 1) {
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int f = rf[j];
      const uint32_t off = f >= 0 ? (uint32_t)(f - item0) * stride + voff0 : kNone;
      v[j] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(pr, (int)off, 0, 0));
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < J; ++j) v[j] = 0.0f;
  for (int k = 0; k < maxch; ++k) {
#pragma unroll
    for (int j0 = 0; j0 < J; j0 += 16) {
      asm volatile("" ::: "memory");  // re-read the row records
#pragma unroll
      for (int j = j0; j < j0 + 16 && j < J; ++j) {
        const int2 q = rs[j];
        const uint32_t off = k < q.y ? (uint32_t)(q.x + k - item0) * stride + voff0 : kNone;
        v[j] += __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(pr, (int)off, 0, 0));
      }
    }
  }
}

// The partials of layer ld as a buffer resource (the callers keep each
// layer's partials below 2^31 bytes).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tail_part_rsrc(const LayerDesc &ld, const float *part, int item_begin,
                                                                 int64_t bc, int Lw) {
  return buf_rsrc(part + (int64_t)(ld.item_off - item_begin) * bc * Lw, (uint32_t)((int64_t)ld.n_items * bc * Lw * 4));
}

// Tail for R <= 64: the R values of a (vector, column) stay in registers
// across all layers (no LDS, no barriers).  R <= 32: one thread per column;
// R = 64: two threads (the two halves of a wave, 32 columns per wave) hold
// rows 32 h + j, H_64 = H_2 (across the halves) (x) H_32 (in registers).  The
// G loads of a layer go out with its partial loads.  Layers are split into
// contiguous groups (blockIdx.y); group gi writes its sum to ysum[gi][bl][:],
// reduced in group order afterwards.
template <int R>
__global__ __launch_bounds__(256, 4) void k_afjl_tail_reg(const LayerDesc *__restrict__ layers,
                                                       const int2 *__restrict__ rslot,
                                                       const int32_t *__restrict__ rfirst, const float *__restrict__ part,
                                                       const float *__restrict__ gtab, TailGroups grp,
                                                       int item_begin, int Lw, int64_t D, int64_t bc, int64_t b_begin,
                                                       int64_t batch, float *__restrict__ ysum) {
  constexpr int H = R > 32 ? 2 : 1, J = R / H;
  const int64_t gid = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  int c, h;
  int64_t bl;
  if (H == 1) {
    c = (int)(gid % Lw);
    bl = gid / Lw;
    h = 0;
  } else {  // Lw % 32 == 0; bl is uniform over the wave
    const int64_t wv = gid >> 6;
    const int nb = Lw / 32;
    bl = wv / nb;
    c = (int)(wv % nb) * 32 + (int)(threadIdx.x & 31);
    h = (int)((threadIdx.x >> 5) & 1);
  }
  if (bl >= bc || b_begin + bl >= batch) return;
  const int l_begin = grp.bound[blockIdx.y], l_end = grp.bound[blockIdx.y + 1];
  float acc[J];
#pragma unroll
  for (int j = 0; j < J; ++j) acc[j] = 0.0f;
  for (int l = l_begin; l < l_end; ++l) {
    const LayerDesc &ld = layers[l];
    const int2 *rs = rslot + ld.rslot_off + h * J;
    const int32_t *rf = rfirst + ld.rslot_off + h * J;
    // G of the layer through a buffer resource: the row offsets are scalars
    const __amdgpu_buffer_rsrc_t gr = buf_rsrc(gtab + (int64_t)l * D, (uint32_t)(D * 4));
    const int goff = (h * J * Lw + c) * 4;
    float v[J], gv[J];
    tail_gather<J>(ld.rmaxch, rs, rf, tail_part_rsrc(ld, part, item_begin, bc, Lw), (uint32_t)(bc * Lw * 4),
                   (uint32_t)((bl * Lw + c) * 4), ld.item_off, v);
    // the G loads go out while the partials are in flight
#pragma unroll
    for (int j = 0; j < J; ++j) gv[j] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(gr, goff, j * Lw * 4, 0));
    fwht_regs_t<J>(v);
    if (H == 2) {
#pragma unroll
      for (int j = 0; j < J; ++j) {
        const float o = __shfl_xor(v[j], 32);
        v[j] = h ? o - v[j] : v[j] + o;
      }
    }
#pragma unroll
    for (int j = 0; j < J; ++j) acc[j] += gv[j] * v[j];
  }
  const float sc = rsqrtf((float)R);
  float *o = ysum + ((int64_t)blockIdx.y * bc + bl) * D + (int64_t)h * J * Lw + c;
#pragma unroll
  for (int j = 0; j < J; ++j) o[(int64_t)j * Lw] = acc[j] * sc;
}

// R = Lw = 1024 with 1024 threads: workgroup per (32 columns, vector), so every
// partial and G row piece is a full 128-byte line; thread (hi, c) holds rows
// hi * 32 + j of column c0 + c, H_R = H_32 (x) H_32 with one LDS transpose
// (128 KB); four waves per SIMD hide the load latency.
__global__ __launch_bounds__(1024) void k_afjl_tail_1024w(const LayerDesc *__restrict__ layers,
                                                          const int2 *__restrict__ rslot,
                                                          const int32_t *__restrict__ rfirst,
                                                          const float *__restrict__ part,
                                                          const float *__restrict__ gtab, int l_begin, int l_end,
                                                          int item_begin, int64_t D, int64_t bc, int64_t b_begin,
                                                          float *__restrict__ out, int accumulate) {
  __shared__ float s[1024 * 32];
  const int c = threadIdx.x & 31, hi = threadIdx.x >> 5;
  // workgroup x runs on XCD x mod 8: each XCD takes 4 consecutive column blocks
  const int c0 = ((blockIdx.x & 7) * 4 + (blockIdx.x >> 3)) * 32;
  const int64_t bl = blockIdx.y;
  float acc[32];
#pragma unroll
  for (int j = 0; j < 32; ++j) acc[j] = 0.0f;
  for (int l = l_begin; l < l_end; ++l) {
    float v[32], gv[32];
    const int2 *rs = rslot + layers[l].rslot_off;
    // the G loads go out while the partials are in flight (one memory
    // latency per layer), through a buffer resource with scalar row offsets
    const __amdgpu_buffer_rsrc_t gr = buf_rsrc(gtab + (int64_t)l * D, (uint32_t)(D * 4));
    const int goff = (hi * 1024 + c0 + c) * 4;
    const LayerDesc &ld = layers[l];
    tail_gather<32>(ld.rmaxch, rs + hi * 32, rfirst + ld.rslot_off + hi * 32, tail_part_rsrc(ld, part, item_begin, bc, 1024),
                    (uint32_t)(bc * 1024 * 4), (uint32_t)((bl * 1024 + c0 + c) * 4), ld.item_off, v);
#pragma unroll
    for (int j = 0; j < 32; ++j) gv[j] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(gr, goff, j * 32 * 4096, 0));
    fwht_regs_t<32>(v);
#pragma unroll
    for (int j = 0; j < 32; ++j) s[(hi * 32 + j) * 32 + c] = v[j];
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 32; ++j) v[j] = s[(j * 32 + hi) * 32 + c];
    __syncthreads();
    fwht_regs_t<32>(v);
#pragma unroll
    for (int j = 0; j < 32; ++j) acc[j] += gv[j] * v[j];
  }
  float *o = out + (b_begin + bl) * D + c0 + c;
#pragma unroll
  for (int j = 0; j < 32; ++j) {
    const int64_t r = j * 32 + hi;
    const float val = acc[j] * (1.0f / 32.0f);
    o[r * 1024] = accumulate ? o[r * 1024] + val : val;
  }
}

void launch_afjl_tail(const sk_sketch *s, int l_begin, int l_end, int item_begin, const float *part, int64_t bc,
                      int64_t b_begin, int64_t batch, float *out, bool accumulate, hipStream_t st) {
  // the register tails read each layer's partials through a buffer resource
  bool small_parts = true;
  for (int l = l_begin; l < l_end; ++l)
    small_parts = small_parts && (int64_t)s->layers[l].n_items * bc * s->Lw * 4 < (1ll << 31);
  if (s->R == 1024 && s->Lw == 1024 && small_parts) {
    const int64_t rows = (batch - b_begin) < bc ? (batch - b_begin) : bc;
    hipLaunchKernelGGL(k_afjl_tail_1024w, dim3(32u, (unsigned)rows), dim3(1024), 0, st, s->d_layers, s->d_rslot,
                       s->d_rfirst, part, s->d_gtab, l_begin, l_end, item_begin, s->D, bc, b_begin, out,
                       (int)accumulate);
    SK_CHECK_LAUNCH();
    return;
  }
  const int R = s->R, Lw = s->Lw;
  if (R <= 64 && small_parts) {
    // balance the layer loop: groups of about equal live destination rows
    TailGroups grp{};
    int64_t total = 0;
    for (int l = l_begin; l < l_end; ++l) total += s->layers[l].n_items;
    const int G = std::min(kTailGroups, l_end - l_begin);
    int ng = 0;
    grp.bound[0] = l_begin;
    int64_t accw = 0;
    for (int l = l_begin; l < l_end; ++l) {
      accw += s->layers[l].n_items;
      if (ng < G - 1 && accw * G >= total * (ng + 1) && l + 1 < l_end) grp.bound[++ng] = l + 1;
    }
    grp.bound[++ng] = l_end;
    float *ysum = s->ws + (s->ws_bytes / 4 - (int64_t)kTailGroups * bc * s->D);
    const int64_t threads = bc * Lw * (R > 32 ? 2 : 1);
    dim3 grid((unsigned)((threads + 255) / 256), (unsigned)ng);
#define SK_TAIL(RR)                                                                                              \
  case RR:                                                                                                       \
    hipLaunchKernelGGL(k_afjl_tail_reg<RR>, grid, dim3(256), 0, st, s->d_layers, s->d_rslot, s->d_rfirst, part,  \
                       s->d_gtab, grp, item_begin, Lw, s->D, bc, b_begin, batch, ysum);                          \
    break;
    switch (R) {
      SK_TAIL(1) SK_TAIL(2) SK_TAIL(4) SK_TAIL(8) SK_TAIL(16) SK_TAIL(32) SK_TAIL(64)
      default: break;
    }
#undef SK_TAIL
    launch_reduce_partials(ysum, ng, bc, s->D, b_begin, out, accumulate, st);
    SK_CHECK_LAUNCH();
    return;
  }
  int lgR = 31 - __builtin_clz(R);
  // tile of R rows x CS columns, at most 4096 elements
  int lgcs = 12 - lgR;
  const int lgLw = 31 - __builtin_clz(Lw);
  if (lgcs > lgLw) lgcs = lgLw;
  if (lgcs < 0) lgcs = 0;
  const int tot = R << lgcs;
  const int64_t rows = (batch - b_begin) < bc ? (batch - b_begin) : bc;
  dim3 grid((unsigned)(Lw >> lgcs), (unsigned)rows);
  const size_t shm = sizeof(float) * tot;
  if (tot <= 256 * 4)
    hipLaunchKernelGGL(k_afjl_tail<4>, grid, dim3(256), shm, st, s->d_layers, s->d_rslot, part, s->d_gtab, l_begin,
                       l_end, item_begin, lgR, Lw, lgcs, s->D, bc, b_begin, batch, out, (int)accumulate);
  else
    hipLaunchKernelGGL(k_afjl_tail<16>, grid, dim3(256), shm, st, s->d_layers, s->d_rslot, part, s->d_gtab, l_begin,
                       l_end, item_begin, lgR, Lw, lgcs, s->D, bc, b_begin, batch, out, (int)accumulate);
  SK_CHECK_LAUNCH();
}

// AFJL transpose.  H_N' R_D^T u = sqrt(D/N') tile(H_D u), so
// AFJL^T z = B Gather_pi1 tile(H_D (g . z)): out[j] = b_j V[pi1(j) mod D].
// The layers of a call go through in groups: one launch forms g_l . z for
// every layer and vector of the group, one set of transform passes covers all
// of them, and one launch writes every output row of the group (a vector
// with one layer per launch would be launch-bound for small batches: three
// launches per tensor).
__global__ void k_afjl_T_prep(const float *__restrict__ gtab, int l_first, const float *__restrict__ z, int64_t D,
                              int64_t b_begin, int64_t bc, float *__restrict__ w) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i >= D) return;
  const int gl = blockIdx.y;
  const float g = gtab[(int64_t)(l_first + gl) * D + i];
  float *wl = w + (int64_t)gl * bc * D;
  for (int64_t v = 0; v < bc; ++v) wl[v * D + i] = g * z[(b_begin + v) * D + i];
}

void launch_afjl_T_prep(const sk_sketch *s, int l_first, int ng, const float *z, int64_t b_begin, int64_t bc,
                        float *w, hipStream_t st) {
  hipLaunchKernelGGL(k_afjl_T_prep, dim3((unsigned)((s->D + 255) / 256), (unsigned)ng), dim3(256), 0, st, s->d_gtab,
                     l_first, z, s->D, b_begin, bc, w);
  SK_CHECK_LAUNCH();
}

// One workgroup per tile of kAfjlTRows source rows of a layer of the group
// (tiles of the group's layers numbered consecutively).  The tile's sign words
// come from one Philox block per 128 coordinates, each computed by one thread
// into LDS (a thread per 4 coordinates would repeat every block 32 times);
// each thread then writes 4 consecutive coordinates per 1024-coordinate step,
// gathering V through the digit permutation, with 16-byte stores where the
// output row allows them.
__global__ __launch_bounds__(256) void k_afjl_T_out(const LayerDesc *__restrict__ layers,
                                                    const uint16_t *__restrict__ ptab, AfjlTGroup g, int ng,
                                                    const float *__restrict__ w, int64_t D, int R, int Lw,
                                                    int64_t bc, int64_t b_begin, int out_dtype, Key key) {
  __shared__ uint32_t sgn[kAfjlTRows * 1024 / 32];
  int gl = 0;
  while (gl + 1 < ng && (int64_t)blockIdx.x >= g.tile0[gl + 1]) ++gl;
  const LayerDesc &ld = layers[g.layer[gl]];
  void *__restrict__ out = g.out[gl];
  const float *__restrict__ theta0 = g.th[gl];
  const float *wl = w + (int64_t)gl * bc * D;
  const int L = ld.L, lgL = ld.lgL;
  const int64_t h0 = ((int64_t)blockIdx.x - g.tile0[gl]) * kAfjlTRows;
  const int64_t e0 = h0 * L;  // a multiple of 512 (L >= 16)
  const int64_t tile_n = ld.n - e0 < (int64_t)kAfjlTRows * L ? ld.n - e0 : (int64_t)kAfjlTRows * L;
  const int t = threadIdx.x;
  if ((int64_t)t * 128 < tile_n) {
    const W4 wd = philox(((uint64_t)e0 >> 7) + (uint64_t)t, (uint32_t)ld.layer_id, ST_SIGN, key);
    *reinterpret_cast<uint4 *>(&sgn[4 * t]) = make_uint4(wd.w[0], wd.w[1], wd.w[2], wd.w[3]);
  }
  __syncthreads();
  const uint16_t *fk = ptab + ld.poff[0][0][ld.K - 1];
  const uint16_t *fk1 = R > 1 ? ptab + ld.poff[0][0][ld.K - 2] : nullptr;
  const bool out16 = out_dtype == SK_F32 && (reinterpret_cast<uintptr_t>(out) & 15u) == 0;
  for (int64_t e = 4 * t; e < tile_n; e += 1024) {
    const int64_t h = h0 + (e >> lgL);
    const int c = (int)(e & (L - 1));
    const int rbase = R > 1 ? ((int)fk1[h & (ld.dk1 - 1)] & (R - 1)) * L : 0;
    int idx[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) idx[q] = R > 1 ? rbase + fk[c + q] : (fk[c + q] & (Lw - 1));
    const uint32_t bits = sgn[e >> 5] >> (e & 31);
    const int64_t j = e0 + e;
    const int64_t lim = tile_n - e;
    float th[4] = {0.f, 0.f, 0.f, 0.f};
    if (theta0) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (q < lim) th[q] = theta0[j + q];
    }
    for (int64_t v = 0; v < bc; ++v) {
      const float *wv = wl + v * D;
      float o[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) o[q] = flip(wv[idx[q]], (bits >> q) & 1u) + th[q];
      const int64_t pos = (b_begin + v) * ld.n + j;
      if (out16 && lim >= 4 && (pos & 3) == 0) {
        *reinterpret_cast<float4 *>((float *)out + pos) = make_float4(o[0], o[1], o[2], o[3]);
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (q < lim) store_out(out, out_dtype, pos + q, o[q]);
      }
    }
  }
}

void launch_afjl_T_out(const sk_sketch *s, const AfjlTGroup &g, int ng, const float *w, int64_t b_begin, int64_t bc,
                       int out_dtype, hipStream_t st) {
  hipLaunchKernelGGL(k_afjl_T_out, dim3((unsigned)g.tile0[ng]), dim3(256), 0, st, s->d_layers, s->d_ptab, g, ng, w,
                     s->D, s->R, s->Lw, bc, b_begin, out_dtype, s->key);
  SK_CHECK_LAUNCH();
}

// ===========================================================================
// AFFD.  w = Scatter_pi1(B x) is written in full (padded rows as zeros) by a
// row kernel that reads source row pi1^{-1}(row) of x; then H_N' (generic
// passes); then, since only the D coordinates pi2(c), c < D, of the second
// transform are needed and those share the top digits h* = pi2_top(0), the
// top digits are contracted first: F[q] = Ttop^{-1/2} sum_t (-1)^{<h*, t>}
// g[t, q] v[t, q] (G fused), followed by H over the low block and the
// gather of pi2_low(c).
// ===========================================================================
template <bool BF16>
__global__ __launch_bounds__(256) void k_affd_prolog(const LayerDesc *__restrict__ layers,
                                                     const uint16_t *__restrict__ ptab, int layer,
                                                     const void *__restrict__ x, int64_t b_begin, int64_t bc,
                                                     float *__restrict__ w, Key key) {
  __shared__ float s[1024];
  const LayerDesc &ld = layers[layer];
  const int64_t prow = blockIdx.x;
  const int L = ld.L;
  // source row = pi1^{-1} over the row digits 0..K-2
  int64_t srow = 0, stride = 1;
  for (int k = ld.K - 2; k >= 0; --k) {
    const int64_t dig = (prow / stride) & ((1ll << ld.lg[k]) - 1);
    srow += (int64_t)ptab[ld.poff[0][1][k] + dig] * stride;
    stride <<= ld.lg[k];
  }
  const int col0 = threadIdx.x * 4;
  const uint16_t *fk = ptab + ld.poff[0][0][ld.K - 1];
  const int64_t j0 = srow * L + col0;
  const int64_t lim = ld.n - j0;
  const bool live = srow < ld.rows_live && col0 < L && lim > 0;
  uint32_t bits = 0;
  int pc[4] = {0, 0, 0, 0};
  if (col0 < L) {
#pragma unroll
    for (int q = 0; q < 4; ++q) pc[q] = fk[col0 + q];
  }
  if (live) bits = sign_word((uint64_t)j0, (uint32_t)ld.layer_id, key) >> (j0 & 31);
  for (int64_t v = 0; v < bc; ++v) {
    float val[4] = {0.f, 0.f, 0.f, 0.f};
    if (live) {
      load4<BF16, false>(x, (b_begin + v) * ld.n + j0, lim, val);
#pragma unroll
      for (int q = 0; q < 4; ++q) val[q] = flip(val[q], (bits >> q) & 1u);
    }
    if (col0 < L) {
#pragma unroll
      for (int q = 0; q < 4; ++q) s[pc[q]] = val[q];
    }
    __syncthreads();
    float *dst = w + v * ld.np + prow * L;
    for (int c = threadIdx.x; c < L; c += 256) dst[c] = s[c];
    __syncthreads();
  }
}

void launch_affd_prolog(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc,
                        float *w, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const unsigned rows = (unsigned)(ld.np / ld.L);
  if (dtype == SK_BF16)
    hipLaunchKernelGGL(k_affd_prolog<true>, dim3(rows), dim3(256), 0, st, s->d_layers, s->d_ptab, layer, x, b_begin,
                       bc, w, s->key);
  else
    hipLaunchKernelGGL(k_affd_prolog<false>, dim3(rows), dim3(256), 0, st, s->d_layers, s->d_ptab, layer, x, b_begin,
                       bc, w, s->key);
  SK_CHECK_LAUNCH();
}

// F[v, q] over q < 2^lo_len_lg; thread: 4 consecutive q, 8 vectors.
__global__ __launch_bounds__(256) void k_affd_fold(const LayerDesc *__restrict__ layers, int layer,
                                                   const float *__restrict__ w, int64_t bc, float *__restrict__ f,
                                                   Key key) {
  const LayerDesc &ld = layers[layer];
  const int64_t lo_len = 1ll << ld.lo_len_lg;
  const int64_t q0 = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) * 4;
  if (q0 >= lo_len) return;
  const int64_t v0 = blockIdx.y * 8;
  const int nv = (int)((bc - v0) < 8 ? (bc - v0) : 8);
  const int64_t ttop = ld.np >> ld.lo_len_lg;
  float acc[8][4];
#pragma unroll
  for (int v = 0; v < 8; ++v)
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[v][i] = 0.0f;
  for (int64_t t = 0; t < ttop; ++t) {
    const uint32_t sgn = __popcll((uint64_t)t & ld.hstar) & 1u;
    const int64_t j = t * lo_len + q0;
    float g[4];
    gauss4((uint64_t)j >> 2, (uint32_t)ld.layer_id, ST_GAUSS, key, g);
#pragma unroll
    for (int v = 0; v < 8; ++v) {
      if (v < nv) {
        const float4 x = *(const float4 *)(w + (v0 + v) * ld.np + j);
        acc[v][0] += flip(g[0] * x.x, sgn);
        acc[v][1] += flip(g[1] * x.y, sgn);
        acc[v][2] += flip(g[2] * x.z, sgn);
        acc[v][3] += flip(g[3] * x.w, sgn);
      }
    }
  }
  const float sc = (float)(1.0 / sqrt((double)ttop));
#pragma unroll
  for (int v = 0; v < 8; ++v) {
    if (v < nv) {
      float4 o = make_float4(acc[v][0] * sc, acc[v][1] * sc, acc[v][2] * sc, acc[v][3] * sc);
      *(float4 *)(f + (v0 + v) * lo_len + q0) = o;
    }
  }
}

void launch_affd_fold(const sk_sketch *s, int layer, const float *w, int64_t bc, float *f, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const int64_t lo_len = 1ll << ld.lo_len_lg;
  dim3 grid((unsigned)((lo_len / 4 + 255) / 256), (unsigned)((bc + 7) / 8));
  hipLaunchKernelGGL(k_affd_fold, grid, dim3(256), 0, st, s->d_layers, layer, w, bc, f, s->key);
  SK_CHECK_LAUNCH();
}

// pi2 on the low block: index c < D -> position in F.
__device__ __forceinline__ int64_t pi2_low(const LayerDesc &ld, const uint16_t *ptab, int64_t c, int64_t D) {
  const int64_t L = ld.L;
  if (D > L) {
    const int64_t a = c >> ld.lgL, b = c & (L - 1);
    return (int64_t)ptab[ld.poff[1][0][ld.K - 2] + a] * L + ptab[ld.poff[1][0][ld.K - 1] + b];
  }
  return ptab[ld.poff[1][0][ld.K - 1] + c];
}

__global__ void k_affd_gather(const LayerDesc *__restrict__ layers, const uint16_t *__restrict__ ptab, int layer,
                              const float *__restrict__ f, int64_t D, int64_t b_begin, int64_t bc,
                              float *__restrict__ out, int accumulate) {
  const LayerDesc &ld = layers[layer];
  const int64_t c = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (c >= D) return;
  const int64_t lo_len = 1ll << ld.lo_len_lg;
  const int64_t p = pi2_low(ld, ptab, c, D);
  const float sc = (float)sqrt((double)ld.np / (double)D);
  for (int64_t v = 0; v < bc; ++v) {
    const float val = sc * f[v * lo_len + p];
    float *o = out + (b_begin + v) * D + c;
    *o = accumulate ? *o + val : val;
  }
}

void launch_affd_gather(const sk_sketch *s, int layer, const float *f, int64_t b_begin, int64_t bc, float *out,
                        bool accumulate, hipStream_t st) {
  hipLaunchKernelGGL(k_affd_gather, dim3((unsigned)((s->D + 255) / 256)), dim3(256), 0, st, s->d_layers, s->d_ptab,
                     layer, f, s->D, b_begin, bc, out, (int)accumulate);
  SK_CHECK_LAUNCH();
}

// AFFD transpose, first step: Scatter_pi2 R_D^T z into a zeroed w.
__global__ void k_affd_T_scatter(const LayerDesc *__restrict__ layers, const uint16_t *__restrict__ ptab, int layer,
                                 const float *__restrict__ z, int64_t D, int64_t b_begin, int64_t bc,
                                 float *__restrict__ w) {
  const LayerDesc &ld = layers[layer];
  const int64_t c = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (c >= D) return;
  const int64_t p = ((int64_t)ld.hstar << ld.lo_len_lg) + pi2_low(ld, ptab, c, D);
  for (int64_t v = 0; v < bc; ++v) w[v * ld.np + p] = z[(b_begin + v) * D + c];
}

void launch_affd_T_scatter(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, float *w,
                           hipStream_t st) {
  hipLaunchKernelGGL(k_affd_T_scatter, dim3((unsigned)((s->D + 255) / 256)), dim3(256), 0, st, s->d_layers,
                     s->d_ptab, layer, z, s->D, b_begin, bc, w);
  SK_CHECK_LAUNCH();
}

__global__ void k_mul_gauss(const LayerDesc *__restrict__ layers, int layer, float *__restrict__ w, int64_t bc,
                            Key key) {
  const LayerDesc &ld = layers[layer];
  const int64_t j = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) * 4;
  if (j >= ld.np) return;
  float g[4];
  gauss4((uint64_t)j >> 2, (uint32_t)ld.layer_id, ST_GAUSS, key, g);
  for (int64_t v = 0; v < bc; ++v) {
    float4 *p = (float4 *)(w + v * ld.np + j);
    float4 x = *p;
    x.x *= g[0];
    x.y *= g[1];
    x.z *= g[2];
    x.w *= g[3];
    *p = x;
  }
}

void launch_mul_gauss(const sk_sketch *s, int layer, float *w, int64_t bc, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  hipLaunchKernelGGL(k_mul_gauss, dim3((unsigned)((ld.np / 4 + 255) / 256)), dim3(256), 0, st, s->d_layers, layer, w,
                     bc, s->key);
  SK_CHECK_LAUNCH();
}

// out[j] = sqrt(N'/D) b_j w[pi1(j)] (+ theta0[j]); one workgroup per source row.
__global__ __launch_bounds__(256) void k_affd_T_out(const LayerDesc *__restrict__ layers,
                                                    const uint16_t *__restrict__ ptab, int layer,
                                                    const float *__restrict__ w, int64_t D, int64_t bc,
                                                    int64_t b_begin, void *__restrict__ out, int out_dtype,
                                                    const float *__restrict__ theta0, Key key) {
  const LayerDesc &ld = layers[layer];
  const int64_t h = blockIdx.x;
  const int L = ld.L;
  const int col0 = threadIdx.x * 4;
  if (col0 >= L) return;
  const int64_t j0 = h * L + col0;
  const int64_t lim = ld.n - j0;
  if (lim <= 0) return;
  int64_t prow = 0, stride = 1;
  for (int k = ld.K - 2; k >= 0; --k) {
    const int64_t dig = (h / stride) & ((1ll << ld.lg[k]) - 1);
    prow += (int64_t)ptab[ld.poff[0][0][k] + dig] * stride;
    stride <<= ld.lg[k];
  }
  const uint16_t *fk = ptab + ld.poff[0][0][ld.K - 1];
  int64_t idx[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) idx[q] = prow * L + fk[col0 + q];
  const uint32_t bits = sign_word((uint64_t)j0, (uint32_t)ld.layer_id, key) >> (j0 & 31);
  const float sc = (float)sqrt((double)ld.np / (double)D);
  float th[4] = {0.f, 0.f, 0.f, 0.f};
  if (theta0) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (q < lim) th[q] = theta0[j0 + q];
  }
  for (int64_t v = 0; v < bc; ++v) {
    const float *wv = w + v * ld.np;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (q < lim)
        store_out(out, out_dtype, (b_begin + v) * ld.n + j0 + q, flip(sc * wv[idx[q]], (bits >> q) & 1u) + th[q]);
  }
}

void launch_affd_T_out(const sk_sketch *s, int layer, const float *w, int64_t b_begin, int64_t bc, void *out,
                       int out_dtype, const float *theta0, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  hipLaunchKernelGGL(k_affd_T_out, dim3((unsigned)ld.rows_live), dim3(256), 0, st, s->d_layers, s->d_ptab, layer, w,
                     s->D, bc, b_begin, out, out_dtype, theta0, s->key);
  SK_CHECK_LAUNCH();
}

// ===========================================================================
// FJL: w = B x zero-padded, H_N' (generic passes), y_i = sqrt(N'/D) g_i w[idx_i].
// ===========================================================================
// FJL forward, first transform pass fused with the signed load: one workgroup per
// (vector, tile of 2^w coordinates of N'), w = min(log2 N', 13); the tile's sign
// words (one Philox block per 128 coordinates) are built in LDS, the signed
// inputs (zeros past n) transformed over bits [0, w) in LDS and written to the
// workspace [vector][N'] with the pass scale.  The remaining bits go through
// fwht_inplace_from(w).
template <bool BF16>
__global__ __launch_bounds__(256) void k_fjl_pass0(const LayerDesc *__restrict__ layers, int layer,
                                                   const void *__restrict__ x, int w, int64_t b_begin,
                                                   float *__restrict__ out, float scale, Key key) {
  extern __shared__ float sm[];
  const LayerDesc &ld = layers[layer];
  const int T = 1 << w;
  float *s = sm;
  uint32_t *sgn = reinterpret_cast<uint32_t *>(sm + ((p16_floats(T) + 3) & ~3));  // 16-byte aligned
  const int64_t tiles = ld.np >> w;
  const int64_t v = blockIdx.x / tiles;
  const int64_t base = (blockIdx.x - v * tiles) << w;
  const int nblk = (T + 127) >> 7;  // T >= 16: base is a multiple of T
  if ((int)threadIdx.x < nblk && base + 128 * (int64_t)threadIdx.x < ld.n) {
    const W4 wd = philox(((uint64_t)base >> 7) + threadIdx.x, (uint32_t)ld.layer_id, ST_SIGN, key);
    *reinterpret_cast<uint4 *>(&sgn[4 * threadIdx.x]) = make_uint4(wd.w[0], wd.w[1], wd.w[2], wd.w[3]);
  }
  __syncthreads();
  const int64_t row = (b_begin + v) * ld.n;
  for (int e = threadIdx.x; e < T; e += 256) {
    const int64_t j = base + e;
    float val = 0.0f;
    if (j < ld.n) {
      const float xv = BF16 ? bf16_to_f32(((const uint16_t *)x)[row + j]) : ((const float *)x)[row + j];
      // base is 128-aligned when T >= 128; smaller tiles are the whole vector (base = 0)
      val = flip(xv, (sgn[((int64_t)e >> 5)] >> (j & 31)) & 1u);
    }
    s[p16(e)] = val;
  }
  lds_fwht_regs(s, w, 0);
  float *o = out + v * ld.np + base;
  for (int e = threadIdx.x; e < T; e += 256) o[e] = s[p16(e)] * scale;
}

void launch_fjl_pass0(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc, float *w,
                      int lgw, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const int64_t tiles = bc * (ld.np >> lgw);
  const size_t shm = sizeof(float) * ((p16_floats(1 << lgw) + 3) & ~3) + sizeof(uint32_t) * ((((1 << lgw) + 127) >> 7) * 4);
  const float scale = (float)(1.0 / std::sqrt((double)(1ll << lgw)));
  if (dtype == SK_BF16)
    hipLaunchKernelGGL(k_fjl_pass0<true>, dim3((unsigned)tiles), dim3(256), shm, st, s->d_layers, layer, x, lgw,
                       b_begin, w, scale, s->key);
  else
    hipLaunchKernelGGL(k_fjl_pass0<false>, dim3((unsigned)tiles), dim3(256), shm, st, s->d_layers, layer, x, lgw,
                       b_begin, w, scale, s->key);
  SK_CHECK_LAUNCH();
}

__global__ void k_fjl_gather(const LayerDesc *__restrict__ layers, const float *__restrict__ gtab, int layer,
                             const float *__restrict__ w, int64_t D, int64_t b_begin, int64_t bc,
                             float *__restrict__ out, int accumulate, Key key) {
  const LayerDesc &ld = layers[layer];
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i >= D) return;
  const uint32_t idx = sample_index((uint64_t)i, (uint32_t)ld.layer_id, key, (uint64_t)ld.np);
  const float g = gtab[(int64_t)layer * D + i] * (float)sqrt((double)ld.np / (double)D);
  for (int64_t v = 0; v < bc; ++v) {
    const float val = g * w[v * ld.np + idx];
    float *o = out + (b_begin + v) * D + i;
    *o = accumulate ? *o + val : val;
  }
}

void launch_fjl_gather(const sk_sketch *s, int layer, const float *w, int64_t b_begin, int64_t bc, float *out,
                       bool accumulate, hipStream_t st) {
  hipLaunchKernelGGL(k_fjl_gather, dim3((unsigned)((s->D + 255) / 256)), dim3(256), 0, st, s->d_layers, s->d_gtab,
                     layer, w, s->D, b_begin, bc, out, (int)accumulate, s->key);
  SK_CHECK_LAUNCH();
}

// FJL forward, last transform pass fused with the gather of the D samples: the
// pass over index bits [lo, lo + w) = the top bits, one workgroup per (vector,
// block of 2^lgcs low positions); after the transform the workgroup writes
// out[i] = sqrt(N'/D) g_i w[idx_i] for the samples whose position falls in its
// block (a list sorted by block at creation), and nothing else.
__global__ __launch_bounds__(256) void k_fjl_last_gather(const float *__restrict__ data, int lgn, int lo, int w,
                                                         int lgcs, float scale, const uint32_t *__restrict__ smp,
                                                         const uint32_t *__restrict__ spos,
                                                         const uint32_t *__restrict__ soff,
                                                         const float *__restrict__ g, float gscale, int64_t D,
                                                         int64_t b_begin, float *__restrict__ out, int accumulate) {
  extern __shared__ float sm[];
  const int64_t n = 1ll << lgn;
  const int64_t tiles = n >> (w + lgcs);
  const int64_t v = blockIdx.x / tiles;
  const int64_t cb = blockIdx.x - v * tiles;
  const float *base = data + v * n + (cb << lgcs);
  const int total = 1 << (w + lgcs);
  const int cmask = (1 << lgcs) - 1;
  for (int e = threadIdx.x; e < total; e += 256) sm[p16(e)] = base[((int64_t)(e >> lgcs) << lo) + (e & cmask)];
  lds_fwht_regs(sm, w + lgcs, lgcs);
  const uint32_t k0 = soff[cb], k1 = soff[cb + 1];
  float *o = out + (b_begin + v) * D;
  for (uint32_t k = k0 + threadIdx.x; k < k1; k += 256) {
    const uint32_t i = smp[k], p = spos[k];
    const int e = (int)(((p >> lo) << lgcs) + (p & cmask));
    const float val = (g[i] * gscale) * (sm[p16(e)] * scale);
    o[i] = accumulate ? o[i] + val : val;
  }
}

void launch_fjl_last_gather(const sk_sketch *s, int layer, const float *w, int64_t b_begin, int64_t bc, float *out,
                            bool accumulate, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  int los[64], ws[64], lgcss[64];
  const int np = fwht_pass_plan(ld.lgnp, std::min(ld.lgnp, 13), los, ws, lgcss);
  const int lo = los[np - 1], wl = ws[np - 1], lgcs = lgcss[np - 1];
  const int64_t tiles = bc * ((1ll << ld.lgnp) >> (wl + lgcs));
  const size_t shm = sizeof(float) * p16_floats(1 << (wl + lgcs));
  const float scale = (float)(1.0 / sqrt((double)(1ll << wl)));
  const int64_t so = s->fjl_loff_at[layer];
  hipLaunchKernelGGL(k_fjl_last_gather, dim3((unsigned)tiles), dim3(256), shm, st, w, ld.lgnp, lo, wl, lgcs, scale,
                     s->d_fjl_lsmp + (int64_t)layer * s->D, s->d_fjl_lpos + (int64_t)layer * s->D, s->d_fjl_loff + so,
                     s->d_gtab + (int64_t)layer * s->D, (float)sqrt((double)ld.np / (double)s->D), s->D, b_begin,
                     out, (int)accumulate);
  SK_CHECK_LAUNCH();
}

// FJL transpose, last transform pass fused with the signed output: the pass
// over index bits [lo, lo + w) (the top bits; runs of 2^lgcs >= 32
// consecutive positions per row of the tile), then
// out[j] = oscale b_j (H w)[j] (+ theta0[j]) for the positions j < n of the
// tile, so the transformed vector is never written back.  The tile's sign
// words are built into LDS first (one word per 32 positions of a run).
__global__ __launch_bounds__(256) void k_fjl_last_signed(const LayerDesc *__restrict__ layers, int layer,
                                                         const float *__restrict__ data, int lo, int w, int lgcs,
                                                         float scale, int64_t b_begin, void *__restrict__ out,
                                                         int out_dtype, const float *__restrict__ theta0, Key key) {
  extern __shared__ float sm[];
  const LayerDesc &ld = layers[layer];
  const int lgn = ld.lgnp;
  const int64_t n = ld.n;
  const int total = 1 << (w + lgcs);
  float *sv = sm;
  uint32_t *sw = reinterpret_cast<uint32_t *>(sm + p16_floats(total));
  const int64_t tiles_per_vec = (1ll << lgn) >> (w + lgcs);
  const int64_t v = blockIdx.x / tiles_per_vec;
  const int64_t tv = blockIdx.x - v * tiles_per_vec;
  const int lgcb = lo - lgcs;
  const int64_t j0 = ((tv >> lgcb) << (lo + w)) + ((tv & ((1ll << lgcb) - 1)) << lgcs);  // first position
  const float *base = data + v * (1ll << lgn) + j0;
  const int cmask = (1 << lgcs) - 1;
  const int lgwpr = lgcs - 5;  // sign words per row of the tile
  for (int k = threadIdx.x; k < (total >> 5); k += 256) {
    const int64_t j = j0 + ((int64_t)(k >> lgwpr) << lo) + ((int64_t)(k & ((1 << lgwpr) - 1)) << 5);
    sw[k] = sign_word((uint64_t)j, (uint32_t)ld.layer_id, key);
  }
  for (int e = threadIdx.x; e < total; e += 256) sv[p16(e)] = base[((int64_t)(e >> lgcs) << lo) + (e & cmask)];
  lds_fwht_regs(sv, w + lgcs, lgcs);
  const int64_t ob = (b_begin + v) * n;
  for (int e = threadIdx.x; e < total; e += 256) {
    const int64_t j = j0 + ((int64_t)(e >> lgcs) << lo) + (e & cmask);
    if (j < n) {
      float val = flip(sv[p16(e)] * scale, (sw[e >> 5] >> (e & 31)) & 1u);
      if (theta0) val += theta0[j];
      store_out(out, out_dtype, ob + j, val);
    }
  }
}

// True when the FJL transpose of a layer ends with a pass that
// k_fjl_last_signed can take (a pass after bit lo0 whose tile rows hold runs of
// at least 32 consecutive positions).
bool fjl_last_signed_ok(const sk_sketch *s, int layer, int lo0) {
  const LayerDesc &ld = s->layers[layer];
  int los[64], ws[64], lgcss[64];
  const int np = fwht_pass_plan(ld.lgnp, lo0, los, ws, lgcss);
  return np >= 1 && lo0 < ld.lgnp && lgcss[np - 1] >= 5;
}

void launch_fjl_last_signed(const sk_sketch *s, int layer, const float *w, int lo0, int64_t b_begin, int64_t bc,
                            void *out, int out_dtype, const float *theta0, float oscale, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  int los[64], ws[64], lgcss[64];
  const int np = fwht_pass_plan(ld.lgnp, lo0, los, ws, lgcss);
  const int lo = los[np - 1], wl = ws[np - 1], lgcs = lgcss[np - 1];
  const int64_t tiles = bc * ((1ll << ld.lgnp) >> (wl + lgcs));
  const size_t shm = sizeof(float) * p16_floats(1 << (wl + lgcs)) + sizeof(uint32_t) * ((1 << (wl + lgcs)) >> 5);
  const float scale = (float)(oscale / std::sqrt((double)(1ll << wl)));
  hipLaunchKernelGGL(k_fjl_last_signed, dim3((unsigned)tiles), dim3(256), shm, st, s->d_layers, layer, w, lo, wl,
                     lgcs, scale, b_begin, out, out_dtype, theta0, s->key);
  SK_CHECK_LAUNCH();
}

// FJL transpose in one pass, 2^14 <= N' <= 2^21, D <= 2^13 (the adjoint of
// eq. ailon_chazelle).  With N' = 2^(13 + H) a coordinate is j = (h, a, c): h
// the top H bits, a the next H, c the low B = 13 - H (>= 5); the normalised
// transform factors as H_N'[j, p] = H[h, p_h] H[a, p_a] H[c, p_c] / sqrt(N').
// Workgroup (a, vector): the 2^H x 2^B tile U[p_h][p_c] = sum over samples i
// at (p_h, p_a, p_c) of H[a, p_a] g_i z_i, its unnormalised 13-bit transform,
// then signs, the scale 1/sqrt(D) and theta0; every output is written once.
// The products H[a, p_a] g_i z_i are made first, all loads of a thread in
// flight together, and staged in LDS in cell order; each cell is then summed
// by one thread in id order (deterministic), the cell offsets loaded in one
// batch.
bool fjl_onepass_T_ok(int lgnp, int64_t D) { return lgnp >= 14 && lgnp <= 21 && D <= (1 << 13); }

template <int R>  // entries per thread: D <= 256 R
__global__ __launch_bounds__(256) void k_fjl_T_onepass(const LayerDesc *__restrict__ layers, int layer,
                                                       const float *__restrict__ gtab,
                                                       const uint32_t *__restrict__ boff,
                                                       const uint32_t *__restrict__ bent,
                                                       const float *__restrict__ z, int D, int64_t b_begin,
                                                       void *__restrict__ out, int out_dtype,
                                                       const float *__restrict__ theta0, float scale, Key key) {
  extern __shared__ float sm[];
  float *tile = sm;                                                        // p16 layout, 2^13 cells
  float *ce = sm;                                                          // first: the D products, cell order
  uint32_t *sw = reinterpret_cast<uint32_t *>(sm + p16_floats(1 << 13));  // sign words in tile order
  const LayerDesc &ld = layers[layer];
  const int H = ld.lgnp - 13, B = 13 - H;
  const int a = blockIdx.x;
  const int64_t v = blockIdx.y;
  const float *g = gtab + (int64_t)layer * D;
  const float *zv = z + (b_begin + v) * D;
  // cell offsets of the thread's 32 cells k = tid + 256 m, both ends
  uint32_t o0[32], o1[32];
#pragma unroll
  for (int m = 0; m < 32; ++m) {
    o0[m] = boff[threadIdx.x + 256 * m];
    o1[m] = boff[threadIdx.x + 256 * m + 1];
  }
  // products of entries e = tid + 256 r (r < R)
  {
    uint32_t q[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int e = threadIdx.x + 256 * r;
      q[r] = e < D ? bent[e] : 0u;
    }
    float gz[R];
    if (R <= 16) {
      // D <= 4096: g z by id, loaded in order, staged after the products (inside the tile), then
      // gathered from LDS in cell order
      float *gzs = sm + D;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int i = threadIdx.x + 256 * r;
        if (i < D) gzs[i] = g[i] * zv[i];
      }
      __syncthreads();
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int e = threadIdx.x + 256 * r;
        gz[r] = e < D ? gzs[q[r] >> 8] : 0.0f;
      }
    } else {
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int e = threadIdx.x + 256 * r;
        const uint32_t i = q[r] >> 8;
        gz[r] = e < D ? g[i] * zv[i] : 0.0f;
      }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int e = threadIdx.x + 256 * r;
      if (e < D) ce[e] = flip(gz[r], (uint32_t)__popc((uint32_t)a & q[r] & 255u) & 1u);
    }
  }
  {
    // word w: tile cells 32 w .. 32 w + 31 = row h = w >> (B - 5), columns from 32 (w mod 2^(B - 5))
    const int w = threadIdx.x;
    const int64_t j = ((int64_t)(w >> (B - 5)) << 13) + ((int64_t)a << B) + ((w & ((1 << (B - 5)) - 1)) << 5);
    sw[w] = sign_word((uint64_t)j, (uint32_t)ld.layer_id, key);
  }
  __syncthreads();
  float u[32];
#pragma unroll
  for (int m = 0; m < 32; ++m) {
    float acc = 0.0f;
    for (uint32_t e = o0[m]; e < o1[m]; ++e) acc += ce[e];
    u[m] = acc;
  }
  __syncthreads();  // the products are read; the tile takes their place
#pragma unroll
  for (int m = 0; m < 32; ++m) tile[p16(threadIdx.x + 256 * m)] = u[m];
  lds_fwht_regs(tile, 13, 0);  // opens and closes with a barrier
  const int64_t row = (b_begin + v) * ld.n;
  for (int m = 0; m < 32; ++m) {
    const int k = threadIdx.x + 256 * m;
    const int64_t j = ((int64_t)(k >> B) << 13) + ((int64_t)a << B) + (k & ((1 << B) - 1));
    if (j < ld.n) {
      float val = flip(tile[p16(k)] * scale, (sw[k >> 5] >> (k & 31)) & 1u);
      if (theta0) val += theta0[j];
      store_out(out, out_dtype, row + j, val);
    }
  }
}

// FJL forward in one pass for the same layers (eq. ailon_chazelle), the
// factorisation above read the other way: workgroup (a, vector) loads the
// tile X[h][c] = b_j x_j of the coordinates j = (h, a, c) (runs of 2^B >= 32
// consecutive ones), transforms it (Y = (H (x) H) X over all 13 bits), and
// writes for every sample i at p = (p_h, p_a, p_c) its share
// H[a, p_a] Y[p_h][p_c] g_i / sqrt(D) into partial slot a; the 2^H slots are
// then summed in a fixed order (launch_reduce_partials).
template <bool BF16, int R>
__global__ __launch_bounds__(256) void k_fjl_fwd_onepass(const LayerDesc *__restrict__ layers, int layer,
                                                         const float *__restrict__ gtab,
                                                         const uint32_t *__restrict__ bpos,
                                                         const void *__restrict__ x, int D, int64_t b_begin,
                                                         int64_t bc, float *__restrict__ part, float scale, Key key) {
  extern __shared__ float sm[];
  float *tile = sm;                                                        // p16 layout, 2^13 cells
  uint32_t *sw = reinterpret_cast<uint32_t *>(sm + p16_floats(1 << 13));  // sign words in tile order
  const LayerDesc &ld = layers[layer];
  const int H = ld.lgnp - 13, B = 13 - H;
  const int a = blockIdx.x;
  const int64_t v = blockIdx.y;
  const int64_t row = (b_begin + v) * ld.n;
  // coordinates past the layer's end read its last one (always valid) and are replaced by zero,
  // a select rather than a branch per element
  // (N' <= 2^21: coordinates fit 32-bit offsets from the row's uniform base)
  const uint16_t *xh = (const uint16_t *)x + row;
  const float *xf = (const float *)x + row;
  const uint32_t nlast = (uint32_t)(ld.n - 1);
  float xv[32];
#pragma unroll
  for (int m = 0; m < 32; ++m) {
    const int k = threadIdx.x + 256 * m;
    const uint32_t j = ((uint32_t)(k >> B) << 13) + ((uint32_t)a << B) + (uint32_t)(k & ((1 << B) - 1));
    const uint32_t jc = j < nlast ? j : nlast;
    const float t = BF16 ? bf16_to_f32(xh[jc]) : xf[jc];
    xv[m] = j <= nlast ? t : 0.0f;
  }
  {
    const int w = threadIdx.x;
    const int64_t j = ((int64_t)(w >> (B - 5)) << 13) + ((int64_t)a << B) + ((w & ((1 << (B - 5)) - 1)) << 5);
    sw[w] = sign_word((uint64_t)j, (uint32_t)ld.layer_id, key);
  }
  __syncthreads();
#pragma unroll
  for (int m = 0; m < 32; ++m) {
    const int k = threadIdx.x + 256 * m;
    tile[p16(k)] = flip(xv[m], (sw[k >> 5] >> (k & 31)) & 1u);
  }
  lds_fwht_regs(tile, 13, 0);  // opens and closes with a barrier
  const float *g = gtab + (int64_t)layer * D;
  float *o = part + ((int64_t)a * bc + v) * D;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int i = threadIdx.x + 256 * r;
    if (i < D) {
      const uint32_t q = bpos[i];
      o[i] = flip(tile[p16((int)(q >> 8))], (uint32_t)__popc((uint32_t)a & q & 255u) & 1u) * (g[i] * scale);
    }
  }
}

void launch_fjl_fwd_onepass(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc,
                            float *part, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const int H = ld.lgnp - 13;
  const size_t shm = sizeof(float) * p16_floats(1 << 13) + sizeof(uint32_t) * 256;
  const float scale = (float)(1.0 / std::sqrt((double)s->D));
  const uint32_t *bpos = s->d_fjlb_pos + s->fjlb_pos_at[layer];
#define SK_FJLF1(BF, R)                                                                                          \
  hipLaunchKernelGGL((k_fjl_fwd_onepass<BF, R>), dim3(1u << H, (unsigned)bc), dim3(256), shm, st, s->d_layers,     \
                     layer, s->d_gtab, bpos, x, (int)s->D, b_begin, bc, part, scale, s->key)
  if (dtype == SK_BF16) {
    if (s->D <= 4096) SK_FJLF1(true, 16); else SK_FJLF1(true, 32);
  } else {
    if (s->D <= 4096) SK_FJLF1(false, 16); else SK_FJLF1(false, 32);
  }
#undef SK_FJLF1
  SK_CHECK_LAUNCH();
}

void launch_fjl_T_onepass(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, void *out,
                          int out_dtype, const float *theta0, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const int H = ld.lgnp - 13;
  const size_t shm = sizeof(float) * p16_floats(1 << 13) + sizeof(uint32_t) * 256;
  const float scale = (float)(1.0 / std::sqrt((double)s->D));
#define SK_FJLT1(R)                                                                                              \
  hipLaunchKernelGGL(k_fjl_T_onepass<R>, dim3(1u << H, (unsigned)bc), dim3(256), shm, st, s->d_layers, layer,      \
                     s->d_gtab, s->d_fjlb_off + s->fjlb_off_at[layer], s->d_fjlb_ent + s->fjlb_ent_at[layer], z,   \
                     (int)s->D, b_begin, out, out_dtype, theta0, scale, s->key)
  if (s->D <= 4096)
    SK_FJLT1(16);
  else
    SK_FJLT1(32);
#undef SK_FJLT1
  SK_CHECK_LAUNCH();
}

// FJL transpose, first transform pass fused with the scatter of the D samples:
// one workgroup per (vector, tile of 2^w positions of N'), w = min(log2 N', 13).
// The tile starts at zero in LDS; every unique sample position inside it (a
// contiguous run of the position-sorted list, located by the tile table) gets
// the sum of g_i z_i over its samples in id order; then bits [0, w) are
// transformed and the tile written to the workspace [vector][N'] with the pass
// scale.  The remaining bits go through fwht_inplace_from(w).
__global__ __launch_bounds__(256) void k_fjl_T_pass0(const float *__restrict__ gtab, int layer,
                                                     const uint32_t *__restrict__ pos, const uint32_t *__restrict__ seg,
                                                     const uint32_t *__restrict__ smp,
                                                     const uint32_t *__restrict__ toff, int64_t np, int w,
                                                     const float *__restrict__ z, int64_t D, int64_t b_begin,
                                                     float *__restrict__ out, float scale) {
  extern __shared__ float sm[];
  const int T = 1 << w;
  const int64_t tiles = np >> w;
  const int64_t v = blockIdx.x / tiles;
  const int64_t t = blockIdx.x - v * tiles;
  const int64_t base = t << w;
  for (int e = threadIdx.x; e < T; e += 256) sm[p16(e)] = 0.0f;
  __syncthreads();
  const float *g = gtab + (int64_t)layer * D;
  const float *zv = z + (b_begin + v) * D;
  const uint32_t u1 = toff[t + 1];
  for (uint32_t u = toff[t] + threadIdx.x; u < u1; u += 256) {
    float acc = 0.0f;
    const uint32_t k1 = seg[u + 1];
    for (uint32_t k = seg[u]; k < k1; ++k) {
      const uint32_t i = smp[k];
      acc += g[i] * zv[i];
    }
    sm[p16((int)(pos[u] - base))] = acc;  // positions are unique: no two threads share a slot
  }
  lds_fwht_regs(sm, w, 0);  // opens and closes with a barrier
  float *o = out + v * np + base;
  for (int e = threadIdx.x; e < T; e += 256) o[e] = sm[p16(e)] * scale;
}

void launch_fjl_T_pass0(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, float *w, int lgw,
                        hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const int64_t u0 = s->fjl_uoff[layer];
  const int64_t seg0 = u0 + layer;  // one sentinel per layer
  const int64_t tiles = bc * (ld.np >> lgw);
  const size_t shm = sizeof(float) * p16_floats(1 << lgw);
  const float scale = (float)(1.0 / std::sqrt((double)(1ll << lgw)));
  hipLaunchKernelGGL(k_fjl_T_pass0, dim3((unsigned)tiles), dim3(256), shm, st, s->d_gtab, layer, s->d_fjl_pos + u0,
                     s->d_fjl_seg + seg0, s->d_fjl_smp, s->d_fjl_toff + s->fjl_toff_at[layer], ld.np, lgw, z, s->D,
                     b_begin, w, scale);
  SK_CHECK_LAUNCH();
}

// out[j] = scale b_j w[j] (+ theta0[j]) for j < n.
__global__ void k_signed_out(const LayerDesc *__restrict__ layers, int layer, const float *__restrict__ w,
                             int64_t b_begin, int64_t bc, void *__restrict__ out, int out_dtype,
                             const float *__restrict__ theta0, float scale, Key key) {
  const LayerDesc &ld = layers[layer];
  const int64_t j0 = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) * 4;
  const int64_t lim = ld.n - j0;
  if (lim <= 0) return;
  const uint32_t bits = sign_word((uint64_t)j0, (uint32_t)ld.layer_id, key) >> (j0 & 31);
  float th[4] = {0.f, 0.f, 0.f, 0.f};
  if (theta0) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (q < lim) th[q] = theta0[j0 + q];
  }
  for (int64_t v = 0; v < bc; ++v) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (q < lim)
        store_out(out, out_dtype, (b_begin + v) * ld.n + j0 + q,
                  flip(scale * w[v * ld.np + j0 + q], (bits >> q) & 1u) + th[q]);
  }
}

void launch_signed_out(const sk_sketch *s, int layer, const float *w, int64_t b_begin, int64_t bc, void *out,
                       int out_dtype, const float *theta0, float scale, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  hipLaunchKernelGGL(k_signed_out, dim3((unsigned)((ld.n / 4 + 1 + 255) / 256)), dim3(256), 0, st, s->d_layers,
                     layer, w, b_begin, bc, out, out_dtype, theta0, scale, s->key);
  SK_CHECK_LAUNCH();
}

// ===========================================================================
// FFD.  Forward (the explicit sketch) y = sum_b B_b H_D Pi_b^T G_b H_D x_b with
// (Pi v)_i = v_{pi_b(i)}; transpose (the feature map of eq. fastfood) block b
// = H_D G_b Pi_b H_D B_b z.  Blocks past the data are all zero (skipped).
// Small D: a whole block lives in LDS.  Large D: generic passes over a
// workspace holding every live block of every vector.
// ===========================================================================
int64_t ffd_live_blocks(const sk_sketch *s, int layer) {
  const LayerDesc &ld = s->layers[layer];
  return (ld.n + s->D - 1) / s->D;
}

// Partial sums of the small-D forward: one per live block (and vector).
int64_t ffd_small_groups(const sk_sketch *s, int layer) { return ffd_live_blocks(s, layer); }

// The random ingredients of the live blocks of a layer (D <= 2^13), made once
// per call by k_ffd_tables into the workspace and read by the block kernels:
// g_b (nlive x D floats), Pi_b (nlive x D 16-bit entries) and the sign bits of
// the block's coordinates (nlive rows of ffd_tab_words(D) words, bit i % 32 of
// word i / 32 for coordinate b D + i).  Nothing is kept between calls.
__host__ __device__ inline int ffd_tab_words(int D) { return D >= 32 ? D / 32 : 1; }

int64_t ffd_small_table_floats(const sk_sketch *s, int layer) {
  const int64_t D = s->D, nl = ffd_live_blocks(s, layer);
  return ((nl * D + nl * D / 2 + nl * ffd_tab_words((int)D)) + 63) & ~63ll;
}

struct FfdTab {
  const float *g;
  const uint16_t *perm;
  const uint32_t *sgn;
};

__host__ __device__ inline FfdTab ffd_tab(const float *tab, int64_t nlive, int D) {
  FfdTab t;
  t.g = tab;
  t.perm = reinterpret_cast<const uint16_t *>(tab + nlive * D);
  t.sgn = reinterpret_cast<const uint32_t *>(tab + nlive * D + nlive * D / 2);
  return t;
}

// One thread per 4 consecutive coordinates i4 .. i4 + 3 of block b = blockIdx.y
// (one Philox block of Gaussians, four permutation entries; the first thread
// of a 32-coordinate run also its sign word); the block's permutation key is
// made once per workgroup.
__global__ __launch_bounds__(256) void k_ffd_tables(const LayerDesc *__restrict__ layers, int layer, int lgD,
                                                    int64_t nlive, float *__restrict__ tab, Key key) {
  __shared__ PermKey s_pk;
  const LayerDesc &ld = layers[layer];
  const int D = 1 << lgD;
  const int64_t b = blockIdx.y;
  if (threadIdx.x == 0) s_pk = perm_key((uint32_t)ld.layer_id, ST_FFDPERM, (uint32_t)b, (uint32_t)lgD, key);
  __syncthreads();
  const int i4 = (blockIdx.x * 256 + threadIdx.x) * 4;
  if (i4 >= D) return;
  float *g = tab + b * D;
  uint16_t *perm = reinterpret_cast<uint16_t *>(tab + nlive * D) + b * D;
  uint32_t *sgn = reinterpret_cast<uint32_t *>(tab + nlive * D + nlive * D / 2) + b * ffd_tab_words(D);
  const int64_t base = b * D;
  float gv[4];
  gauss4((uint64_t)(base + i4) >> 2, (uint32_t)ld.layer_id, ST_GAUSS, key, gv);
  *reinterpret_cast<float4 *>(g + i4) = make_float4(gv[0], gv[1], gv[2], gv[3]);
  const PermKey pk = s_pk;
  uint32_t pp[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) pp[q] = perm_fwd(pk, (uint32_t)(i4 + q));
  *reinterpret_cast<uint2 *>(perm + i4) = make_uint2(pp[0] | (pp[1] << 16), pp[2] | (pp[3] << 16));
  if ((i4 & 31) == 0) {
    // bits of coordinates base + i4 .. + 31 (or the D = 16 coordinates of a block that
    // starts half-way through a global 32-coordinate word)
    const int64_t j = base + i4;
    const int sh = (int)(j & 31);
    uint32_t w = sign_word((uint64_t)j, (uint32_t)ld.layer_id, key) >> sh;
    if (sh) w |= sign_word((uint64_t)(j + 32), (uint32_t)ld.layer_id, key) << (32 - sh);
    sgn[i4 >> 5] = w;
  }
}

void launch_ffd_tables(const sk_sketch *s, int layer, float *tab, hipStream_t st) {
  const int lgD = log2_exact(s->D);
  const int64_t nlive = ffd_live_blocks(s, layer);
  const dim3 grid((unsigned)((s->D / 4 + 255) / 256), (unsigned)nlive);
  hipLaunchKernelGGL(k_ffd_tables, grid, dim3(256), 0, st, s->d_layers, layer, lgD, nlive, tab, s->key);
  SK_CHECK_LAUNCH();
}

// Thread t's share of block b's tables: coordinates i = t + 256 k (k < PER;
// with PER = 1 only t < D).  pv[k] = p16(Pi_b(i)), the LDS place of the
// permuted coordinate.
template <int PER>
__device__ __forceinline__ void ffd_load_tab(const FfdTab &tb, int64_t b, int D, float (&gv)[PER], int (&pv)[PER],
                                             uint32_t &sb) {
  // row bases are uniform; per-thread offsets are 32-bit
  const float *g = tb.g + b * D;
  const uint16_t *pm = tb.perm + b * D;
  const uint32_t *sw = tb.sgn + b * ffd_tab_words(D);
  sb = 0;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const uint32_t i = threadIdx.x + k * 256;
    gv[k] = 0.0f;
    pv[k] = 0;
    if (PER > 1 || i < (uint32_t)D) {
      gv[k] = g[i];
      pv[k] = p16(pm[i]);
      sb |= ((sw[i >> 5] >> (i & 31)) & 1u) << k;
    }
  }
}

// LDS place of coordinate t + 256 k in the p16 layout: p16(t) + 272 k.
__device__ __forceinline__ int ffd_p16_base() {
  const int t = threadIdx.x;
  return p16(t);
}

// Forward, D <= 2^13: a workgroup takes one block and VT vectors; per vector:
// load, H_D, scatter through Pi_b with g, H_D, signs, kept in registers
// (PER = D / 256 values per thread and vector) and written as the block's
// partial sum.  One LDS tile (the scatter goes through registers), so that
// several workgroups share a compute unit.
template <bool BF16, int VT, int PER>
__global__ __launch_bounds__(256) void k_ffd_small_fwd(const LayerDesc *__restrict__ layers, int layer,
                                                       const void *__restrict__ x, int lgD, int64_t b_begin,
                                                       int64_t bc, float *__restrict__ part, int64_t slot0,
                                                       int64_t nlive, const float *__restrict__ tab) {
  extern __shared__ float sm[];
  const int D = 1 << lgD;
  float *s = sm;  // p16 layout
  const LayerDesc &ld = layers[layer];
  const int64_t v0 = (int64_t)blockIdx.y * VT;
  const int64_t b = blockIdx.x;
  const int64_t base = b * D;
  const bool act = PER > 1 || (int)threadIdx.x < D;  // PER = 1: threads past D hold nothing
  float gv[PER];
  int pv[PER];
  uint32_t sb;
  ffd_load_tab<PER>(ffd_tab(tab, nlive, D), b, D, gv, pv, sb);
  // coordinates of this block present in the vector (only the last block may be cut)
  const int lim = ld.n - base < D ? (int)(ld.n - base) : D;
  float xr[PER];
  auto load_x = [&](int64_t vv) {
    const int64_t row = (b_begin + vv) * ld.n + base;
    const uint16_t *xh = (const uint16_t *)x + row;
    const float *xf = (const float *)x + row;
    const bool full = lim == D && vv < bc;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const uint32_t i = threadIdx.x + k * 256;
      float val = 0.0f;
      if (full ? act : ((int)i < lim && vv < bc)) val = BF16 ? bf16_to_f32(xh[i]) : xf[i];
      xr[k] = val;
    }
  };
  load_x(v0);
  const float inv = 1.0f / (float)D;
  float acc[VT][PER];
#pragma unroll
  for (int v = 0; v < VT; ++v) {
#pragma unroll
    for (int k = 0; k < PER; ++k) acc[v][k] = 0.0f;
    if (v0 + v >= bc) break;
    if (v > 0) __syncthreads();  // the previous vector's last reads of s are done
    float *sp = s + ffd_p16_base();
    if (act) {
#pragma unroll
      for (int k = 0; k < PER; ++k) sp[272 * k] = xr[k];
    }
    if (v + 1 < VT) load_x(v0 + v + 1);
    lds_fwht_regs(s, lgD, 0);
    float t[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) t[k] = act ? sp[272 * k] : 0.0f;
    __syncthreads();
    if (act) {
#pragma unroll
      for (int k = 0; k < PER; ++k) s[pv[k]] = gv[k] * t[k];
    }
    lds_fwht_regs(s, lgD, 0);
    if (act) {
#pragma unroll
      for (int k = 0; k < PER; ++k) acc[v][k] = flip(sp[272 * k] * inv, (sb >> k) & 1u);
    }
  }
  if (!act) return;
#pragma unroll
  for (int v = 0; v < VT; ++v) {
    if (v0 + v >= bc) break;
    float *dst = part + ((slot0 + b) * bc + v0 + v) * D;
#pragma unroll
    for (int k = 0; k < PER; ++k) dst[threadIdx.x + k * 256] = acc[v][k];
  }
}

// LDS of the small-D FFD kernels: one p16 tile of D floats (36 KB at D = 2^13).
static size_t ffd_small_shm(int64_t D) { return (size_t)p16_floats((int)D) * 4; }

template <int VT>
static void ffd_small_fwd_go(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc,
                             float *part, int64_t slot0, int64_t groups, int lgD, const float *tab, hipStream_t st) {
  const dim3 grid((unsigned)groups, (unsigned)((bc + VT - 1) / VT));
  const size_t shm = ffd_small_shm(s->D);
  const int64_t nlive = ffd_live_blocks(s, layer);
#define SK_FFDS(PER)                                                                                             \
  do {                                                                                                           \
    if (dtype == SK_BF16)                                                                                        \
      hipLaunchKernelGGL((k_ffd_small_fwd<true, VT, PER>), grid, dim3(256), shm, st, s->d_layers, layer, x, lgD, \
                         b_begin, bc, part, slot0, nlive, tab);                                                   \
    else                                                                                                         \
      hipLaunchKernelGGL((k_ffd_small_fwd<false, VT, PER>), grid, dim3(256), shm, st, s->d_layers, layer, x,     \
                         lgD, b_begin, bc, part, slot0, nlive, tab);                                              \
  } while (0)
  switch (lgD <= 8 ? 1 : 1 << (lgD - 8)) {
    case 1: SK_FFDS(1); break;
    case 2: SK_FFDS(2); break;
    case 4: SK_FFDS(4); break;
    case 8: SK_FFDS(8); break;
    case 16: SK_FFDS(16); break;
    default: SK_FFDS(32); break;
  }
#undef SK_FFDS
}

// Vectors per workgroup of the small-D kernels (2^20-entry vectors, batch 8,
// D = 4096, per call, forward / transpose: 1 vector 29 / 30 us, 2 31 / 35,
// 4 36 / 35; the kernels that made their tables in LDS per workgroup took
// 56 / 56 at their best, 4 vectors)
constexpr int kFfdVtFwd = 1;
constexpr int kFfdVtT = 1;

void launch_ffd_small_fwd(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc,
                          float *part, int64_t slot0, int64_t groups, const float *tab, hipStream_t st) {
  const int lgD = log2_exact(s->D);
  if (lgD < 4 || lgD > kFfdSmallMax) return;  // the small-D path: 2^4 <= D <= 2^13
  ffd_small_fwd_go<kFfdVtFwd>(s, layer, x, dtype, b_begin, bc, part, slot0, groups, lgD, tab, st);
  SK_CHECK_LAUNCH();
}

__global__ void k_reduce_partials(const float *__restrict__ part, int64_t nslots, int64_t bc, int64_t D,
                                  int64_t b_begin, float *__restrict__ out, int accumulate) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i >= bc * D) return;
  const int64_t v = i / D, c = i - v * D;
  float acc = 0.0f;
  for (int64_t k = 0; k < nslots; ++k) acc += part[(k * bc + v) * D + c];
  float *o = out + (b_begin + v) * D + c;
  *o = accumulate ? *o + acc : acc;
}

// The same sum for D % 4 == 0 and 16-byte aligned buffers, in 16-byte pieces: a
// 1024-thread workgroup owns 32 pieces (128 consecutive outputs); lane l of wave
// q takes piece l % 32 and sums slots k = r, r + 32, r + 64, ... with
// r = 2 q + l / 32; the 32 residue sums are then added in the order r = 0 .. 31.
// The order depends on nslots only (not on the batch), and nothing is atomic.
__global__ __launch_bounds__(1024) void k_reduce_partials4(const float *__restrict__ part, int64_t nslots,
                                                           int64_t n4, int64_t D, int64_t b_begin,
                                                           float *__restrict__ out, int accumulate) {
  __shared__ float4 red[32][33];
  const int lane = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int c = lane & 31, r = 2 * q + (lane >> 5);
  const int64_t p = (int64_t)blockIdx.x * 32 + c;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  if (p < n4) {
    const float4 *src = reinterpret_cast<const float4 *>(part) + p;
    for (int64_t k = r; k < nslots; k += 32) {
      const float4 a = src[k * n4];
      acc.x += a.x;
      acc.y += a.y;
      acc.z += a.z;
      acc.w += a.w;
    }
  }
  red[r][c] = acc;
  __syncthreads();
  if (threadIdx.x < 32 && p < n4) {
    float4 t = red[0][c];
    for (int k = 1; k < 32; ++k) {
      const float4 a = red[k][c];
      t.x += a.x;
      t.y += a.y;
      t.z += a.z;
      t.w += a.w;
    }
    const int64_t i = p * 4, v = i / D;
    float4 *o = reinterpret_cast<float4 *>(out + (b_begin + v) * D + (i - v * D));
    if (accumulate) {
      const float4 a = *o;
      t.x += a.x;
      t.y += a.y;
      t.z += a.z;
      t.w += a.w;
    }
    *o = t;
  }
}

// The same sum for at most 16 slots: one 16-byte piece per thread with every
// slot's load in flight together, added from zero in slot order (the order
// k_reduce_partials4 takes for these counts, so the results are identical).
__global__ __launch_bounds__(256) void k_reduce_partials4_few(const float *__restrict__ part, int nslots, int64_t n4,
                                                              int64_t D, int64_t b_begin, float *__restrict__ out,
                                                              int accumulate) {
  const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (p >= n4) return;
  const float4 *src = reinterpret_cast<const float4 *>(part) + p;
  float4 t[16];
#pragma unroll
  for (int k = 0; k < 16; ++k)
    if (k < nslots) t[k] = src[k * n4];
  float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int k = 0; k < 16; ++k)
    if (k < nslots) {
      a.x += t[k].x;
      a.y += t[k].y;
      a.z += t[k].z;
      a.w += t[k].w;
    }
  const int64_t i = p * 4, v = i / D;
  float4 *o = reinterpret_cast<float4 *>(out + (b_begin + v) * D + (i - v * D));
  if (accumulate) {
    const float4 q = *o;
    a.x += q.x;
    a.y += q.y;
    a.z += q.z;
    a.w += q.w;
  }
  *o = a;
}

void launch_reduce_partials(const float *part, int64_t nslots, int64_t bc, int64_t D, int64_t b_begin, float *out,
                            bool accumulate, hipStream_t st) {
  if (nslots <= 16 && D % 4 == 0 && ((uintptr_t)part & 15) == 0 && ((uintptr_t)out & 15) == 0) {
    const int64_t n4 = bc * D / 4;
    hipLaunchKernelGGL(k_reduce_partials4_few, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, st, part,
                       (int)nslots, n4, D, b_begin, out, (int)accumulate);
    SK_CHECK_LAUNCH();
    return;
  }
  if (D % 4 == 0 && ((uintptr_t)part & 15) == 0 && ((uintptr_t)out & 15) == 0) {
    const int64_t n4 = bc * D / 4;
    hipLaunchKernelGGL(k_reduce_partials4, dim3((unsigned)((n4 + 31) / 32)), dim3(1024), 0, st, part, nslots, n4, D,
                       b_begin, out, (int)accumulate);
    SK_CHECK_LAUNCH();
    return;
  }
  hipLaunchKernelGGL(k_reduce_partials, dim3((unsigned)((bc * D + 255) / 256)), dim3(256), 0, st, part, nslots, bc, D,
                     b_begin, out, (int)accumulate);
  SK_CHECK_LAUNCH();
}

// Transpose, D <= 2^13: a workgroup takes one block and VT vectors; per
// vector: signs, H_D, gather through Pi_b with g, H_D, theta0, store.  One
// LDS tile, as in the forward.
template <int VT, int PER>
__global__ __launch_bounds__(256) void k_ffd_small_T(const LayerDesc *__restrict__ layers, int layer,
                                                     const float *__restrict__ z, int lgD, int64_t b_begin,
                                                     int64_t bc, void *__restrict__ out, int out_dtype,
                                                     const float *__restrict__ theta0, int64_t nlive,
                                                     const float *__restrict__ tab) {
  extern __shared__ float sm[];
  const int D = 1 << lgD;
  float *s = sm;  // p16 layout
  const LayerDesc &ld = layers[layer];
  const int64_t b = blockIdx.x;
  const int64_t v0 = (int64_t)blockIdx.y * VT;
  const int64_t base = b * D;
  const bool act = PER > 1 || (int)threadIdx.x < D;
  float gv[PER];
  int pv[PER];
  uint32_t sb;
  ffd_load_tab<PER>(ffd_tab(tab, nlive, D), b, D, gv, pv, sb);
  const int lim = ld.n - base < D ? (int)(ld.n - base) : D;
  const float inv = 1.0f / (float)D;
  float zr[PER];
  auto load_z = [&](int64_t vv) {
    const float *zv = z + (b_begin + vv) * D;
    const bool ok = act && vv < bc;
#pragma unroll
    for (int k = 0; k < PER; ++k) zr[k] = ok ? zv[threadIdx.x + k * 256] : 0.0f;
  };
  load_z(v0);
#pragma unroll 1
  for (int v = 0; v < VT; ++v) {
    if (v0 + v >= bc) break;
    if (v > 0) __syncthreads();  // the previous vector's last reads of s are done
    float *sp = s + ffd_p16_base();
    if (act) {
#pragma unroll
      for (int k = 0; k < PER; ++k) sp[272 * k] = flip(zr[k], (sb >> k) & 1u);
    }
    if (v + 1 < VT) load_z(v0 + v + 1);
    lds_fwht_regs(s, lgD, 0);
    float t[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) t[k] = act ? s[pv[k]] : 0.0f;
    __syncthreads();
    if (act) {
#pragma unroll
      for (int k = 0; k < PER; ++k) sp[272 * k] = gv[k] * t[k];
    }
    lds_fwht_regs(s, lgD, 0);
    if (!act) continue;
    const int64_t row = (b_begin + v0 + v) * ld.n + base;
    uint16_t *oh = (uint16_t *)out + row;
    float *of = (float *)out + row;
    const float *th = theta0 ? theta0 + base : nullptr;
    const bool full = lim == D;
    float r[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) r[k] = sp[272 * k] * inv;
    if (th) {
#pragma unroll
      for (int k = 0; k < PER; ++k) {
        const uint32_t i = threadIdx.x + k * 256;
        if (full || (int)i < lim) r[k] += th[i];
      }
    }
    if (out_dtype == SK_BF16) {
#pragma unroll
      for (int k = 0; k < PER; ++k) {
        const uint32_t i = threadIdx.x + k * 256;
        if (full || (int)i < lim) oh[i] = f32_to_bf16(r[k]);
      }
    } else {
#pragma unroll
      for (int k = 0; k < PER; ++k) {
        const uint32_t i = threadIdx.x + k * 256;
        if (full || (int)i < lim) of[i] = r[k];
      }
    }
  }
}

void launch_ffd_small_T(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, void *out,
                        int out_dtype, const float *theta0, const float *tab, hipStream_t st) {
  const int lgD = log2_exact(s->D);
  if (lgD < 4 || lgD > kFfdSmallMax) return;  // the small-D path: 2^4 <= D <= 2^13
  constexpr int VT = kFfdVtT;
  const int64_t nlive = ffd_live_blocks(s, layer);
  const dim3 grid((unsigned)nlive, (unsigned)((bc + VT - 1) / VT));
  const size_t shm = ffd_small_shm(s->D);
#define SK_FFDT(PER)                                                                                              \
  hipLaunchKernelGGL((k_ffd_small_T<VT, PER>), grid, dim3(256), shm, st, s->d_layers, layer, z, lgD, b_begin, bc, \
                     out, out_dtype, theta0, nlive, tab)
  switch (lgD <= 8 ? 1 : 1 << (lgD - 8)) {
    case 1: SK_FFDT(1); break;
    case 2: SK_FFDT(2); break;
    case 4: SK_FFDT(4); break;
    case 8: SK_FFDT(8); break;
    case 16: SK_FFDT(16); break;
    default: SK_FFDT(32); break;
  }
#undef SK_FFDT
  SK_CHECK_LAUNCH();
}

// --- large D: workspace w[v][bb][i], bb < nlive ---
template <bool BF16>
__global__ void k_ffd_copy_blocks(const LayerDesc *__restrict__ layers, int layer, const void *__restrict__ x,
                                  int64_t span, int64_t b_begin, float *__restrict__ w) {
  const LayerDesc &ld = layers[layer];
  const int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;  // within the live span
  if (j >= span) return;
  const int64_t v = blockIdx.y;
  float val = 0.0f;
  if (j < ld.n) {
    const int64_t e = (b_begin + v) * ld.n + j;
    val = BF16 ? bf16_to_f32(((const uint16_t *)x)[e]) : ((const float *)x)[e];
  }
  w[v * span + j] = val;
}

void launch_ffd_copy_blocks(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc,
                            float *w, hipStream_t st) {
  const int64_t span = ffd_live_blocks(s, layer) * s->D;
  dim3 grid((unsigned)((span + 255) / 256), (unsigned)bc);
  if (dtype == SK_BF16)
    hipLaunchKernelGGL(k_ffd_copy_blocks<true>, grid, dim3(256), 0, st, s->d_layers, layer, x, span, b_begin, w);
  else
    hipLaunchKernelGGL(k_ffd_copy_blocks<false>, grid, dim3(256), 0, st, s->d_layers, layer, x, span, b_begin, w);
  SK_CHECK_LAUNCH();
}

// w2[v][bb][pi_b(k)] = g_{b,k} w[v][bb][k]; one thread per 4 consecutive k, all vectors.
__global__ void k_ffd_gperm_fwd(const LayerDesc *__restrict__ layers, int layer, const float *__restrict__ w,
                                int lgD, int64_t nlive, int64_t bc, float *__restrict__ w2, Key key) {
  const LayerDesc &ld = layers[layer];
  const int64_t D = 1ll << lgD;
  const int64_t t = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) * 4;
  const int64_t bb = t >> lgD;
  if (bb >= nlive) return;
  const int64_t k0 = t & (D - 1);
  const PermKey pk = perm_key((uint32_t)ld.layer_id, ST_FFDPERM, (uint32_t)bb, (uint32_t)lgD, key);
  float g[4];
  gauss4((uint64_t)(bb * D + k0) >> 2, (uint32_t)ld.layer_id, ST_GAUSS, key, g);
  uint32_t p[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) p[q] = perm_fwd(pk, (uint32_t)(k0 + q));
  const int64_t span = nlive * D;
  for (int64_t v = 0; v < bc; ++v) {
    const float4 x = *(const float4 *)(w + v * span + t);
    float *dst = w2 + v * span + bb * D;
    dst[p[0]] = g[0] * x.x;
    dst[p[1]] = g[1] * x.y;
    dst[p[2]] = g[2] * x.z;
    dst[p[3]] = g[3] * x.w;
  }
}

void launch_ffd_gperm_fwd(const sk_sketch *s, int layer, const float *w, int64_t bc, float *w2, hipStream_t st) {
  const int lgD = log2_exact(s->D);
  if (lgD < 4 || lgD > 20) return;  // create() admits 2^4 <= D <= 2^20 only
  const int64_t nlive = ffd_live_blocks(s, layer);
  const int64_t th = nlive * s->D / 4;
  hipLaunchKernelGGL(k_ffd_gperm_fwd, dim3((unsigned)((th + 255) / 256)), dim3(256), 0, st, s->d_layers, layer, w,
                     lgD, nlive, bc, w2, s->key);
  SK_CHECK_LAUNCH();
}

__global__ void k_ffd_sum_signed(const LayerDesc *__restrict__ layers, int layer, const float *__restrict__ w2,
                                 int64_t D, int64_t nlive, int64_t b_begin, int64_t bc, float *__restrict__ out,
                                 int accumulate, Key key) {
  const LayerDesc &ld = layers[layer];
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i >= D) return;
  const int64_t v = blockIdx.y;
  float acc = 0.0f;
  for (int64_t bb = 0; bb < nlive; ++bb) {
    const int64_t j = bb * D + i;
    const uint32_t bit = (sign_word((uint64_t)j, (uint32_t)ld.layer_id, key) >> (j & 31)) & 1u;
    acc += flip(w2[v * nlive * D + j], bit);
  }
  float *o = out + (b_begin + v) * D + i;
  *o = accumulate ? *o + acc : acc;
}

void launch_ffd_sum_signed(const sk_sketch *s, int layer, const float *w2, int64_t b_begin, int64_t bc, float *out,
                           bool accumulate, hipStream_t st) {
  dim3 grid((unsigned)((s->D + 255) / 256), (unsigned)bc);
  hipLaunchKernelGGL(k_ffd_sum_signed, grid, dim3(256), 0, st, s->d_layers, layer, w2, s->D,
                     ffd_live_blocks(s, layer), b_begin, bc, out, (int)accumulate, s->key);
  SK_CHECK_LAUNCH();
}

__global__ void k_ffd_expand_z(const LayerDesc *__restrict__ layers, int layer, const float *__restrict__ z,
                               int lgD, int64_t nlive, int64_t b_begin, float *__restrict__ w, Key key) {
  const LayerDesc &ld = layers[layer];
  const int64_t D = 1ll << lgD;
  const int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (j >= nlive * D) return;
  const int64_t v = blockIdx.y;
  const uint32_t bit = (sign_word((uint64_t)j, (uint32_t)ld.layer_id, key) >> (j & 31)) & 1u;
  w[v * nlive * D + j] = flip(z[(b_begin + v) * D + (j & (D - 1))], bit);
}

void launch_ffd_expand_z(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, float *w,
                         hipStream_t st) {
  const int lgD = log2_exact(s->D);
  if (lgD < 4 || lgD > 20) return;  // create() admits 2^4 <= D <= 2^20 only
  const int64_t nlive = ffd_live_blocks(s, layer);
  dim3 grid((unsigned)((nlive * s->D + 255) / 256), (unsigned)bc);
  hipLaunchKernelGGL(k_ffd_expand_z, grid, dim3(256), 0, st, s->d_layers, layer, z, lgD, nlive, b_begin, w, s->key);
  SK_CHECK_LAUNCH();
}

// w2[v][bb][i] = g_{b,i} w[v][bb][pi_b(i)]
__global__ void k_ffd_permg_T(const LayerDesc *__restrict__ layers, int layer, const float *__restrict__ w, int lgD,
                              int64_t nlive, int64_t bc, float *__restrict__ w2, Key key) {
  const LayerDesc &ld = layers[layer];
  const int64_t D = 1ll << lgD;
  const int64_t t = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) * 4;
  const int64_t bb = t >> lgD;
  if (bb >= nlive) return;
  const int64_t i0 = t & (D - 1);
  const PermKey pk = perm_key((uint32_t)ld.layer_id, ST_FFDPERM, (uint32_t)bb, (uint32_t)lgD, key);
  float g[4];
  gauss4((uint64_t)(bb * D + i0) >> 2, (uint32_t)ld.layer_id, ST_GAUSS, key, g);
  uint32_t p[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) p[q] = perm_fwd(pk, (uint32_t)(i0 + q));
  const int64_t span = nlive * D;
  for (int64_t v = 0; v < bc; ++v) {
    const float *src = w + v * span + bb * D;
    float4 o = make_float4(g[0] * src[p[0]], g[1] * src[p[1]], g[2] * src[p[2]], g[3] * src[p[3]]);
    *(float4 *)(w2 + v * span + t) = o;
  }
}

void launch_ffd_permg_T(const sk_sketch *s, int layer, const float *w, int64_t bc, float *w2, hipStream_t st) {
  const int lgD = log2_exact(s->D);
  if (lgD < 4 || lgD > 20) return;  // create() admits 2^4 <= D <= 2^20 only
  const int64_t nlive = ffd_live_blocks(s, layer);
  const int64_t th = nlive * s->D / 4;
  hipLaunchKernelGGL(k_ffd_permg_T, dim3((unsigned)((th + 255) / 256)), dim3(256), 0, st, s->d_layers, layer, w, lgD,
                     nlive, bc, w2, s->key);
  SK_CHECK_LAUNCH();
}

__global__ void k_ffd_T_out(const LayerDesc *__restrict__ layers, int layer, const float *__restrict__ w2,
                            int64_t span, int64_t b_begin, void *__restrict__ out, int out_dtype,
                            const float *__restrict__ theta0) {
  const LayerDesc &ld = layers[layer];
  const int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (j >= ld.n) return;
  const int64_t v = blockIdx.y;
  store_out(out, out_dtype, (b_begin + v) * ld.n + j, w2[v * span + j] + (theta0 ? theta0[j] : 0.0f));
}

void launch_ffd_T_out(const sk_sketch *s, int layer, const float *w2, int64_t b_begin, int64_t bc, void *out,
                      int out_dtype, const float *theta0, hipStream_t st) {
  const LayerDesc &ld = s->layers[layer];
  const int64_t span = ffd_live_blocks(s, layer) * s->D;
  dim3 grid((unsigned)((ld.n + 255) / 256), (unsigned)bc);
  hipLaunchKernelGGL(k_ffd_T_out, grid, dim3(256), 0, st, s->d_layers, layer, w2, span, b_begin, out, out_dtype,
                     theta0);
  SK_CHECK_LAUNCH();
}

// ===========================================================================
// Tables and stream export.
// ===========================================================================
__global__ void k_gauss_table(const LayerDesc *__restrict__ layers, int nl, int64_t D, float *__restrict__ gtab,
                              Key key) {
  const int64_t t = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) * 4;
  const int l = blockIdx.y;
  if (t >= D || l >= nl) return;
  float g[4];
  gauss4((uint64_t)t >> 2, (uint32_t)layers[l].layer_id, ST_GAUSS, key, g);
#pragma unroll
  for (int q = 0; q < 4; ++q)
    if (t + q < D) gtab[(int64_t)l * D + t + q] = g[q];
}

void launch_gauss_table(const sk_sketch *s, float *gtab, hipStream_t st) {
  dim3 grid((unsigned)((s->D / 4 + 255) / 256 + 1), (unsigned)s->layers.size());
  hipLaunchKernelGGL(k_gauss_table, grid, dim3(256), 0, st, s->d_layers, (int)s->layers.size(), s->D, gtab, s->key);
  SK_CHECK_LAUNCH();
}

__global__ void k_debug_stream(const LayerDesc *__restrict__ layers, const uint16_t *__restrict__ ptab, int layer,
                               int stream_id, uint64_t start, uint64_t count, uint64_t aux, int lgD, void *dout,
                               Key key) {
  const uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x;
  if (i >= count) return;
  const LayerDesc &ld = layers[layer];
  const uint64_t j = start + i;
  const uint32_t lid = (uint32_t)ld.layer_id;
  switch (stream_id) {
    case ST_SIGN:
      ((int8_t *)dout)[i] = ((sign_word(j, lid, key) >> (j & 31)) & 1u) ? -1 : 1;
      break;
    case ST_GAUSS:
    case ST_QKA:
    case ST_QKB:
      ((float *)dout)[i] = gauss(j, lid, (uint32_t)stream_id, key);
      break;
    case ST_INDEX:
      ((uint32_t *)dout)[i] = sample_index(j, lid, key, (uint64_t)ld.np);
      break;
    case ST_PI1:
    case ST_PI2: {
      const int sidx = stream_id == ST_PI1 ? 0 : 1;
      uint64_t r = 0, stride = 1;
      for (int k = ld.K - 1; k >= 0; --k) {
        const uint64_t dig = (j / stride) & ((1ull << ld.lg[k]) - 1);
        r += (uint64_t)ptab[ld.poff[sidx][0][k] + dig] * stride;
        stride <<= ld.lg[k];
      }
      ((uint32_t *)dout)[i] = (uint32_t)r;
      break;
    }
    case ST_FFDPERM: {
      const PermKey pk = perm_key(lid, ST_FFDPERM, (uint32_t)aux, (uint32_t)lgD, key);
      ((uint32_t *)dout)[i] = perm_fwd(pk, (uint32_t)j);
      break;
    }
    default:
      break;
  }
}

void launch_debug_stream(const sk_sketch *s, int layer, int stream_id, uint64_t start, uint64_t count, uint64_t aux,
                         void *dout, hipStream_t st) {
  const int lgD = log2_exact(s->D);
  if (lgD < 4 || lgD > 20) return;  // create() admits 2^4 <= D <= 2^20 only
  hipLaunchKernelGGL(k_debug_stream, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, st, s->d_layers, s->d_ptab,
                     layer, stream_id, start, count, aux, lgD, dout, s->key);
  SK_CHECK_LAUNCH();
}

}  // namespace sk
