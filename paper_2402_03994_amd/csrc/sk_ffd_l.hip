// sk_ffd_l.hip -- FFD (eq. fastfood) blocks of D = 2^20.
//
// A block index i splits into (r, c) = (i >> 10, i & 1023) and
// H_D = H_1024(r) (x) H_1024(c).  Intermediates are kept transposed: position
// pos(i) = c 1024 + r holds element i, so that both 1024-point transforms read
// and write whole rows:
//   rows kernel  32 rows r of a block: gather / load, H over c, write pos()
//   cols kernel  32 columns c (contiguous in pos order): H over r, epilogue
// Forward y = sum_b B_b H Pi_b^T G_b H x_b:
//   rows(x) -> cols(. g, pos order) -> rows(gather k = pi^{-1}(d)) -> sum over
//   blocks of B_b . cols(.) in registers -> y.
// Transpose block b = H G_b Pi_b H B_b z:
//   rows(B_b z) -> cols -> rows(g_i . gather k = pi(i)) -> cols -> theta.
// Batches that are a multiple of four run the middle passes on groups of four
// vectors with interleaved intermediates, and move the data through Pi_b by
// buckets (a counting sort in LDS by destination chunk) instead of a gather.
// Each kernel applies 1/32 (a normalised H_1024).
#include "sk_kcommon.h"
#include "sk_launch.h"

namespace sk {

namespace {

constexpr int kLgD = 20;
constexpr int64_t kD = 1ll << kLgD;

__device__ __forceinline__ uint32_t tpos(uint32_t i) { return ((i & 1023u) << 10) | (i >> 10); }

enum RowsMode { kRowsX = 0, kRowsZ = 1, kRowsPermFwd = 2, kRowsPermT = 3 };

// Rows kernel: 1024 threads per (32 rows r0.., block b, vector v).  After the
// transform thread (ri = tid % 32, rc = tid / 32) holds columns c = 32 rc + m
// of row r0 + ri, so for each m the 32 lanes of a column write 32 consecutive
// positions pos = c 1024 + r0 .. r0 + 31: one 128-byte line.
template <int MODE, bool BF16>
__global__ __launch_bounds__(1024) void k_ffdL_rows(const LayerDesc *__restrict__ layers, int layer,
                                                    const void *__restrict__ src, int64_t b_begin, int64_t nlive,
                                                    float *__restrict__ dst, Key key) {
  using L = Lds1024R32;
  __shared__ __align__(16) float s[L::kFloats];
  __shared__ __align__(16) uint32_t sg[32 * 32];
  const LayerDesc &ld = layers[layer];
  int r0 = blockIdx.x * 32;
  int64_t b = blockIdx.y, v = blockIdx.z;
  if ((MODE == kRowsPermFwd || MODE == kRowsPermT) && (nlive * gridDim.z) % 8 == 0) {
    // workgroup id g runs on XCD g mod 8: XCD x takes (vector, block) pairs
    // x, x + 8, ... one at a time, so its random reads stay in its own L2
    const int64_t g = blockIdx.x + 32 * (blockIdx.y + nlive * blockIdx.z);
    const int64_t k = g >> 3;
    const int64_t pair = 8 * (k >> 5) + (g & 7);
    r0 = (int)(k & 31) * 32;
    v = pair / nlive;
    b = pair - v * nlive;
  }
  const int64_t blk = (v * nlive + b) * kD;  // this block in the workspace
  if (MODE == kRowsZ) {
    // B_b signs of the 32 rows: 8 Philox blocks of 128 per row, shared in LDS
    if (threadIdx.x < 256) {
      const int i = threadIdx.x >> 3;
      const W4 q = philox((uint64_t)((b * kD + (int64_t)(r0 + i) * 1024) >> 7) + (threadIdx.x & 7),
                          (uint32_t)ld.layer_id, ST_SIGN, key);
      *(uint4 *)(sg + 4 * threadIdx.x) = make_uint4(q.w[0], q.w[1], q.w[2], q.w[3]);
    }
    __syncthreads();
  }
  PermKey pk;
  if (MODE == kRowsPermFwd || MODE == kRowsPermT)
    pk = perm_key((uint32_t)ld.layer_id, ST_FFDPERM, (uint32_t)b, (uint32_t)kLgD, key);
  // thread: rows 4 k + quarter (k < 8); all its loads are issued before any LDS write
  const int quarter = threadIdx.x >> 8, t = threadIdx.x & 255;
  float val[8][4];
  if (MODE == kRowsPermT) {
    // u_i = g_i w[pi(i)]: four consecutive columns per thread share one Philox block
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const uint32_t e0 = (uint32_t)(r0 + 4 * k + quarter) * 1024u + 4u * t;
#pragma unroll
      for (int q = 0; q < 4; ++q) val[k][q] = ((const float *)src)[blk + tpos(perm_fwd(pk, e0 + q))];
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int i = 4 * k + quarter;
      const uint32_t e0 = (uint32_t)(r0 + i) * 1024u + 4u * t;
      float g[4];
      gauss4((uint64_t)(b * kD + e0) >> 2, (uint32_t)ld.layer_id, ST_GAUSS, key, g);
#pragma unroll
      for (int q = 0; q < 4; ++q) s[L::idx(i, 4 * t + q)] = g[q] * val[k][q];
    }
  } else {
    // thread: columns c = t + 256 q (q < 4), consecutive over the lanes
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int i = 4 * k + quarter;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c = t + 256 * q;
        const uint32_t e = (uint32_t)(r0 + i) * 1024u + (uint32_t)c;
        if (MODE == kRowsX) {
          // past the layer the index is clamped and the value selected, so no load waits behind a branch
          const int64_t j = b * kD + e;
          const int64_t x = (b_begin + v) * ld.n + (j < ld.n ? j : ld.n - 1);
          const float t = BF16 ? bf16_to_f32(((const uint16_t *)src)[x]) : ((const float *)src)[x];
          val[k][q] = j < ld.n ? t : 0.0f;
        } else if (MODE == kRowsZ) {
          const uint32_t bit = (sg[i * 32 + (c >> 5)] >> (c & 31)) & 1u;
          val[k][q] = flip(((const float *)src)[(b_begin + v) * kD + e], bit);
        } else {  // kRowsPermFwd: d = e, k = pi^{-1}(d)
          val[k][q] = ((const float *)src)[blk + tpos(perm_inv(pk, e))];
        }
      }
    }
#pragma unroll
    for (int k = 0; k < 8; ++k)
#pragma unroll
      for (int q = 0; q < 4; ++q) s[L::idx(4 * k + quarter, t + 256 * q)] = val[k][q];
  }
  __syncthreads();
  float e[32];
  fwht1024_rows32(s, e);
  const int ri = threadIdx.x & 31, rc = threadIdx.x >> 5;
  // column 32 rc + m, row r0 + ri: byte (32 rc + m) 4096 + 4 (r0 + ri) of the block
  const __amdgpu_buffer_rsrc_t ws = buf_rsrc(dst + blk + r0, (uint32_t)((kD - r0) * 4));
  const int soff = (32 * rc * 1024 + ri) * 4;
#pragma unroll
  for (int m = 0; m < 32; ++m)
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(e[m] * (1.0f / 32.0f)), ws, soff, m * 4096, 0);
}

enum ColsMode { kColsG = 0, kColsPlain = 1, kColsOutT = 2 };

// Cols kernel: 1024 threads per (32 columns c0.., block b, vector v); the 32
// columns are 32 contiguous rows (4 KB each) of the transposed block.  After
// the transform thread (ri, rc) holds r = 32 rc + m of column c0 + ri:
// kColsOutT writes the natural order from registers (32 lanes = 32
// consecutive columns of a row r); the other modes go back through LDS and
// write pos order with the lanes along r (and gauss4 per 4 columns for g).
template <int MODE>
__global__ __launch_bounds__(1024) void k_ffdL_cols(const LayerDesc *__restrict__ layers, int layer,
                                                    const float *__restrict__ src, int64_t b_begin, int64_t nlive,
                                                    float *__restrict__ dst, void *__restrict__ out, int out_dtype,
                                                    const float *__restrict__ theta0, Key key) {
  using L = Lds1024R32;
  __shared__ __align__(16) float s[L::kFloats];
  const LayerDesc &ld = layers[layer];
  int c0 = blockIdx.x * 32;
  int64_t b = blockIdx.y, v = blockIdx.z;
  if (MODE == kColsOutT && theta0) {
    // workgroup id g runs on XCD g mod 8; the vectors of one (column block,
    // block) follow each other on one XCD, so theta0 is read from HBM once
    const int64_t g = blockIdx.x + 32 * (blockIdx.y + nlive * blockIdx.z);
    const int64_t k = g >> 3, bc = gridDim.z;
    v = k % bc;
    const int64_t u = (k / bc) * 8 + (g & 7);
    c0 = (int)(u & 31) * 32;
    b = u >> 5;
  }
  const int64_t blk = (v * nlive + b) * kD;
  // kColsOutT: this thread's theta0 values (row 32 rc + m, column c0 + ri after the transform) are loaded
  // with the block, so the transform hides their latency; positions past n read the last one
  float th[32];
  if (MODE == kColsOutT && theta0) {
    const int ri0 = threadIdx.x & 31, rc0 = threadIdx.x >> 5;
    const float *tb = theta0 + b * kD + c0 + ri0;
    const int64_t lim = ld.n - 1 - (b * kD + c0 + ri0);  // last valid offset from tb
#pragma unroll
    for (int m = 0; m < 32; ++m) {
      const int64_t o = (int64_t)(32 * rc0 + m) * 1024;
      const float tv = tb[o < lim ? o : lim];
      th[m] = o <= lim ? tv : 0.0f;
    }
  }
  {
    // thread: rows 4 k + quarter, elements r = 4 t .. 4 t + 3 (16-byte loads)
    const int quarter = threadIdx.x >> 8, t = threadIdx.x & 255;
    float4 val[8];
#pragma unroll
    for (int k = 0; k < 8; ++k)
      val[k] = *(const float4 *)(src + blk + (int64_t)(c0 + 4 * k + quarter) * 1024 + 4 * t);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int i = 4 * k + quarter;
      s[L::idx(i, 4 * t)] = val[k].x;
      s[L::idx(i, 4 * t + 1)] = val[k].y;
      s[L::idx(i, 4 * t + 2)] = val[k].z;
      s[L::idx(i, 4 * t + 3)] = val[k].w;
    }
  }
  __syncthreads();
  float e[32];
  fwht1024_rows32(s, e);
  const int ri = threadIdx.x & 31, rc = threadIdx.x >> 5;
  if (MODE == kColsOutT) {
#pragma unroll
    for (int m = 0; m < 32; ++m) {
      const int r = 32 * rc + m;
      const int64_t jj = b * kD + (int64_t)r * 1024 + c0 + ri;
      if (jj < ld.n)
        store_out(out, out_dtype, (b_begin + v) * ld.n + jj, e[m] * (1.0f / 32.0f) + (theta0 ? th[m] : 0.0f));
    }
    return;
  }
  // back to the block (column c0 + ri at row ri, element r), then thread r
  // takes the 32 columns of its row
  __syncthreads();  // every thread's pass-2 reads are done
  float *bq = s + ri * L::kStride + 33 * rc;
#pragma unroll
  for (int m = 0; m < 32; ++m) bq[m] = e[m];
  __syncthreads();
  const int r = threadIdx.x;
#pragma unroll
  for (int a = 0; a < 8; ++a) {
    float g[4] = {1.0f, 1.0f, 1.0f, 1.0f};
    if (MODE == kColsG)
      gauss4((uint64_t)(b * kD + (int64_t)r * 1024 + c0 + 4 * a) >> 2, (uint32_t)ld.layer_id, ST_GAUSS, key, g);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int cc = 4 * a + q;
      dst[blk + (int64_t)(c0 + cc) * 1024 + r] = g[q] * (s[L::idx(cc, r)] * (1.0f / 32.0f));
    }
  }
}

// Forward epilogue: out[v][i] (+)= sum_b B_b(i) (H over r of block b)[i] for 8
// columns per workgroup; the next block's columns load during the current one.
// blockIdx.z picks a run of bseg consecutive blocks; with part set, run z
// writes its sum to part[(z bc + v) D + i] (summed afterwards in the order of
// z), else the one run covers every block and goes to out.
__global__ __launch_bounds__(256) void k_ffdL_sum(const LayerDesc *__restrict__ layers, int layer,
                                                  const float *__restrict__ src, int64_t b_begin, int64_t nlive,
                                                  int64_t bseg, float *__restrict__ part, float *__restrict__ out,
                                                  int accumulate, Key key) {
  using L = Lds1024<8>;
  __shared__ __align__(16) float lds[L::kFloats];
  const LayerDesc &ld = layers[layer];
  const int c0 = blockIdx.x * 8;
  const int64_t v = blockIdx.y;
  const int64_t b_lo = (int64_t)blockIdx.z * bseg;
  const int64_t b_hi = b_lo + bseg < nlive ? b_lo + bseg : nlive;
  // thread: rows r = tid + 256 j (j < 4), column groups c0 + 4 q4 (q4 < 2)
  float acc[4][2][4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int q4 = 0; q4 < 2; ++q4)
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[j][q4][q] = 0.0f;
  float e[32];
  const float *base = src + (int64_t)(c0 + (threadIdx.x >> 5)) * 1024 + (threadIdx.x & 31);
  auto fetch = [&](int64_t b) {
    const float *p = base + (v * nlive + b) * kD;
#pragma unroll
    for (int k = 0; k < 32; ++k) e[k] = p[32 * k];
  };
  fetch(b_lo);
  for (int64_t b = b_lo; b < b_hi; ++b) {
    float cur[32];
#pragma unroll
    for (int k = 0; k < 32; ++k) cur[k] = e[k];
    if (b + 1 < b_hi) fetch(b + 1);
    __syncthreads();  // the previous block's reads of lds are done
    fwht1024_lds_regs<8>(lds, cur);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = threadIdx.x + 256 * j;
      // columns c0 .. c0 + 7 (c0 a multiple of 8) lie in one 32-coordinate sign word
      const int64_t jj = b * kD + (int64_t)r * 1024 + c0;
      const uint32_t bits = sign_word((uint64_t)jj, (uint32_t)ld.layer_id, key) >> (jj & 31);
#pragma unroll
      for (int q4 = 0; q4 < 2; ++q4)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[j][q4][q] += flip(lds[L::idx(4 * q4 + q, r)], (bits >> (4 * q4 + q)) & 1u);
    }
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = threadIdx.x + 256 * j;
#pragma unroll
    for (int q4 = 0; q4 < 2; ++q4) {
      float *o = (part ? part + ((int64_t)blockIdx.z * gridDim.y + v) * kD : out + (b_begin + v) * kD) +
                 (int64_t)r * 1024 + c0 + 4 * q4;
      float4 a = make_float4(acc[j][q4][0], acc[j][q4][1], acc[j][q4][2], acc[j][q4][3]);
      a.x *= 1.0f / 32.0f;
      a.y *= 1.0f / 32.0f;
      a.z *= 1.0f / 32.0f;
      a.w *= 1.0f / 32.0f;
      if (accumulate && !part) {
        const float4 p = *(const float4 *)o;
        a.x += p.x;
        a.y += p.y;
        a.z += p.z;
        a.w += p.w;
      }
      *(float4 *)o = a;
    }
  }
}

// Groups of four vectors (calls whose vector count is a multiple of 4).  The
// intermediates that the permutation gathers from and writes to keep the four
// vectors of group u interleaved: I4[((u nlive + b) D + pos) 4 + w] holds
// position pos of block b of vector 4 u + w.  One 16-byte gather then fetches
// a coordinate of all four vectors (a quarter of the cache-line requests of
// four 4-byte gathers), and the permutation, g and the signs are evaluated
// once per group instead of once per vector.

// H over r of 8 columns c0.. of the group's four vectors (tile row 8 w + cq);
// src per vector in pos order.  kColsG / kColsPlain: times g (kColsG), written
// I4.  kColsOutT: src is I4; + theta0, natural order out (8 consecutive
// outputs per vector and row; the four workgroups of a 32-column block run
// back to back on one XCD, whose L2 joins their pieces of a line).
template <int MODE>
__global__ __launch_bounds__(1024) void k_ffdL_cols4(const LayerDesc *__restrict__ layers, int layer,
                                                     const float *__restrict__ src, int64_t b_begin, int64_t nlive,
                                                     float *__restrict__ dst, void *__restrict__ out, int out_dtype,
                                                     const float *__restrict__ theta0, Key key) {
  using L = Lds1024R32;
  __shared__ __align__(16) float s[L::kFloats];
  const LayerDesc &ld = layers[layer];
  int c0 = blockIdx.x * 8;
  int64_t b = blockIdx.y, u = blockIdx.z;
  const int64_t ng = gridDim.z;
  if (MODE == kColsOutT && (nlive * ng) % 8 == 0) {
    // workgroup id g runs on XCD g mod 8; XCD x takes (block, group) pairs x,
    // x + 8, ... (groups fastest, so theta0 is read from HBM once), and per
    // pair the 32-column blocks one at a time, each as 4 consecutive tasks
    const int64_t g = blockIdx.x + 128 * (blockIdx.y + nlive * blockIdx.z);
    const int64_t k = g >> 3;
    const int64_t pair = 8 * (k >> 7) + (g & 7);
    c0 = (int)(k & 127) * 8;
    b = pair / ng;
    u = pair - b * ng;
  }
  const int ri = threadIdx.x & 31, rc = threadIdx.x >> 5;
  // kColsOutT: theta0 of row 32 rc + m, column c0 + (ri & 7), loaded with the
  // block so the transform hides its latency; positions past n read the last one
  float th[32];
  if (MODE == kColsOutT && theta0) {
    const float *tb = theta0 + b * kD + c0 + (ri & 7);
    const int64_t lim = ld.n - 1 - (b * kD + c0 + (ri & 7));
#pragma unroll
    for (int m = 0; m < 32; ++m) {
      const int64_t o = (int64_t)(32 * rc + m) * 1024;
      const float tv = tb[o < lim ? o : lim];
      th[m] = o <= lim ? tv : 0.0f;
    }
  }
  {
    const int quarter = threadIdx.x >> 8, t = threadIdx.x & 255;
    if (MODE == kColsOutT) {
      // I4 source: thread takes r = 256 quarter + t of the 8 columns, 4 vectors per load
      const float4 *p = (const float4 *)src + (u * nlive + b) * kD + (int64_t)c0 * 1024 + 256 * quarter + t;
      float4 val[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) val[k] = p[k * 1024];
      const int r = 256 * quarter + t;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        s[L::idx(k, r)] = val[k].x;
        s[L::idx(8 + k, r)] = val[k].y;
        s[L::idx(16 + k, r)] = val[k].z;
        s[L::idx(24 + k, r)] = val[k].w;
      }
    } else {
      // per-vector source: thread takes vector 4 u + quarter, r = 4 t .. 4 t + 3 of each column
      const float *p = src + ((4 * u + quarter) * nlive + b) * kD + (int64_t)c0 * 1024 + 4 * t;
      float4 val[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) val[k] = *(const float4 *)(p + k * 1024);
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int i = 8 * quarter + k;
        s[L::idx(i, 4 * t)] = val[k].x;
        s[L::idx(i, 4 * t + 1)] = val[k].y;
        s[L::idx(i, 4 * t + 2)] = val[k].z;
        s[L::idx(i, 4 * t + 3)] = val[k].w;
      }
    }
  }
  __syncthreads();
  float e[32];
  fwht1024_rows32(s, e);
  if (MODE == kColsOutT) {
    // lanes ri = 8 w + cq: row r of vector 4 u + w, column c0 + cq
    const int64_t v = 4 * u + (ri >> 3);
#pragma unroll
    for (int m = 0; m < 32; ++m) {
      const int r = 32 * rc + m;
      const int64_t jj = b * kD + (int64_t)r * 1024 + c0 + (ri & 7);
      if (jj < ld.n)
        store_out(out, out_dtype, (b_begin + v) * ld.n + jj, e[m] * (1.0f / 32.0f) + (theta0 ? th[m] : 0.0f));
    }
    return;
  }
  // back to the block (tile row ri, element r), then thread r writes the 8
  // columns of its row, four vectors per 16-byte store
  __syncthreads();  // every thread's pass-2 reads are done
  float *bq = s + ri * L::kStride + 33 * rc;
#pragma unroll
  for (int m = 0; m < 32; ++m) bq[m] = e[m];
  __syncthreads();
  const int r = threadIdx.x;
  float4 *d4 = (float4 *)dst + (u * nlive + b) * kD + (int64_t)c0 * 1024 + r;
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    float g[4] = {1.0f, 1.0f, 1.0f, 1.0f};
    if (MODE == kColsG)
      gauss4((uint64_t)(b * kD + (int64_t)r * 1024 + c0 + 4 * a) >> 2, (uint32_t)ld.layer_id, ST_GAUSS, key, g);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int cq = 4 * a + q;
      const float f = g[q] * (1.0f / 32.0f);
      d4[cq * 1024] = make_float4(s[L::idx(cq, r)] * f, s[L::idx(8 + cq, r)] * f, s[L::idx(16 + cq, r)] * f,
                                  s[L::idx(24 + cq, r)] * f);
    }
  }
}

// Gather through the permutation and H over c for 8 rows r0.. of the group's
// four vectors (tile row 4 rr + w), I4 in and I4 out (for each column the
// 8 rows x 4 vectors are 32 consecutive floats: one 128-byte line).
// kRowsPermFwd: k = pi^{-1}(d); kRowsPermT: g_i w[pi(i)].
template <int MODE>
__global__ __launch_bounds__(1024) void k_ffdL_rows4(const LayerDesc *__restrict__ layers, int layer,
                                                     const float *__restrict__ src, int64_t nlive,
                                                     float *__restrict__ dst, Key key) {
  using L = Lds1024R32;
  __shared__ __align__(16) float s[L::kFloats];
  const LayerDesc &ld = layers[layer];
  int r0 = blockIdx.x * 8;
  int64_t b = blockIdx.y, u = blockIdx.z;
  if ((nlive * gridDim.z) % 8 == 0) {
    // workgroup id g runs on XCD g mod 8: XCD x takes (group, block) pairs
    // x, x + 8, ... one at a time, so its random reads stay in its own L2
    const int64_t g = blockIdx.x + 128 * (blockIdx.y + nlive * blockIdx.z);
    const int64_t k = g >> 3;
    const int64_t pair = 8 * (k >> 7) + (g & 7);
    r0 = (int)(k & 127) * 8;
    u = pair / nlive;
    b = pair - u * nlive;
  }
  const int64_t blk = (u * nlive + b) * kD;  // this block's I4 region, in float4
  const PermKey pk = perm_key((uint32_t)ld.layer_id, ST_FFDPERM, (uint32_t)b, (uint32_t)kLgD, key);
  const float4 *s4 = (const float4 *)src + blk;
  // thread: rows rr = 2 quarter + h (h < 2); all its gathers are issued first
  const int quarter = threadIdx.x >> 8, t = threadIdx.x & 255;
  float4 val[2][4];
  if (MODE == kRowsPermT) {
    // columns 4 t + q, which share one Philox block of g
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t e0 = (uint32_t)(r0 + 2 * quarter + h) * 1024u + 4u * t;
#pragma unroll
      for (int q = 0; q < 4; ++q) val[h][q] = s4[tpos(perm_fwd(pk, e0 + q))];
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int rr = 2 * quarter + h;
      const uint32_t e0 = (uint32_t)(r0 + rr) * 1024u + 4u * t;
      float g[4];
      gauss4((uint64_t)(b * kD + e0) >> 2, (uint32_t)ld.layer_id, ST_GAUSS, key, g);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c = 4 * t + q;
        s[L::idx(4 * rr, c)] = g[q] * val[h][q].x;
        s[L::idx(4 * rr + 1, c)] = g[q] * val[h][q].y;
        s[L::idx(4 * rr + 2, c)] = g[q] * val[h][q].z;
        s[L::idx(4 * rr + 3, c)] = g[q] * val[h][q].w;
      }
    }
  } else {
    // columns t + 256 q, consecutive over the lanes
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        val[h][q] = s4[tpos(perm_inv(pk, (uint32_t)(r0 + 2 * quarter + h) * 1024u + (uint32_t)(t + 256 * q)))];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int rr = 2 * quarter + h;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c = t + 256 * q;
        s[L::idx(4 * rr, c)] = val[h][q].x;
        s[L::idx(4 * rr + 1, c)] = val[h][q].y;
        s[L::idx(4 * rr + 2, c)] = val[h][q].z;
        s[L::idx(4 * rr + 3, c)] = val[h][q].w;
      }
    }
  }
  __syncthreads();
  float e[32];
  fwht1024_rows32(s, e);
  const int ri = threadIdx.x & 31, rc = threadIdx.x >> 5;
  // column 32 rc + m, tile row ri: float ((32 rc + m) 1024 + r0) 4 + ri of the block's I4 region
  const __amdgpu_buffer_rsrc_t ws = buf_rsrc(dst + (blk + r0) * 4, (uint32_t)((kD - r0) * 16));
  const int soff = (32 * rc * 4096 + ri) * 4;
#pragma unroll
  for (int m = 0; m < 32; ++m)
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(e[m] * (1.0f / 32.0f)), ws, soff, m * 16384, 0);
}

// Forward epilogue of a group: for 2 columns c0.. of the four vectors (tile
// row 4 cq + w), sum over the blocks b_lo .. b_hi - 1 of run z of B_b times
// H over r; the next block's columns load during the current one.  Writes
// part[((z bc + v) 1024 + c) 1024 + r] (k_ffdL_outT turns it into out).
__global__ __launch_bounds__(256) void k_ffdL_sum4(const LayerDesc *__restrict__ layers, int layer,
                                                   const float *__restrict__ src, int64_t nlive, int64_t bseg,
                                                   float *__restrict__ part, Key key) {
  using L = Lds1024<8>;
  __shared__ __align__(16) float lds[L::kFloats];
  const LayerDesc &ld = layers[layer];
  const int c0 = blockIdx.x * 2;
  const int64_t u = blockIdx.y, bc = 4 * (int64_t)gridDim.y;
  const int64_t b_lo = (int64_t)blockIdx.z * bseg;
  const int64_t b_hi = b_lo + bseg < nlive ? b_lo + bseg : nlive;
  float acc[4][8];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[j][q] = 0.0f;
  // loads: column c0 + cq0, rows rl + 128 k, four vectors each
  const int cq0 = threadIdx.x >> 7, rl = threadIdx.x & 127;
  const float4 *base = (const float4 *)src + (int64_t)(c0 + cq0) * 1024 + rl;
  float4 e[8];
  auto fetch = [&](int64_t b) {
    const float4 *p = base + (u * nlive + b) * kD;
#pragma unroll
    for (int k = 0; k < 8; ++k) e[k] = p[128 * k];
  };
  fetch(b_lo);
  for (int64_t b = b_lo; b < b_hi; ++b) {
    float4 cur[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) cur[k] = e[k];
    if (b + 1 < b_hi) fetch(b + 1);
    __syncthreads();  // the previous block's reads of lds are done
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int r = rl + 128 * k;
      lds[L::idx(4 * cq0, r)] = cur[k].x;
      lds[L::idx(4 * cq0 + 1, r)] = cur[k].y;
      lds[L::idx(4 * cq0 + 2, r)] = cur[k].z;
      lds[L::idx(4 * cq0 + 3, r)] = cur[k].w;
    }
    __syncthreads();
    fwht1024_lds<8>(lds);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = threadIdx.x + 256 * j;
      // columns c0, c0 + 1 (c0 even) lie in one 32-coordinate sign word
      const int64_t jj = b * kD + (int64_t)r * 1024 + c0;
      const uint32_t bits = sign_word((uint64_t)jj, (uint32_t)ld.layer_id, key) >> (jj & 31);
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[j][q] += flip(lds[L::idx(q, r)], (bits >> (q >> 2)) & 1u);
    }
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = threadIdx.x + 256 * j;
#pragma unroll
    for (int q = 0; q < 8; ++q)
      part[(((int64_t)blockIdx.z * bc + 4 * u + (q & 3)) * 1024 + c0 + (q >> 2)) * 1024 + r] =
          acc[j][q] * (1.0f / 32.0f);
  }
}

// out[v][i] (+)= sum over runs z < nseg (at most 8) of part[(z bc + v) D + i],
// in the order of z: one float4 per thread, all its runs' loads in flight.
__global__ __launch_bounds__(256) void k_ffdL_segsum(const float *__restrict__ part, int nseg, int64_t bc,
                                                     int64_t b_begin, float *__restrict__ out, int accumulate) {
  const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;  // float4 index within the vector
  const int64_t v = blockIdx.y;
  float4 t[8];
#pragma unroll
  for (int z = 0; z < 8; ++z)
    if (z < nseg) t[z] = ((const float4 *)part)[(z * bc + v) * (kD / 4) + p];
  float4 a = t[0];
#pragma unroll
  for (int z = 1; z < 8; ++z)
    if (z < nseg) {
      a.x += t[z].x;
      a.y += t[z].y;
      a.z += t[z].z;
      a.w += t[z].w;
    }
  float4 *o = (float4 *)(out + (b_begin + v) * kD) + p;
  if (accumulate) {
    const float4 q = *o;
    a.x += q.x;
    a.y += q.y;
    a.z += q.z;
    a.w += q.w;
  }
  *o = a;
}

// out[v][r 1024 + c] (+)= sum over runs z < nseg of part[((z bc + v) 1024 + c)
// 1024 + r], in the order of z; 32 x 32 tiles through LDS (128-byte reads and
// writes).  Grid (32, 32, bc).
__global__ __launch_bounds__(256) void k_ffdL_outT(const float *__restrict__ part, int64_t nseg, int64_t bc,
                                                   int64_t b_begin, float *__restrict__ out, int accumulate) {
  __shared__ float tl[32][33];
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
  const int64_t v = blockIdx.z;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int c = c0 + ty + 8 * k;
    float a = 0.0f;
    for (int64_t z = 0; z < nseg; ++z) a += part[((z * bc + v) * 1024 + c) * 1024 + r0 + tx];
    tl[ty + 8 * k][tx] = a;
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int r = r0 + ty + 8 * k;
    float *o = out + (b_begin + v) * kD + (int64_t)r * 1024 + c0 + tx;
    float a = tl[tx][ty + 8 * k];
    if (accumulate) a += *o;
    *o = a;
  }
}

// Permutation through buckets (groups of four vectors, bucket offsets stored
// at creation).  The producer (a cols pass: source positions k of 8 columns
// c0.. and all rows, source group s = c0 / 8) computes each destination d,
// counting-sorts its 8192 coordinates in LDS by destination chunk q = d >> 13
// (8 rows), and writes each chunk's run, four vectors per 16-byte word, at its
// offset in chunk q's bucket of 8192 words, with d & 8191 beside it (uint16).
// The consumer (a rows pass over chunk q) reads the bucket as one contiguous
// range and places every word at its destination in LDS: both passes read and
// write whole lines, where the gather read a line per coordinate.  The order
// inside a run follows LDS atomics; the placement, hence the result, does not.

// Per (source group s, block b, direction): how many of its 8192 coordinates
// go to each destination chunk.
__global__ __launch_bounds__(1024) void k_ffdL_bcount(const LayerDesc *__restrict__ layers, int layer,
                                                      uint16_t *__restrict__ tab, Key key) {
  __shared__ uint32_t hist[128];
  const LayerDesc &ld = layers[layer];
  const int sg = blockIdx.x, dir = blockIdx.z;
  const int64_t b = blockIdx.y;
  if (threadIdx.x < 128) hist[threadIdx.x] = 0u;
  __syncthreads();
  const PermKey pk = perm_key((uint32_t)ld.layer_id, ST_FFDPERM, (uint32_t)b, (uint32_t)kLgD, key);
#pragma unroll
  for (int cq = 0; cq < 8; ++cq) {
    const uint32_t k = (uint32_t)threadIdx.x * 1024u + 8u * sg + cq;
    const uint32_t d = dir ? perm_inv(pk, k) : perm_fwd(pk, k);
    atomicAdd(&hist[d >> 13], 1u);
  }
  __syncthreads();
  if (threadIdx.x < 128) tab[((b * 2 + dir) * 128 + sg) * 128 + threadIdx.x] = (uint16_t)hist[threadIdx.x];
}

// Counts -> run starts: exclusive prefix over the source groups of each chunk.
__global__ __launch_bounds__(128) void k_ffdL_bscan(uint16_t *__restrict__ tab) {
  uint16_t *t = tab + (int64_t)blockIdx.x * 128 * 128 + threadIdx.x;
  uint32_t run = 0;
  for (int sg = 0; sg < 128; ++sg) {
    const uint32_t c = t[sg * 128];
    t[sg * 128] = (uint16_t)run;
    run += c;
  }
}

// Producer: H over r of 8 columns c0.. of the group's four vectors (as
// k_ffdL_cols4, times g for kColsG), then the bucket writes.  kColsG (forward)
// sends k to d = pi(k), kColsPlain (transpose) to d = pi^{-1}(k).
template <int MODE>
__global__ __launch_bounds__(1024) void k_ffdL_cols4b(const LayerDesc *__restrict__ layers, int layer,
                                                      const float *__restrict__ src, int64_t nlive,
                                                      const uint16_t *__restrict__ tab, float *__restrict__ dst,
                                                      uint16_t *__restrict__ didx, Key key) {
  using L = Lds1024R32;
  // after the transform: 8192 words, their uint16 destinations and uint8
  // chunks; past the tile: counts, run starts in this workgroup and run
  // starts in the buckets
  constexpr int kStage = 8192 * 4 + 8192 / 2 + 8192 / 4;
  constexpr int kFl = (kStage > L::kFloats ? kStage : L::kFloats) + 3 * 128;
  __shared__ __align__(16) float s[kFl];
  const LayerDesc &ld = layers[layer];
  const int sg = blockIdx.x, c0 = 8 * sg;
  const int64_t b = blockIdx.y, u = blockIdx.z;
  constexpr int dir = MODE == kColsG ? 0 : 1;
  uint32_t *cnt = (uint32_t *)(s + kFl - 3 * 128), *loc = cnt + 128, *boff = cnt + 256;
  // the run starts, then the tile, are loaded first; everything that depends
  // only on positions (destinations, ranks, run offsets, g) is made while the
  // tile is in flight
  uint32_t tb = 0;
  if (threadIdx.x < 128) tb = tab[((b * 2 + dir) * 128 + sg) * 128 + threadIdx.x];
  const int quarter = threadIdx.x >> 8, t = threadIdx.x & 255;
  float4 val[8];
  {
    const float *p = src + ((4 * u + quarter) * nlive + b) * kD + (int64_t)c0 * 1024 + 4 * t;
#pragma unroll
    for (int k = 0; k < 8; ++k) val[k] = *(const float4 *)(p + k * 1024);
  }
  if (threadIdx.x < 128) cnt[threadIdx.x] = 0u;
  // thread r: sources k = r 1024 + c0 + cq of row r
  const int r = threadIdx.x;
  const PermKey pk = perm_key((uint32_t)ld.layer_id, ST_FFDPERM, (uint32_t)b, (uint32_t)kLgD, key);
  uint32_t dd[8], rank[8];
#pragma unroll
  for (int cq = 0; cq < 8; ++cq) {
    const uint32_t k = (uint32_t)r * 1024u + (uint32_t)(c0 + cq);
    dd[cq] = dir ? perm_inv(pk, k) : perm_fwd(pk, k);
  }
  float g[8];
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    if (MODE == kColsG)
      gauss4((uint64_t)(b * kD + (int64_t)r * 1024 + c0 + 4 * a) >> 2, (uint32_t)ld.layer_id, ST_GAUSS, key, g + 4 * a);
    else
      g[4 * a] = g[4 * a + 1] = g[4 * a + 2] = g[4 * a + 3] = 1.0f;
  }
  if (threadIdx.x < 128) boff[threadIdx.x] = tb;
  __syncthreads();  // counters zeroed
#pragma unroll
  for (int cq = 0; cq < 8; ++cq) rank[cq] = atomicAdd(&cnt[dd[cq] >> 13], 1u);
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t run = 0;
#pragma unroll 8
    for (int q = 0; q < 128; ++q) {
      loc[q] = run;
      run += cnt[q];
    }
  }
  // tile: H over r of the 8 columns of the four vectors (tile row 8 w + cq)
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int i = 8 * quarter + k;
    s[L::idx(i, 4 * t)] = val[k].x;
    s[L::idx(i, 4 * t + 1)] = val[k].y;
    s[L::idx(i, 4 * t + 2)] = val[k].z;
    s[L::idx(i, 4 * t + 3)] = val[k].w;
  }
  __syncthreads();
  float e[32];
  fwht1024_rows32(s, e);
  const int ri = threadIdx.x & 31, rc = threadIdx.x >> 5;
  __syncthreads();  // every thread's pass-2 reads are done
  {
    float *bq = s + ri * L::kStride + 33 * rc;
#pragma unroll
    for (int m = 0; m < 32; ++m) bq[m] = e[m];
  }
  __syncthreads();
  float4 v4[8];
#pragma unroll
  for (int cq = 0; cq < 8; ++cq) {
    const float f = g[cq] * (1.0f / 32.0f);
    v4[cq] = make_float4(s[L::idx(cq, r)] * f, s[L::idx(8 + cq, r)] * f, s[L::idx(16 + cq, r)] * f,
                         s[L::idx(24 + cq, r)] * f);
  }
  float4 *stg = (float4 *)s;
  uint16_t *sdd = (uint16_t *)(s + 8192 * 4);
  uint8_t *sq = (uint8_t *)(s + 8192 * 4 + 8192 / 2);
  __syncthreads();  // the tile has been read: its space becomes the staging area
#pragma unroll
  for (int cq = 0; cq < 8; ++cq) {
    const uint32_t q = dd[cq] >> 13, pos = loc[q] + rank[cq];
    stg[pos] = v4[cq];
    sdd[pos] = (uint16_t)(dd[cq] & 8191u);
    sq[pos] = (uint8_t)q;
  }
  __syncthreads();
  float4 *d4 = (float4 *)dst + (u * nlive + b) * kD;
  uint16_t *dx = didx + (u * nlive + b) * kD;
#pragma unroll
  for (int m = 0; m < 8; ++m) {
    const uint32_t j = threadIdx.x + 1024u * m;
    const uint32_t q = sq[j];
    const uint32_t at = boff[q] + (j - loc[q]);
    if (at < 8192u) {
      d4[q * 8192 + at] = stg[j];
      dx[q * 8192 + at] = sdd[j];
    }
  }
}

// Consumer: chunk q (rows 8 q ..) of the group's four vectors from its bucket
// (tile row 4 rr + w), g_i for kRowsPermT, H over c, written I4 as k_ffdL_rows4.
template <int MODE>
__global__ __launch_bounds__(1024) void k_ffdL_rows4b(const LayerDesc *__restrict__ layers, int layer,
                                                      const float *__restrict__ src,
                                                      const uint16_t *__restrict__ didx, int64_t nlive,
                                                      float *__restrict__ dst, Key key) {
  using L = Lds1024R32;
  __shared__ __align__(16) float s[L::kFloats];
  const LayerDesc &ld = layers[layer];
  const int q = blockIdx.x, r0 = 8 * q;
  const int64_t b = blockIdx.y, u = blockIdx.z;
  const int64_t blk = (u * nlive + b) * kD;
  const int quarter = threadIdx.x >> 8, t = threadIdx.x & 255;
  float g[2][4];
  {
    const float4 *s4 = (const float4 *)src + blk + q * 8192;
    const uint16_t *ix = didx + blk + q * 8192;
    float4 val[8];
    uint32_t dd[8];
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      val[m] = s4[threadIdx.x + 1024 * m];
      dd[m] = ix[threadIdx.x + 1024 * m];
    }
    // kRowsPermT: g_i of the destinations columns 4 t + qq of rows 2 quarter + h,
    // made while the bucket is in flight
    if (MODE == kRowsPermT)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        gauss4((uint64_t)(b * kD + (int64_t)(r0 + 2 * quarter + h) * 1024 + 4 * t) >> 2, (uint32_t)ld.layer_id,
               ST_GAUSS, key, g[h]);
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      const int rr = (int)(dd[m] >> 10) & 7, c = (int)(dd[m] & 1023u);
      s[L::idx(4 * rr, c)] = val[m].x;
      s[L::idx(4 * rr + 1, c)] = val[m].y;
      s[L::idx(4 * rr + 2, c)] = val[m].z;
      s[L::idx(4 * rr + 3, c)] = val[m].w;
    }
  }
  __syncthreads();
  if (MODE == kRowsPermT) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int rr = 2 * quarter + h;
#pragma unroll
      for (int qq = 0; qq < 4; ++qq)
#pragma unroll
        for (int w = 0; w < 4; ++w) s[L::idx(4 * rr + w, 4 * t + qq)] *= g[h][qq];
    }
    __syncthreads();
  }
  float e[32];
  fwht1024_rows32(s, e);
  const int ri = threadIdx.x & 31, rc = threadIdx.x >> 5;
  const __amdgpu_buffer_rsrc_t ws = buf_rsrc(dst + (blk + r0) * 4, (uint32_t)((kD - r0) * 16));
  const int soff = (32 * rc * 4096 + ri) * 4;
#pragma unroll
  for (int m = 0; m < 32; ++m)
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(e[m] * (1.0f / 32.0f)), ws, soff, m * 16384, 0);
}

}  // namespace

bool ffd_large_path(const sk_sketch *s) { return s->D == kD; }

void launch_ffd_bucket_tab(const sk_sketch *s, int layer, uint16_t *tab, hipStream_t st) {
  const int64_t nlive = ffd_live_blocks(s, layer);
  hipLaunchKernelGGL(k_ffdL_bcount, dim3(128u, (unsigned)nlive, 2u), dim3(1024), 0, st, s->d_layers, layer, tab,
                     s->key);
  hipLaunchKernelGGL(k_ffdL_bscan, dim3((unsigned)(nlive * 2)), dim3(128), 0, st, tab);
  (void)hipGetLastError();
}

void run_ffd_large_fwd(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc,
                       float *out, bool accumulate, int phases, hipStream_t st) {
  const int64_t nlive = ffd_live_blocks(s, layer);
  float *A = s->ws, *B = s->ws + bc * nlive * kD;
  const dim3 gr(32u, (unsigned)nlive, (unsigned)bc);
  if (phases & 1) {
    if (dtype == SK_BF16)
      hipLaunchKernelGGL((k_ffdL_rows<kRowsX, true>), gr, dim3(1024), 0, st, s->d_layers, layer, x, b_begin, nlive, A,
                         s->key);
    else
      hipLaunchKernelGGL((k_ffdL_rows<kRowsX, false>), gr, dim3(1024), 0, st, s->d_layers, layer, x, b_begin, nlive,
                         A, s->key);
  }
  if ((phases & 2) && bc % 4 == 0) {
    const int64_t ng = bc / 4;
    const dim3 g4(128u, (unsigned)nlive, (unsigned)ng);
    if (s->d_ffdb && s->ffdb_off[layer] >= 0) {
      uint16_t *ix = (uint16_t *)(s->ws + 2 * bc * nlive * kD);
      hipLaunchKernelGGL(k_ffdL_cols4b<kColsG>, g4, dim3(1024), 0, st, s->d_layers, layer, A, nlive,
                         s->d_ffdb + s->ffdb_off[layer], B, ix, s->key);
      hipLaunchKernelGGL(k_ffdL_rows4b<kRowsPermFwd>, g4, dim3(1024), 0, st, s->d_layers, layer, B, ix, nlive, A,
                         s->key);
    } else {
      hipLaunchKernelGGL(k_ffdL_cols4<kColsG>, g4, dim3(1024), 0, st, s->d_layers, layer, A, b_begin, nlive, B,
                         nullptr, 0, nullptr, s->key);
      hipLaunchKernelGGL(k_ffdL_rows4<kRowsPermFwd>, g4, dim3(1024), 0, st, s->d_layers, layer, B, nlive, A, s->key);
    }
    // 512 column pairs per group: split the blocks into runs only when that
    // leaves under two workgroups per CU
    const int64_t want = 512 * ng < 512 ? 2 : 1;
    const int64_t nseg0 = want < nlive ? want : nlive;
    const int64_t bseg = (nlive + nseg0 - 1) / nseg0, nseg = (nlive + bseg - 1) / bseg;
    hipLaunchKernelGGL(k_ffdL_sum4, dim3(512u, (unsigned)ng, (unsigned)nseg), dim3(256), 0, st, s->d_layers, layer, A,
                       nlive, bseg, B, s->key);
    hipLaunchKernelGGL(k_ffdL_outT, dim3(32u, 32u, (unsigned)bc), dim3(256), 0, st, B, nseg, bc, b_begin, out,
                       (int)accumulate);
  } else if (phases & 2) {
    hipLaunchKernelGGL(k_ffdL_cols<kColsG>, gr, dim3(1024), 0, st, s->d_layers, layer, A, b_begin, nlive, B, nullptr,
                       0, nullptr, s->key);
    hipLaunchKernelGGL((k_ffdL_rows<kRowsPermFwd, false>), gr, dim3(1024), 0, st, s->d_layers, layer, B, b_begin,
                       nlive, A, s->key);
    // Under two workgroups per CU (128 column groups per vector), the blocks
    // split into runs, for about four per CU, whose partial sums land in B
    // (free here); at two or more the extra pass costs more than it gains.
    const int64_t want = 128 * bc < 512 ? (1024 + 128 * bc - 1) / (128 * bc) : 1;
    const int64_t nseg0 = want < nlive ? want : nlive;
    const int64_t bseg = (nlive + nseg0 - 1) / nseg0, nseg = (nlive + bseg - 1) / bseg;
    hipLaunchKernelGGL(k_ffdL_sum, dim3(128u, (unsigned)bc, (unsigned)nseg), dim3(256), 0, st, s->d_layers, layer, A,
                       b_begin, nlive, bseg, nseg > 1 ? B : nullptr, out, (int)accumulate, s->key);
    if (nseg > 1 && ((uintptr_t)out & 15) == 0)  // nseg <= 8 here
      hipLaunchKernelGGL(k_ffdL_segsum, dim3((unsigned)(kD / 4 / 256), (unsigned)bc), dim3(256), 0, st, B, (int)nseg,
                         bc, b_begin, out, (int)accumulate);
    else if (nseg > 1)
      launch_reduce_partials(B, nseg, bc, kD, b_begin, out, accumulate, st);
  }
  (void)hipGetLastError();
}

void run_ffd_large_T(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, void *out,
                     int out_dtype, const float *theta0, int phases, hipStream_t st) {
  const int64_t nlive = ffd_live_blocks(s, layer);
  float *A = s->ws, *B = s->ws + bc * nlive * kD;
  const dim3 gr(32u, (unsigned)nlive, (unsigned)bc);
  if (bc % 4 == 0) {
    const dim3 g4(128u, (unsigned)nlive, (unsigned)(bc / 4));
    if (phases & 1) {
      hipLaunchKernelGGL((k_ffdL_rows<kRowsZ, false>), gr, dim3(1024), 0, st, s->d_layers, layer, z, b_begin, nlive,
                         A, s->key);
      if (s->d_ffdb && s->ffdb_off[layer] >= 0) {
        uint16_t *ix = (uint16_t *)(s->ws + 2 * bc * nlive * kD);
        hipLaunchKernelGGL(k_ffdL_cols4b<kColsPlain>, g4, dim3(1024), 0, st, s->d_layers, layer, A, nlive,
                           s->d_ffdb + s->ffdb_off[layer], B, ix, s->key);
        hipLaunchKernelGGL(k_ffdL_rows4b<kRowsPermT>, g4, dim3(1024), 0, st, s->d_layers, layer, B, ix, nlive, A,
                           s->key);
      } else {
        hipLaunchKernelGGL(k_ffdL_cols4<kColsPlain>, g4, dim3(1024), 0, st, s->d_layers, layer, A, b_begin, nlive,
                           B, nullptr, 0, nullptr, s->key);
        hipLaunchKernelGGL(k_ffdL_rows4<kRowsPermT>, g4, dim3(1024), 0, st, s->d_layers, layer, B, nlive, A, s->key);
      }
    }
    if (phases & 2)
      hipLaunchKernelGGL(k_ffdL_cols4<kColsOutT>, g4, dim3(1024), 0, st, s->d_layers, layer, A, b_begin, nlive,
                         nullptr, out, out_dtype, theta0, s->key);
    (void)hipGetLastError();
    return;
  }
  if (phases & 1) {
    hipLaunchKernelGGL((k_ffdL_rows<kRowsZ, false>), gr, dim3(1024), 0, st, s->d_layers, layer, z, b_begin, nlive, A,
                       s->key);
    hipLaunchKernelGGL(k_ffdL_cols<kColsPlain>, gr, dim3(1024), 0, st, s->d_layers, layer, A, b_begin, nlive, B,
                       nullptr, 0, nullptr, s->key);
    hipLaunchKernelGGL((k_ffdL_rows<kRowsPermT, false>), gr, dim3(1024), 0, st, s->d_layers, layer, B, b_begin, nlive,
                       A, s->key);
  }
  if (phases & 2)
    hipLaunchKernelGGL(k_ffdL_cols<kColsOutT>, gr, dim3(1024), 0, st, s->d_layers, layer, A, b_begin, nlive, nullptr,
                       out, out_dtype, theta0, s->key);
  (void)hipGetLastError();
}

}  // namespace sk
