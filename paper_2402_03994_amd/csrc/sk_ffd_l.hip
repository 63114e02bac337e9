// sk_ffd_l.hip -- FFD (eq. fastfood) blocks of D = 2^20.
//
// A block index i splits into (r, c) = (i >> 10, i & 1023) and
// H_D = H_1024(r) (x) H_1024(c).  Intermediates are kept transposed: position
// pos(i) = c 1024 + r holds element i, so that both 1024-point transforms read
// and write whole rows:
//   rows kernel  16 rows r of a block: gather / load, H over c, write pos()
//   cols kernel  16 columns c (contiguous in pos order): H over r, epilogue
// Forward y = sum_b B_b H Pi_b^T G_b H x_b:
//   rows(x) -> cols(. g, pos order) -> rows(gather k = pi^{-1}(d)) -> sum over
//   blocks of B_b . cols(.) in registers -> y.
// Transpose block b = H G_b Pi_b H B_b z:
//   rows(B_b z) -> cols -> rows(g_i . gather k = pi(i)) -> cols -> theta.
// Each kernel applies 1/32 (a normalised H_1024).
#include "sk_kcommon.h"
#include "sk_launch.h"

namespace sk {

namespace {

constexpr int kLgD = 20;
constexpr int64_t kD = 1ll << kLgD;

__device__ __forceinline__ uint32_t tpos(uint32_t i) { return ((i & 1023u) << 10) | (i >> 10); }

enum RowsMode { kRowsX = 0, kRowsZ = 1, kRowsPermFwd = 2, kRowsPermT = 3 };

// Rows kernel: workgroup per (16 rows r0.., block b, vector v).
template <int MODE, bool BF16>
__global__ __launch_bounds__(256) void k_ffdL_rows(const LayerDesc *__restrict__ layers, int layer,
                                                   const void *__restrict__ src, int64_t b_begin, int64_t nlive,
                                                   float *__restrict__ dst, Key key) {
  using L = Lds1024R;
  __shared__ __align__(16) float s[L::kFloats];
  __shared__ __align__(16) uint32_t sg[16 * 32];
  const LayerDesc &ld = layers[layer];
  int r0 = blockIdx.x * 16;
  int64_t b = blockIdx.y, v = blockIdx.z;
  if ((MODE == kRowsPermFwd || MODE == kRowsPermT) && (nlive * gridDim.z) % 8 == 0) {
    // workgroup id g runs on XCD g mod 8: XCD x takes (vector, block) pairs
    // x, x + 8, ... one at a time, so its random reads stay in its own L2
    const int64_t g = blockIdx.x + 64 * (blockIdx.y + nlive * blockIdx.z);
    const int64_t k = g >> 3;
    const int64_t pair = 8 * (k >> 6) + (g & 7);
    r0 = (int)(k & 63) * 16;
    v = pair / nlive;
    b = pair - v * nlive;
  }
  const int64_t blk = (v * nlive + b) * kD;  // this block in the workspace
  if (MODE == kRowsZ) {
    // B_b signs of the 16 rows: 8 Philox blocks of 128 per row, shared in LDS
    if (threadIdx.x < 128) {
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
  // all 64 loads of a thread are issued before any LDS write
  float val[16][4];
  if (MODE == kRowsPermT) {
    // u_i = g_i w[pi(i)]: four consecutive columns per thread share one Philox block
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const uint32_t e0 = (uint32_t)(r0 + i) * 1024u + 4u * threadIdx.x;
#pragma unroll
      for (int q = 0; q < 4; ++q) val[i][q] = ((const float *)src)[blk + tpos(perm_fwd(pk, e0 + q))];
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const uint32_t e0 = (uint32_t)(r0 + i) * 1024u + 4u * threadIdx.x;
      float g[4];
      gauss4((uint64_t)(b * kD + e0) >> 2, (uint32_t)ld.layer_id, ST_GAUSS, key, g);
#pragma unroll
      for (int q = 0; q < 4; ++q) s[L::idx(i, 4 * threadIdx.x + q)] = g[q] * val[i][q];
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int c = threadIdx.x + 256 * k;
        const uint32_t e = (uint32_t)(r0 + i) * 1024u + (uint32_t)c;
        if (MODE == kRowsX) {
          const int64_t j = b * kD + e;
          const int64_t x = (b_begin + v) * ld.n + j;
          val[i][k] = j < ld.n ? (BF16 ? bf16_to_f32(((const uint16_t *)src)[x]) : ((const float *)src)[x]) : 0.0f;
        } else if (MODE == kRowsZ) {
          const uint32_t bit = (sg[i * 32 + (c >> 5)] >> (c & 31)) & 1u;
          val[i][k] = flip(((const float *)src)[(b_begin + v) * kD + e], bit);
        } else {  // kRowsPermFwd: d = e, k = pi^{-1}(d)
          val[i][k] = ((const float *)src)[blk + tpos(perm_inv(pk, e))];
        }
      }
    }
#pragma unroll
    for (int i = 0; i < 16; ++i)
#pragma unroll
      for (int k = 0; k < 4; ++k) s[L::idx(i, threadIdx.x + 256 * k)] = val[i][k];
  }
  __syncthreads();
  float e[64];
  fwht1024_rows16_r(s, e);
  const int ri = threadIdx.x & 15, rc = threadIdx.x >> 4;
  float *o = dst + blk + (int64_t)(64 * rc) * 1024 + r0 + ri;
#pragma unroll
  for (int m = 0; m < 64; ++m) o[(int64_t)m * 1024] = e[m] * (1.0f / 32.0f);
}

enum ColsMode { kColsG = 0, kColsPlain = 1, kColsOutT = 2 };

// Cols kernel: workgroup per (16 columns c0.., block b, vector v); the 16
// columns are 16 contiguous rows of the transposed block.
template <int MODE>
__global__ __launch_bounds__(256) void k_ffdL_cols(const LayerDesc *__restrict__ layers, int layer,
                                                   const float *__restrict__ src, int64_t b_begin, int64_t nlive,
                                                   float *__restrict__ dst, void *__restrict__ out, int out_dtype,
                                                   const float *__restrict__ theta0, Key key) {
  using L = Lds1024<16>;
  __shared__ __align__(16) float lds[L::kFloats];
  const LayerDesc &ld = layers[layer];
  const int c0 = blockIdx.x * 16;
  const int64_t b = blockIdx.y, v = blockIdx.z;
  const int64_t blk = (v * nlive + b) * kD;
  float e[64];
  {
    const float *p = src + blk + (int64_t)(c0 + (threadIdx.x >> 4)) * 1024 + (threadIdx.x & 15);
#pragma unroll
    for (int k = 0; k < 64; ++k) e[k] = p[16 * k];
  }
  fwht1024_lds_regs<16>(lds, e);
  if (MODE == kColsOutT) {
    // natural order: the 16 lanes of a row r write its 16 columns (64 bytes)
    const int cc = threadIdx.x & 15;
#pragma unroll 8
    for (int j = 0; j < 64; ++j) {
      const int r = (threadIdx.x >> 4) + 16 * j;
      const int64_t jj = b * kD + (int64_t)r * 1024 + c0 + cc;
      if (jj < ld.n)
        store_out(out, out_dtype, (b_begin + v) * ld.n + jj,
                  lds[L::idx(cc, r)] * (1.0f / 32.0f) + (theta0 ? theta0[jj] : 0.0f));
    }
    return;
  }
  // thread: rows r = tid + 256 j, column groups c0 + 4 q4 .. + 3; writes in pos order
#pragma unroll 2
  for (int j = 0; j < 4; ++j) {
    const int r = threadIdx.x + 256 * j;
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const int cb = c0 + 4 * q4;
      float val[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) val[q] = lds[L::idx(4 * q4 + q, r)] * (1.0f / 32.0f);
      if (MODE == kColsG) {
        float g[4];
        gauss4((uint64_t)(b * kD + (int64_t)r * 1024 + cb) >> 2, (uint32_t)ld.layer_id, ST_GAUSS, key, g);
#pragma unroll
        for (int q = 0; q < 4; ++q) dst[blk + (int64_t)(cb + q) * 1024 + r] = g[q] * val[q];
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) dst[blk + (int64_t)(cb + q) * 1024 + r] = val[q];
      }
    }
  }
}

// Forward epilogue: out[v][i] (+)= sum_b B_b(i) (H over r of block b)[i] for 8
// columns per workgroup; the next block's columns load during the current one.
__global__ __launch_bounds__(256) void k_ffdL_sum(const LayerDesc *__restrict__ layers, int layer,
                                                  const float *__restrict__ src, int64_t b_begin, int64_t nlive,
                                                  float *__restrict__ out, int accumulate, Key key) {
  using L = Lds1024<8>;
  __shared__ __align__(16) float lds[L::kFloats];
  const LayerDesc &ld = layers[layer];
  const int c0 = blockIdx.x * 8;
  const int64_t v = blockIdx.y;
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
  fetch(0);
  for (int64_t b = 0; b < nlive; ++b) {
    float cur[32];
#pragma unroll
    for (int k = 0; k < 32; ++k) cur[k] = e[k];
    if (b + 1 < nlive) fetch(b + 1);
    __syncthreads();  // the previous block's reads of lds are done
    fwht1024_lds_regs<8>(lds, cur);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = threadIdx.x + 256 * j;
#pragma unroll
      for (int q4 = 0; q4 < 2; ++q4) {
        const int64_t jj = b * kD + (int64_t)r * 1024 + c0 + 4 * q4;
        const uint32_t bits = sign_word((uint64_t)jj, (uint32_t)ld.layer_id, key) >> (jj & 31);
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[j][q4][q] += flip(lds[L::idx(4 * q4 + q, r)], (bits >> q) & 1u);
      }
    }
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = threadIdx.x + 256 * j;
#pragma unroll
    for (int q4 = 0; q4 < 2; ++q4) {
      float *o = out + (b_begin + v) * kD + (int64_t)r * 1024 + c0 + 4 * q4;
      float4 a = make_float4(acc[j][q4][0], acc[j][q4][1], acc[j][q4][2], acc[j][q4][3]);
      a.x *= 1.0f / 32.0f;
      a.y *= 1.0f / 32.0f;
      a.z *= 1.0f / 32.0f;
      a.w *= 1.0f / 32.0f;
      if (accumulate) {
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

}  // namespace

bool ffd_large_path(const sk_sketch *s) { return s->D == kD; }

void run_ffd_large_fwd(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc,
                       float *out, bool accumulate, int phases, hipStream_t st) {
  const int64_t nlive = ffd_live_blocks(s, layer);
  float *A = s->ws, *B = s->ws + bc * nlive * kD;
  const dim3 gr(64u, (unsigned)nlive, (unsigned)bc);
  if (phases & 1) {
    if (dtype == SK_BF16)
      hipLaunchKernelGGL((k_ffdL_rows<kRowsX, true>), gr, dim3(256), 0, st, s->d_layers, layer, x, b_begin, nlive, A,
                         s->key);
    else
      hipLaunchKernelGGL((k_ffdL_rows<kRowsX, false>), gr, dim3(256), 0, st, s->d_layers, layer, x, b_begin, nlive,
                         A, s->key);
  }
  if (phases & 2) {
    hipLaunchKernelGGL(k_ffdL_cols<kColsG>, gr, dim3(256), 0, st, s->d_layers, layer, A, b_begin, nlive, B, nullptr,
                       0, nullptr, s->key);
    hipLaunchKernelGGL((k_ffdL_rows<kRowsPermFwd, false>), gr, dim3(256), 0, st, s->d_layers, layer, B, b_begin,
                       nlive, A, s->key);
    hipLaunchKernelGGL(k_ffdL_sum, dim3(128u, (unsigned)bc), dim3(256), 0, st, s->d_layers, layer, A, b_begin, nlive,
                       out, (int)accumulate, s->key);
  }
  (void)hipGetLastError();
}

void run_ffd_large_T(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, void *out,
                     int out_dtype, const float *theta0, int phases, hipStream_t st) {
  const int64_t nlive = ffd_live_blocks(s, layer);
  float *A = s->ws, *B = s->ws + bc * nlive * kD;
  const dim3 gr(64u, (unsigned)nlive, (unsigned)bc);
  if (phases & 1) {
    hipLaunchKernelGGL((k_ffdL_rows<kRowsZ, false>), gr, dim3(256), 0, st, s->d_layers, layer, z, b_begin, nlive, A,
                       s->key);
    hipLaunchKernelGGL(k_ffdL_cols<kColsPlain>, gr, dim3(256), 0, st, s->d_layers, layer, A, b_begin, nlive, B,
                       nullptr, 0, nullptr, s->key);
    hipLaunchKernelGGL((k_ffdL_rows<kRowsPermT, false>), gr, dim3(256), 0, st, s->d_layers, layer, B, b_begin, nlive,
                       A, s->key);
  }
  if (phases & 2)
    hipLaunchKernelGGL(k_ffdL_cols<kColsOutT>, gr, dim3(256), 0, st, s->d_layers, layer, A, b_begin, nlive, nullptr,
                       out, out_dtype, theta0, s->key);
  (void)hipGetLastError();
}

}  // namespace sk
