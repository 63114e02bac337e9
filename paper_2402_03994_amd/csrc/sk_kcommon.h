// sk_kcommon.h -- device helpers shared by the Walsh-Hadamard kernels.
#pragma once

#include "sk_internal.h"

namespace sk {

__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

__device__ __forceinline__ void store_out(void *out, int out_dtype, int64_t i, float v) {
  if (out_dtype == SK_BF16)
    ((uint16_t *)out)[i] = f32_to_bf16(v);
  else
    ((float *)out)[i] = v;
}

// Load up to 4 consecutive input elements starting at element e of a vector
// whose valid prefix has `lim` (>= 1) elements from e on; missing -> 0.
template <bool BF16, bool VEC>
__device__ __forceinline__ void load4(const void *x, int64_t e, int64_t lim, float v[4]) {
  if (VEC && lim >= 4) {
    if (BF16) {
      const uint2 u = *(const uint2 *)((const uint16_t *)x + e);
      v[0] = __uint_as_float(u.x << 16);
      v[1] = __uint_as_float(u.x & 0xFFFF0000u);
      v[2] = __uint_as_float(u.y << 16);
      v[3] = __uint_as_float(u.y & 0xFFFF0000u);
    } else {
      const float4 f = *(const float4 *)((const float *)x + e);
      v[0] = f.x;
      v[1] = f.y;
      v[2] = f.z;
      v[3] = f.w;
    }
    return;
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    if (q < lim)
      v[q] = BF16 ? bf16_to_f32(((const uint16_t *)x)[e + q]) : ((const float *)x)[e + q];
    else
      v[q] = 0.0f;
  }
}

// In-place unnormalised radix-2 Walsh-Hadamard transform along the rows of an
// LDS tile s[r << lgcs | c], 2^lgrows rows, 2^lgcs columns.  Ends synchronised.
__device__ __forceinline__ void lds_fwht(float *s, int lgrows, int lgcs) {
  const int npairs = 1 << (lgrows - 1 + lgcs);
  const int cmask = (1 << lgcs) - 1;
  for (int st = 0; st < lgrows; ++st) {
    __syncthreads();
    const int hmask = (1 << st) - 1;
    for (int p = threadIdx.x; p < npairs; p += blockDim.x) {
      const int q = p >> lgcs, c = p & cmask;
      const int r = ((q & ~hmask) << 1) | (q & hmask);
      float *a = s + ((r << lgcs) | c);
      float *b = a + (1 << (st + lgcs));
      const float u = *a, w = *b;
      *a = u + w;
      *b = u - w;
    }
  }
  __syncthreads();
}

// Unnormalised Walsh-Hadamard transform of N values held in registers (the
// stages are expanded at compile time so every index is static).
template <int N, int H>
struct FwhtStage {
  static __device__ __forceinline__ void run(float *v) {
    if constexpr (H < N) {
#pragma clang loop unroll(full)
      for (int i = 0; i < N; i += 2 * H)
#pragma clang loop unroll(full)
        for (int j = i; j < i + H; ++j) {
          const float a = v[j], b = v[j + H];
          v[j] = a + b;
          v[j + H] = a - b;
        }
      FwhtStage<N, 2 * H>::run(v);
    }
  }
};

template <int N>
__device__ __forceinline__ void fwht_regs_t(float *v) {
  FwhtStage<N, 1>::run(v);
}

// LDS tiles in the "p16" layout: one pad word after every 16 floats
// (element i at i + i / 16), so that the register passes below touch 32
// distinct banks per half-wave whichever index bits they hold.
__device__ __forceinline__ int p16(int i) { return i + (i >> 4); }
__host__ __device__ constexpr int p16_floats(int n) { return n + n / 16; }

// One pass of lds_fwht_regs: every thread takes groups of 2^W elements that
// differ in index bits [p, p + W) (the other bits from the group number),
// transforms them in registers and writes them back.
template <int W>
__device__ __forceinline__ void fwht_pass_p16(float *s, int lgn, int p) {
  constexpr int G = 1 << W;
  const int ngroups = 1 << (lgn - W);
  const int lowmask = (1 << p) - 1;
  for (int g = threadIdx.x; g < ngroups; g += blockDim.x) {
    const int base = ((g >> p) << (p + W)) | (g & lowmask);
    float e[G];
#pragma unroll
    for (int m = 0; m < G; ++m) e[m] = s[p16(base + (m << p))];
    fwht_regs_t<G>(e);
#pragma unroll
    for (int m = 0; m < G; ++m) s[p16(base + (m << p))] = e[m];
  }
}

// In-place unnormalised Walsh-Hadamard transform along index bits
// [p0, lgn) of a 2^lgn-element LDS tile in the p16 layout (p0 > 0 leaves the
// low bits as independent columns), four bits per pass held in registers:
// a quarter of the barriers and LDS round trips of the radix-2 lds_fwht.
// Ends synchronised.
__device__ __forceinline__ void lds_fwht_regs(float *s, int lgn, int p0) {
  int p = p0;
  for (; p + 4 <= lgn; p += 4) {
    __syncthreads();
    fwht_pass_p16<4>(s, lgn, p);
  }
  const int rem = lgn - p;
  if (rem > 0) {
    __syncthreads();
    if (rem == 1)
      fwht_pass_p16<1>(s, lgn, p);
    else if (rem == 2)
      fwht_pass_p16<2>(s, lgn, p);
    else
      fwht_pass_p16<3>(s, lgn, p);
  }
  __syncthreads();
}

// 1024-point unnormalised Walsh-Hadamard transform of NV rows spread over a
// 256-thread workgroup.  On entry thread t holds columns 4t .. 4t+3 of every
// row in v[r][0..3]; on exit it holds columns t, t+256, t+512, t+768 in
// v[r][0..3].  Column bits 0-1 are transformed in the thread, bits 2-7 (lane
// bits 0-5) by cross-lane exchanges, bits 8-9 (wave index) after one pass
// through `lds` (NV x 1024 floats).  Ends synchronised.
template <int NV>
__device__ __forceinline__ void fwht1024_rows(float (&v)[NV][4], float *lds) {
  const int tid = threadIdx.x, lane = tid & 63;
#pragma unroll
  for (int r = 0; r < NV; ++r) {
    const float a0 = v[r][0] + v[r][1], a1 = v[r][0] - v[r][1];
    const float a2 = v[r][2] + v[r][3], a3 = v[r][2] - v[r][3];
    v[r][0] = a0 + a2;
    v[r][1] = a1 + a3;
    v[r][2] = a0 - a2;
    v[r][3] = a1 - a3;
  }
#pragma unroll
  for (int sbit = 0; sbit < 6; ++sbit) {
    const int mask = 1 << sbit;
    const bool upper = (lane & mask) != 0;
#pragma unroll
    for (int r = 0; r < NV; ++r)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float o = __shfl_xor(v[r][q], mask, 64);
        v[r][q] = upper ? o - v[r][q] : v[r][q] + o;
      }
  }
  __syncthreads();  // lds may still be read by the caller's previous step
#pragma unroll
  for (int r = 0; r < NV; ++r)
    *(float4 *)(lds + r * 1024 + 4 * tid) = make_float4(v[r][0], v[r][1], v[r][2], v[r][3]);
  __syncthreads();
#pragma unroll
  for (int r = 0; r < NV; ++r) {
    const float b0 = lds[r * 1024 + tid], b1 = lds[r * 1024 + tid + 256];
    const float b2 = lds[r * 1024 + tid + 512], b3 = lds[r * 1024 + tid + 768];
    const float a0 = b0 + b1, a1 = b0 - b1, a2 = b2 + b3, a3 = b2 - b3;
    v[r][0] = a0 + a2;
    v[r][1] = a1 + a3;
    v[r][2] = a0 - a2;
    v[r][3] = a1 - a3;
  }
  __syncthreads();
}


// NV (8 or 16) rows of 1024 floats in LDS: one pad word after every E = 4 NV
// floats and a row stride of 16 (NV = 16) or 32 (NV = 8) banks modulo 32, so
// that both passes of fwht1024_lds touch 32 distinct banks per half-wave.
template <int NV>
struct Lds1024 {
  static_assert(NV == 8 || NV == 16, "8 or 16 rows");
  static constexpr int kLgE = NV == 16 ? 6 : 5;
  static constexpr int kStride = NV == 16 ? 1040 : 1056;
  static constexpr int kFloats = NV * kStride;
  static __device__ __forceinline__ int idx(int row, int l) { return row * kStride + l + (l >> kLgE); }
};

// In-place unnormalised 1024-point Walsh-Hadamard transform of the NV rows of
// an Lds1024<NV> block; 256 threads; every butterfly runs inside a thread.
// Thread (row i = tid / C, c = tid % C), C = 256 / NV, E = 1024 / C values:
// pass 1 holds columns c + C k and transforms column bits log2 C .. 9; pass 2
// holds the E consecutive columns E c .. E c + E - 1 (G = E / C runs of C)
// and transforms bits 0 .. log2 C - 1.  The caller synchronises after
// filling the block; ends synchronised.
template <int NV>
__device__ __forceinline__ void fwht1024_lds_pass2(float *lds) {
  constexpr int C = 256 / NV, E = 1024 / C, G = E / C;
  using L = Lds1024<NV>;
  const int i = threadIdx.x / C, c = threadIdx.x % C;
  // columns E c + m (m < E) sit at (E + 1) c + m
  float *b = lds + i * L::kStride + (E + 1) * c;
  float e[E];
#pragma unroll
  for (int m = 0; m < E; ++m) e[m] = b[m];
#pragma unroll
  for (int g = 0; g < G; ++g) fwht_regs_t<C>(e + g * C);
#pragma unroll
  for (int m = 0; m < E; ++m) b[m] = e[m];
  __syncthreads();
}

// Offset of column c + C k from column c in an Lds1024<NV> row (c < C).
template <int NV>
__device__ __forceinline__ constexpr int lds1024_pass1_off(int k) {
  constexpr int C = 256 / NV;
  return C * k + ((C * k) >> Lds1024<NV>::kLgE);
}

template <int NV>
__device__ __forceinline__ void fwht1024_lds(float *lds) {
  constexpr int C = 256 / NV, E = 1024 / C;
  using L = Lds1024<NV>;
  static_assert(E == (1 << L::kLgE), "pad period");
  const int i = threadIdx.x / C, c = threadIdx.x % C;
  float *b = lds + i * L::kStride + c;
  float e[E];
#pragma unroll
  for (int k = 0; k < E; ++k) e[k] = b[lds1024_pass1_off<NV>(k)];
  fwht_regs_t<E>(e);
#pragma unroll
  for (int k = 0; k < E; ++k) b[lds1024_pass1_off<NV>(k)] = e[k];
  __syncthreads();
  fwht1024_lds_pass2<NV>(lds);
}

// Same transform with the first pass fed from registers: e[k] holds column
// c + C k of row i (i = tid / C, c = tid % C), e.g. straight from global
// memory.  The block needs no synchronisation on entry beyond the caller's
// own (its previous readers must be done); ends synchronised.
template <int NV>
__device__ __forceinline__ void fwht1024_lds_regs(float *lds, float (&e)[1024 * NV / 256]) {
  constexpr int C = 256 / NV;
  using L = Lds1024<NV>;
  const int i = threadIdx.x / C, c = threadIdx.x % C;
  fwht_regs_t<1024 * NV / 256>(e);
  float *b = lds + i * L::kStride + c;
#pragma unroll
  for (int k = 0; k < 1024 * NV / 256; ++k) b[lds1024_pass1_off<NV>(k)] = e[k];
  __syncthreads();
  fwht1024_lds_pass2<NV>(lds);
}

// LDS block of 16 rows of 1024 for the row kernels: one pad word per 64 floats
// and a row stride of 2 banks modulo 32.  The transform runs with the row
// index fastest (thread (i = tid % 16, c = tid / 16)): pass 1 holds columns
// c + 16 k, pass 2 the 64 consecutive columns 64 c .. 64 c + 63, so in both
// passes a half-wave touches 32 distinct banks, and after pass 2 the 16 lanes
// of a column write its 16 consecutive p (64 bytes) straight from registers.
struct Lds1024R {
  static constexpr int kStride = 1058;
  static constexpr int kFloats = 16 * kStride;
  static __device__ __forceinline__ int idx(int row, int l) { return row * kStride + l + (l >> 6); }
};


// Unnormalised 1024-point transform of the 16 rows of an Lds1024R block that
// the caller has filled and synchronised.  On return thread (ri = tid % 16,
// rc = tid / 16) holds columns 64 rc + m of row ri in e[m]; the block holds
// pass-1 data and may be refilled after the caller's next barrier.
__device__ __forceinline__ void fwht1024_rows16_r(float *s, float (&e)[64]) {
  using L = Lds1024R;
  const int ri = threadIdx.x & 15, rc = threadIdx.x >> 4;
  {
    float *b = s + ri * L::kStride + rc;
#pragma unroll
    for (int k = 0; k < 64; ++k) e[k] = b[16 * k + (k >> 2)];
    fwht_regs_t<64>(e);
#pragma unroll
    for (int k = 0; k < 64; ++k) b[16 * k + (k >> 2)] = e[k];
  }
  __syncthreads();
  const float *b = s + ri * L::kStride + 65 * rc;
#pragma unroll
  for (int m = 0; m < 64; ++m) e[m] = b[m];
#pragma unroll
  for (int g = 0; g < 4; ++g) fwht_regs_t<16>(e + 16 * g);
}


// Row-fastest 32-row block for 1024-thread workgroups: one pad word per 32
// floats and an odd row stride, so that both passes of fwht1024_rows32 touch
// 32 distinct banks in every half-wave (the 32 rows of one column group).
struct Lds1024R32 {
  static constexpr int kRows = 32;
  static constexpr int kStride = 1057;  // 1056 used
  static constexpr int kFloats = kRows * kStride;
  static __device__ __forceinline__ int idx(int row, int l) { return row * kStride + l + (l >> 5); }
};

// Unnormalised 1024-point transform of the 32 rows of an Lds1024R32 block
// that the caller has filled and synchronised, by 1024 threads.  Pass 1:
// thread (ri = tid % 32, rc = tid / 32) transforms columns rc + 32 k (the high
// five column bits); pass 2: columns 32 rc + m (the low five).  On return e[m]
// holds column 32 rc + m of row ri, so the 32 lanes of a column hold its 32
// consecutive rows; the block may be refilled after the caller's next barrier.
__device__ __forceinline__ void fwht1024_rows32(float *s, float (&e)[32]) {
  using L = Lds1024R32;
  const int ri = threadIdx.x & 31, rc = threadIdx.x >> 5;
  {
    float *b = s + ri * L::kStride + rc;  // column rc + 32 k sits at rc + 33 k
#pragma unroll
    for (int k = 0; k < 32; ++k) e[k] = b[33 * k];
    fwht_regs_t<32>(e);
#pragma unroll
    for (int k = 0; k < 32; ++k) b[33 * k] = e[k];
  }
  __syncthreads();
  const float *b = s + ri * L::kStride + 33 * rc;  // column 32 rc + m sits at 33 rc + m
#pragma unroll
  for (int m = 0; m < 32; ++m) e[m] = b[m];
  fwht_regs_t<32>(e);
}

// Raw buffer resource over [base, base + bytes): loads past the end return
// zero, stores past the end are dropped (offsets are bytes, unsigned 32-bit).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}

// Cache-policy operand of the buffer load/store builtins for data touched
// once: the non-temporal (nt) bit.
constexpr int kNt = 2;

// 16-byte global load with the non-temporal hint, for inputs a kernel reads
// once where one wave instruction covers whole 128-byte lines (streamed
// gradients): they then displace less of the caches that hold the data a
// kernel or its successor reads again.  Where the lanes of an instruction
// cover only parts of lines that later instructions complete, the hint costs
// re-fetches instead (measured 40% slower on the QK contraction).
__device__ __forceinline__ uint4 ld_nt16(const void *p) {
  typedef unsigned int u4v __attribute__((ext_vector_type(4)));
  const u4v r = __builtin_nontemporal_load((const u4v *)p);
  return make_uint4(r.x, r.y, r.z, r.w);
}

}  // namespace sk
