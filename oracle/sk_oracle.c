/*
 * sk_oracle.c -- fp64 CPU oracle for the structured sketches of
 * "Efficient Sketches for Training Data Attribution and Studying the Loss
 * Landscape" (Schioppa, NeurIPS 2024, arXiv 2402.03994).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  The product (the HIP
 * library under paper_2402_03994_amd/) never links, loads or calls it, and the
 * two share no code: this file re-implements the random streams from their
 * published definitions (Philox4x32-10, Box-Muller, a Feistel network) and
 * applies every sketch as the literal chain of dense-definition operators, in
 * double precision, with a textbook in-place Walsh-Hadamard transform.
 *
 * Operators (paper notation, all per parameter tensor "layer" l, N = N'_l):
 *   H_N   normalised Sylvester Walsh-Hadamard matrix, natural order
 *         (Appendix "Definition of the Walsh-Hadamard transform").
 *   B     diag of Rademacher signs; G diag of N(0,1) entries.
 *   R_D   restriction to the first D coordinates (Sec. 3, eq. bami).
 *   pi    digit-wise permutation over the Kronecker factor shapes of N
 *         (Sec. 3 "Removing the lookup bottleneck"; factor shapes follow the
 *         paper's Kronecker shape rule with a maximal block of 1024).
 *   FJL   y = sqrt(N/D) G_s H_N B x                    (eq. ailon_chazelle)
 *   FFD   y = sum_b B_b H_D Pi_b^T G_b H_D x_b          (transpose of eq. fastfood,
 *         sigma_F = 1 as required in the proof of Thm. fastfood_bad_inputs)
 *   AFFD  y = R_D(sqrt(N/D) H^{pi2}_N G H^{pi1}_N B x)  (eq. bami)
 *   AFJL  y = R_D(sqrt(N/D) G H^{pi1}_N B x)            (eq. frikadel)
 *   QK    Y = A X B^T, per weight matrix                (eq. straight with two
 *         Kronecker factors, contraction as in eq. qk_proof_tensor_dec)
 *   Transposes are the exact adjoints of the forward maps.
 *
 * Readings where the paper is silent (padding, sigma_F, G_s density, the random
 * streams) are listed in the repository's design notes.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { K_FJL = 0, K_FFD = 1, K_AFFD = 2, K_AFJL = 3, K_QK = 4 };
enum { T_F32 = 0, T_BF16 = 1 };

/* Stream tags: the fourth Philox counter word. */
enum {
  ST_SIGN = 1,  /* B: Rademacher signs                        */
  ST_GAUSS = 2, /* G: N(0,1) diagonal                          */
  ST_INDEX = 3, /* FJL sample positions                        */
  ST_FFDPERM = 4, /* FFD block permutations Pi_b                */
  ST_PI1 = 5,   /* AFFD/AFJL digit permutations before 1st H   */
  ST_PI2 = 6,   /* AFFD digit permutations after 2nd H         */
  ST_QKA = 7,   /* QK left factor A                            */
  ST_QKB = 8    /* QK right factor B                           */
};

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as   */
/* easy as 1, 2, 3", SC'11): 10 rounds of the S-box with multipliers         */
/* 0xD2511F53 / 0xCD9E8D57 and Weyl key increments 0x9E3779B9 / 0xBB67AE85.  */
/* ------------------------------------------------------------------------ */
void orc_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
  uint32_t k0 = key_in[0], k1 = key_in[1];
  for (int round = 0; round < 10; ++round) {
    uint64_t p0 = (uint64_t)0xD2511F53u * c0;
    uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t n0 = hi1 ^ c1 ^ k0;
    uint32_t n1 = lo1;
    uint32_t n2 = hi0 ^ c3 ^ k1;
    uint32_t n3 = lo0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* One Philox block for (seed, layer, stream) at 64-bit block counter `ctr`. */
static void block(uint64_t seed, uint32_t layer, uint32_t stream, uint64_t ctr, uint32_t w[4]) {
  uint32_t c[4] = {(uint32_t)ctr, (uint32_t)(ctr >> 32), layer, stream};
  uint32_t k[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  orc_philox4x32_10(c, k, w);
}

/* Rademacher sign of coordinate j: bit (j mod 32) of word ((j/32) mod 4) of
 * block j/128; bit 1 means -1. */
int orc_sign(uint64_t seed, uint32_t layer, uint64_t j) {
  uint32_t w[4];
  block(seed, layer, ST_SIGN, j >> 7, w);
  uint32_t bit = (w[(j >> 5) & 3] >> (j & 31)) & 1u;
  return bit ? -1 : 1;
}

/* Standard normal number j of a stream, by the Box-Muller transform on the
 * two 24-bit uniforms of word pair (j/2 mod 2) of block j/4:
 *   u1 = (top24(wa) + 1) / 2^24 in (0,1],  u2 = top24(wb) / 2^24 in [0,1),
 *   g  = sqrt(-2 ln u1) * (cos 2 pi u2 if j even else sin 2 pi u2). */
double orc_gauss(uint64_t seed, uint32_t layer, uint32_t stream, uint64_t j) {
  uint32_t w[4];
  block(seed, layer, stream, j >> 2, w);
  uint32_t wa = w[((j >> 1) & 1) * 2], wb = w[((j >> 1) & 1) * 2 + 1];
  double u1 = ((double)(wa >> 8) + 1.0) * (1.0 / 16777216.0);
  double u2 = (double)(wb >> 8) * (1.0 / 16777216.0);
  double r = sqrt(-2.0 * log(u1));
  double t = 2.0 * M_PI * u2;
  return (j & 1) ? r * sin(t) : r * cos(t);
}

/* FJL sample position i: word (i mod 4) of block i/4, masked to [0, Np). */
/* FJL sample position i in [0, np): word i mod 4 of block i / 4, masked to
 * np - 1 (np a power of two of at most 2^32, so the mask is exactly uniform). */
uint64_t orc_index(uint64_t seed, uint32_t layer, uint64_t i, uint64_t np) {
  uint32_t w[4];
  block(seed, layer, ST_INDEX, i >> 2, w);
  return (uint64_t)w[i & 3] & (np - 1);
}

/* 32-bit finaliser used as the Feistel round function. */
static uint32_t mix32(uint32_t h) {
  h ^= h >> 16; h *= 0x85EBCA6Bu;
  h ^= h >> 13; h *= 0xC2B2AE35u;
  h ^= h >> 16;
  return h;
}

/* Keyed permutation of [0, 2^w): an 8-round alternating Feistel network on
 * the split (high ceil(w/2) bits, low floor(w/2) bits).  Round keys are the
 * 8 words of blocks 2*pid and 2*pid+1 of the stream.  Even rounds update the
 * high part from the low part, odd rounds the low part from the high part. */
static void perm_keys(uint64_t seed, uint32_t layer, uint32_t stream, uint32_t pid, uint32_t k[8]) {
  block(seed, layer, stream, 2ull * pid, k);
  block(seed, layer, stream, 2ull * pid + 1, k + 4);
}

uint32_t orc_perm(uint64_t seed, uint32_t layer, uint32_t stream, uint32_t pid, uint32_t w, uint32_t x) {
  if (w == 0) return 0;
  uint32_t k[8];
  perm_keys(seed, layer, stream, pid, k);
  uint32_t wl = w / 2, wh = w - wl;
  uint32_t ml = (1u << wl) - 1u, mh = (1u << wh) - 1u;
  uint32_t hi = x >> wl, lo = x & ml;
  for (int r = 0; r < 8; ++r) {
    if ((r & 1) == 0) hi ^= mix32(lo ^ k[r]) & mh;
    else lo ^= mix32(hi ^ k[r]) & ml;
  }
  return (hi << wl) | lo;
}

uint32_t orc_perm_inv(uint64_t seed, uint32_t layer, uint32_t stream, uint32_t pid, uint32_t w, uint32_t y) {
  if (w == 0) return 0;
  uint32_t k[8];
  perm_keys(seed, layer, stream, pid, k);
  uint32_t wl = w / 2, wh = w - wl;
  uint32_t ml = (1u << wl) - 1u, mh = (1u << wh) - 1u;
  uint32_t hi = y >> wl, lo = y & ml;
  for (int r = 7; r >= 0; --r) {
    if ((r & 1) == 0) hi ^= mix32(lo ^ k[r]) & mh;
    else lo ^= mix32(hi ^ k[r]) & ml;
  }
  return (hi << wl) | lo;
}

/* Kronecker factor shapes of n = 2^L (Sec. 3, "Removing the lookup
 * bottleneck": H_{AB} = H_A (x) H_B with factors of at most 1024 columns).
 * The fewest factors of at most 2^10 whose product is n: K = ceil(L / 10);
 * every factor but the most significant is 1024, the most significant takes
 * what is left, 2^(L - 10 (K - 1)).  dims[0] is the most significant factor
 * (row-major digit order).  n = 1 has no factor.  Returns K. */
int orc_kron_shapes(uint64_t n, uint64_t dims[8]) {
  int L = 0;
  while ((1ull << L) < n) ++L;
  const int K = (L + 9) / 10;
  for (int k = 0; k < K; ++k) dims[k] = 1024;
  if (K > 0) dims[0] = 1ull << (L - 10 * (K - 1));
  return K;
}

/* Normalised Walsh-Hadamard transform in place: the textbook radix-2 butterfly
 * over every bit, then a single scale by n^{-1/2}. */
void orc_fwht(double *v, uint64_t n) {
  for (uint64_t h = 1; h < n; h <<= 1)
    for (uint64_t i = 0; i < n; i += 2 * h)
      for (uint64_t j = i; j < i + h; ++j) {
        double a = v[j], b = v[j + h];
        v[j] = a + b;
        v[j + h] = a - b;
      }
  double s = 1.0 / sqrt((double)n);
  for (uint64_t j = 0; j < n; ++j) v[j] *= s;
}

static uint64_t next_pow2(uint64_t v) {
  uint64_t p = 1;
  while (p < v) p <<= 1;
  return p;
}

/* Padded length of a layer: the smallest power of two >= max(n, D). */
uint64_t orc_padded(uint64_t n, uint64_t d) { return next_pow2(n > d ? n : d); }

static int log2u(uint64_t v) {
  int l = 0;
  while ((1ull << l) < v) ++l;
  return l;
}

/* Digit permutation tables for stream `st` of layer `layer` over the factor
 * shapes of np: table k holds pi_k over [0, dims[k]). */
typedef struct {
  int K;
  uint64_t dims[8];
  uint64_t stride[8];
  uint32_t *tab[8];
} digit_perm;

static void dp_init(digit_perm *p, uint64_t seed, uint32_t layer, uint32_t st, uint64_t np) {
  p->K = orc_kron_shapes(np, p->dims);
  uint64_t s = 1;
  for (int k = p->K - 1; k >= 0; --k) {
    p->stride[k] = s;
    s *= p->dims[k];
  }
  for (int k = 0; k < p->K; ++k) {
    uint32_t w = (uint32_t)log2u(p->dims[k]);
    p->tab[k] = (uint32_t *)malloc(sizeof(uint32_t) * p->dims[k]);
    for (uint32_t x = 0; x < p->dims[k]; ++x) p->tab[k][x] = orc_perm(seed, layer, st, (uint32_t)k, w, x);
  }
}

static void dp_free(digit_perm *p) {
  for (int k = 0; k < p->K; ++k) free(p->tab[k]);
}

/* pi(i): apply pi_k to digit k of i (digit 0 most significant). */
static uint64_t dp_apply(const digit_perm *p, uint64_t i) {
  uint64_t r = 0;
  for (int k = 0; k < p->K; ++k) {
    uint64_t d = (i / p->stride[k]) % p->dims[k];
    r += (uint64_t)p->tab[k][d] * p->stride[k];
  }
  return r;
}

/* Full digit permutation of length np as a table (used by the dense pins). */
void orc_digit_perm_table(uint64_t seed, uint32_t layer, uint32_t stream, uint64_t np, uint64_t *out) {
  digit_perm p;
  dp_init(&p, seed, layer, stream, np);
  for (uint64_t i = 0; i < np; ++i) out[i] = dp_apply(&p, i);
  dp_free(&p);
}

static double load_elem(const void *x, int dtype, uint64_t i) {
  if (dtype == T_BF16) {
    uint32_t bits = (uint32_t)((const uint16_t *)x)[i] << 16;
    float f;
    memcpy(&f, &bits, 4);
    return (double)f;
  }
  return (double)((const float *)x)[i];
}

/* fp64 -> fp32 (round to nearest even by the C conversion) -> bf16 (round to
 * nearest even on the fp32 bit pattern) -> back to double. */
double orc_round_bf16(double v) {
  float f = (float)v;
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  u &= 0xFFFF0000u;
  memcpy(&f, &u, 4);
  return (double)f;
}

/* ------------------------------------------------------------------------ */
/* Forward sketches of one layer, one vector: y[0..D) += S_l x.             */
/* ------------------------------------------------------------------------ */

/* w = B x, zero-padded to np. */
static void signed_padded(double *w, const void *x, int dtype, uint64_t n, uint64_t np,
                          uint64_t seed, uint32_t layer) {
  for (uint64_t j = 0; j < np; ++j) w[j] = 0.0;
  for (uint64_t j = 0; j < n; ++j) w[j] = orc_sign(seed, layer, j) * load_elem(x, dtype, j);
}

static void fjl_fwd(const void *x, int dtype, uint64_t n, uint64_t d, uint64_t seed, uint32_t layer,
                    double *y, double *w) {
  uint64_t np = orc_padded(n, d);
  signed_padded(w, x, dtype, n, np, seed, layer);
  orc_fwht(w, np);
  double sc = sqrt((double)np / (double)d);
  for (uint64_t i = 0; i < d; ++i)
    y[i] += sc * orc_gauss(seed, layer, ST_GAUSS, i) * w[orc_index(seed, layer, i, np)];
}

static void afjl_affd_fwd(int kind, const void *x, int dtype, uint64_t n, uint64_t d, uint64_t seed,
                          uint32_t layer, double *y, double *w) {
  uint64_t np = orc_padded(n, d);
  digit_perm p1;
  dp_init(&p1, seed, layer, ST_PI1, np);
  /* Scatter_pi1 B x: w[pi1(j)] = b_j x_j */
  for (uint64_t j = 0; j < np; ++j) w[j] = 0.0;
  for (uint64_t j = 0; j < n; ++j) w[dp_apply(&p1, j)] = orc_sign(seed, layer, j) * load_elem(x, dtype, j);
  dp_free(&p1);
  orc_fwht(w, np);
  double sc = sqrt((double)np / (double)d);
  if (kind == K_AFJL) {
    for (uint64_t c = 0; c < d; ++c) y[c] += sc * orc_gauss(seed, layer, ST_GAUSS, c) * w[c];
    return;
  }
  for (uint64_t j = 0; j < np; ++j) w[j] *= orc_gauss(seed, layer, ST_GAUSS, j);
  orc_fwht(w, np);
  digit_perm p2;
  dp_init(&p2, seed, layer, ST_PI2, np);
  for (uint64_t c = 0; c < d; ++c) y[c] += sc * w[dp_apply(&p2, c)];
  dp_free(&p2);
}

/* FFD block b of the sketch: B_b H_D Pi_b^T G_b H_D x_b, where (Pi v)_i =
 * v_{pi_b(i)}, so (Pi^T v)_{pi_b(k)} = v_k.  Block-local coordinate i of
 * block b is global coordinate b*D + i for the sign and Gaussian streams. */
static void ffd_fwd(const void *x, int dtype, uint64_t n, uint64_t d, uint64_t seed, uint32_t layer,
                    double *y, double *v, double *u) {
  uint64_t np = orc_padded(n, d);
  uint32_t wd = (uint32_t)log2u(d);
  for (uint64_t b = 0; b < np / d; ++b) {
    for (uint64_t i = 0; i < d; ++i) {
      uint64_t j = b * d + i;
      v[i] = j < n ? load_elem(x, dtype, j) : 0.0;
    }
    orc_fwht(v, d);
    for (uint64_t i = 0; i < d; ++i) v[i] *= orc_gauss(seed, layer, ST_GAUSS, b * d + i);
    for (uint64_t k = 0; k < d; ++k) u[orc_perm(seed, layer, ST_FFDPERM, (uint32_t)b, wd, (uint32_t)k)] = v[k];
    orc_fwht(u, d);
    for (uint64_t i = 0; i < d; ++i) y[i] += orc_sign(seed, layer, b * d + i) * u[i];
  }
}

/* QK factors: A is dA x m with entries N(0,1/dA), B is dB x n with entries
 * N(0,1/dB), both row-major over their own Gaussian streams.  With
 * `bf16` set, each entry is rounded through fp32 to bf16. */
static void qk_factors(uint64_t seed, uint32_t layer, uint64_t m, uint64_t n, uint64_t da, uint64_t db,
                       int bf16, double *A, double *B) {
  double sa = 1.0 / sqrt((double)da), sb = 1.0 / sqrt((double)db);
  for (uint64_t i = 0; i < da * m; ++i) {
    double v = orc_gauss(seed, layer, ST_QKA, i) * sa;
    A[i] = bf16 ? orc_round_bf16(v) : v;
  }
  for (uint64_t i = 0; i < db * n; ++i) {
    double v = orc_gauss(seed, layer, ST_QKB, i) * sb;
    B[i] = bf16 ? orc_round_bf16(v) : v;
  }
}

/* Y = A X B^T written row-major into y[0 .. dA*dB). */
static void qk_fwd(const void *x, int dtype, uint64_t m, uint64_t n, uint64_t da, uint64_t db,
                   const double *A, const double *B, double *y) {
  double *t = (double *)calloc(m * db, sizeof(double)); /* T = X B^T, m x dB */
  for (uint64_t i = 0; i < m; ++i)
    for (uint64_t c = 0; c < db; ++c) {
      double s = 0.0;
      for (uint64_t j = 0; j < n; ++j) s += load_elem(x, dtype, i * n + j) * B[c * n + j];
      t[i * db + c] = s;
    }
  for (uint64_t a = 0; a < da; ++a)
    for (uint64_t c = 0; c < db; ++c) {
      double s = 0.0;
      for (uint64_t i = 0; i < m; ++i) s += A[a * m + i] * t[i * db + c];
      y[a * db + c] = s;
    }
  free(t);
}

/* ------------------------------------------------------------------------ */
/* Transposes of one layer, one vector: out[0..n) = S_l^T z.                */
/* ------------------------------------------------------------------------ */
static void fjl_T(const double *z, uint64_t n, uint64_t d, uint64_t seed, uint32_t layer, double *out,
                  double *w) {
  uint64_t np = orc_padded(n, d);
  for (uint64_t j = 0; j < np; ++j) w[j] = 0.0;
  for (uint64_t i = 0; i < d; ++i) w[orc_index(seed, layer, i, np)] += orc_gauss(seed, layer, ST_GAUSS, i) * z[i];
  orc_fwht(w, np);
  double sc = sqrt((double)np / (double)d);
  for (uint64_t j = 0; j < n; ++j) out[j] = sc * orc_sign(seed, layer, j) * w[j];
}

static void afjl_affd_T(int kind, const double *z, uint64_t n, uint64_t d, uint64_t seed, uint32_t layer,
                        double *out, double *w) {
  uint64_t np = orc_padded(n, d);
  for (uint64_t j = 0; j < np; ++j) w[j] = 0.0;
  if (kind == K_AFJL) {
    for (uint64_t c = 0; c < d; ++c) w[c] = orc_gauss(seed, layer, ST_GAUSS, c) * z[c];
  } else {
    digit_perm p2;
    dp_init(&p2, seed, layer, ST_PI2, np);
    for (uint64_t c = 0; c < d; ++c) w[dp_apply(&p2, c)] = z[c]; /* Scatter_pi2 R_D^T z */
    dp_free(&p2);
    orc_fwht(w, np);
    for (uint64_t j = 0; j < np; ++j) w[j] *= orc_gauss(seed, layer, ST_GAUSS, j);
  }
  orc_fwht(w, np);
  digit_perm p1;
  dp_init(&p1, seed, layer, ST_PI1, np);
  double sc = sqrt((double)np / (double)d);
  for (uint64_t j = 0; j < n; ++j) out[j] = sc * orc_sign(seed, layer, j) * w[dp_apply(&p1, j)]; /* B Gather_pi1 */
  dp_free(&p1);
}

/* FFD feature map, block b: H_D G_b Pi_b H_D B_b z (eq. fastfood, sigma_F = 1). */
static void ffd_T(const double *z, uint64_t n, uint64_t d, uint64_t seed, uint32_t layer, double *out,
                  double *v, double *u) {
  uint64_t np = orc_padded(n, d);
  uint32_t wd = (uint32_t)log2u(d);
  for (uint64_t b = 0; b < np / d; ++b) {
    if (b * d >= n) break;
    for (uint64_t i = 0; i < d; ++i) v[i] = orc_sign(seed, layer, b * d + i) * z[i];
    orc_fwht(v, d);
    for (uint64_t i = 0; i < d; ++i) u[i] = v[orc_perm(seed, layer, ST_FFDPERM, (uint32_t)b, wd, (uint32_t)i)];
    for (uint64_t i = 0; i < d; ++i) u[i] *= orc_gauss(seed, layer, ST_GAUSS, b * d + i);
    orc_fwht(u, d);
    for (uint64_t i = 0; i < d && b * d + i < n; ++i) out[b * d + i] = u[i];
  }
}

/* X' = A^T Z B, m x n, with Z the dA x dB block of z. */
static void qk_T(const double *z, uint64_t m, uint64_t n, uint64_t da, uint64_t db, const double *A,
                 const double *B, double *out) {
  double *t = (double *)calloc(m * db, sizeof(double)); /* A^T Z, m x dB */
  for (uint64_t i = 0; i < m; ++i)
    for (uint64_t c = 0; c < db; ++c) {
      double s = 0.0;
      for (uint64_t a = 0; a < da; ++a) s += A[a * m + i] * z[a * db + c];
      t[i * db + c] = s;
    }
  for (uint64_t i = 0; i < m; ++i)
    for (uint64_t j = 0; j < n; ++j) {
      double s = 0.0;
      for (uint64_t c = 0; c < db; ++c) s += t[i * db + c] * B[c * n + j];
      out[i * n + j] = s;
    }
  free(t);
}

/* ------------------------------------------------------------------------ */
/* Batched multi-layer drivers.                                             */
/*   layers l = 0..n_layers-1 carry RNG layer ids layer0 + l.               */
/*   x[l] is [batch, rows[l]*cols[l]] row-major in `dtype`.                 */
/*   y is [batch, D] (FWHT kinds: sum over layers; QK: concatenation of the */
/*   dA*dB blocks in layer order, starting at column qk_offset0).           */
/* Work items (layer, row) run in parallel; per-row partial sums are added  */
/* in layer order so the result does not depend on the thread count.        */
/* ------------------------------------------------------------------------ */
/* The FJL position stream is defined for padded lengths up to 2^32. */
static int fjl_sizes_ok(int n_layers, const int64_t *rows, const int64_t *cols, int64_t d) {
  for (int l = 0; l < n_layers; ++l)
    if (orc_padded((uint64_t)rows[l] * (uint64_t)cols[l], (uint64_t)d) > (1ull << 32)) return 0;
  return 1;
}

int orc_apply(int kind, int layer0, int n_layers, const int64_t *rows, const int64_t *cols, const int32_t *da,
              const int32_t *db, int64_t d, uint64_t seed, int64_t batch, int dtype, const void *const *x,
              double *y, int nthreads, int qk_bf16) {
  if (d < 1 || batch < 1 || n_layers < 1) return -1;
  if (kind == K_QK) {
    int64_t tot = 0;
    for (int l = 0; l < n_layers; ++l) tot += (int64_t)da[l] * db[l];
    if (tot != d) return -1;
  }
  if (kind == K_FJL && !fjl_sizes_ok(n_layers, rows, cols, d)) return -1;
  int64_t nitems = (int64_t)n_layers * batch;
  double **part = (double **)calloc((size_t)nitems, sizeof(double *));
  int64_t *qoff = (int64_t *)calloc((size_t)n_layers + 1, sizeof(int64_t));
  for (int l = 0; l < n_layers; ++l) qoff[l + 1] = qoff[l] + (kind == K_QK ? (int64_t)da[l] * db[l] : 0);
  int err = 0;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
  for (int64_t it = 0; it < nitems; ++it) {
    int l = (int)(it / batch);
    int64_t r = it % batch;
    uint64_t n = (uint64_t)rows[l] * (uint64_t)cols[l];
    uint32_t lid = (uint32_t)(layer0 + l);
    const void *xr = (dtype == T_BF16) ? (const void *)((const uint16_t *)x[l] + r * n)
                                       : (const void *)((const float *)x[l] + r * n);
    if (kind == K_QK) {
      uint64_t m = (uint64_t)rows[l], nc = (uint64_t)cols[l];
      double *A = (double *)malloc(sizeof(double) * da[l] * m);
      double *B = (double *)malloc(sizeof(double) * db[l] * nc);
      double *yy = (double *)calloc((size_t)da[l] * db[l], sizeof(double));
      qk_factors(seed, lid, m, nc, (uint64_t)da[l], (uint64_t)db[l], qk_bf16, A, B);
      qk_fwd(xr, dtype, m, nc, (uint64_t)da[l], (uint64_t)db[l], A, B, yy);
      free(A);
      free(B);
      part[it] = yy;
      continue;
    }
    uint64_t np = orc_padded(n, (uint64_t)d);
    double *yy = (double *)calloc((size_t)d, sizeof(double));
    if (kind == K_FFD) {
      double *v = (double *)malloc(sizeof(double) * d), *u = (double *)malloc(sizeof(double) * d);
      ffd_fwd(xr, dtype, n, (uint64_t)d, seed, lid, yy, v, u);
      free(v);
      free(u);
    } else {
      double *w = (double *)malloc(sizeof(double) * np);
      if (!w) {
        err = -2;
        part[it] = yy;
        continue;
      }
      if (kind == K_FJL) fjl_fwd(xr, dtype, n, (uint64_t)d, seed, lid, yy, w);
      else afjl_affd_fwd(kind, xr, dtype, n, (uint64_t)d, seed, lid, yy, w);
      free(w);
    }
    part[it] = yy;
  }
  for (int64_t r = 0; r < batch; ++r) {
    double *yr = y + r * d;
    for (int64_t c = 0; c < d; ++c) yr[c] = 0.0;
    for (int l = 0; l < n_layers; ++l) {
      double *p = part[(int64_t)l * batch + r];
      if (kind == K_QK) {
        for (int64_t c = 0; c < (int64_t)da[l] * db[l]; ++c) yr[qoff[l] + c] = p[c];
      } else {
        for (int64_t c = 0; c < d; ++c) yr[c] += p[c];
      }
    }
  }
  for (int64_t it = 0; it < nitems; ++it) free(part[it]);
  free(part);
  free(qoff);
  return err;
}

/* out[l] is [batch, rows[l]*cols[l]] fp64; z is [batch, D] fp64 (for QK the
 * layer's block starts at the running sum of dA*dB). */
int orc_apply_T(int kind, int layer0, int n_layers, const int64_t *rows, const int64_t *cols, const int32_t *da,
                const int32_t *db, int64_t d, uint64_t seed, int64_t batch, const double *z, double *const *out,
                int nthreads, int qk_bf16) {
  if (d < 1 || batch < 1 || n_layers < 1) return -1;
  if (kind == K_FJL && !fjl_sizes_ok(n_layers, rows, cols, d)) return -1;
  int64_t *qoff = (int64_t *)calloc((size_t)n_layers + 1, sizeof(int64_t));
  for (int l = 0; l < n_layers; ++l) qoff[l + 1] = qoff[l] + (kind == K_QK ? (int64_t)da[l] * db[l] : 0);
  int64_t nitems = (int64_t)n_layers * batch;
  int err = 0;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
  for (int64_t it = 0; it < nitems; ++it) {
    int l = (int)(it / batch);
    int64_t r = it % batch;
    uint64_t n = (uint64_t)rows[l] * (uint64_t)cols[l];
    uint32_t lid = (uint32_t)(layer0 + l);
    const double *zr = z + r * d;
    double *o = out[l] + r * n;
    if (kind == K_QK) {
      uint64_t m = (uint64_t)rows[l], nc = (uint64_t)cols[l];
      double *A = (double *)malloc(sizeof(double) * da[l] * m);
      double *B = (double *)malloc(sizeof(double) * db[l] * nc);
      qk_factors(seed, lid, m, nc, (uint64_t)da[l], (uint64_t)db[l], qk_bf16, A, B);
      qk_T(zr + qoff[l], m, nc, (uint64_t)da[l], (uint64_t)db[l], A, B, o);
      free(A);
      free(B);
      continue;
    }
    uint64_t np = orc_padded(n, (uint64_t)d);
    if (kind == K_FFD) {
      double *v = (double *)malloc(sizeof(double) * d), *u = (double *)malloc(sizeof(double) * d);
      ffd_T(zr, n, (uint64_t)d, seed, lid, o, v, u);
      free(v);
      free(u);
      continue;
    }
    double *w = (double *)malloc(sizeof(double) * np);
    if (!w) {
      err = -2;
      continue;
    }
    if (kind == K_FJL) fjl_T(zr, n, (uint64_t)d, seed, lid, o, w);
    else afjl_affd_T(kind, zr, n, (uint64_t)d, seed, lid, o, w);
    free(w);
  }
  free(qoff);
  return err;
}

/* Ingredient export for the dense pins and for the RNG tests. */
void orc_signs(uint64_t seed, uint32_t layer, uint64_t start, uint64_t count, int8_t *out) {
  for (uint64_t i = 0; i < count; ++i) out[i] = (int8_t)orc_sign(seed, layer, start + i);
}
void orc_gauss_range(uint64_t seed, uint32_t layer, uint32_t stream, uint64_t start, uint64_t count, double *out) {
  for (uint64_t i = 0; i < count; ++i) out[i] = orc_gauss(seed, layer, stream, start + i);
}
void orc_index_range(uint64_t seed, uint32_t layer, uint64_t start, uint64_t count, uint64_t np, uint64_t *out) {
  for (uint64_t i = 0; i < count; ++i) out[i] = orc_index(seed, layer, start + i, np);
}
void orc_perm_table(uint64_t seed, uint32_t layer, uint32_t stream, uint32_t pid, uint32_t w, uint32_t *out) {
  for (uint32_t x = 0; x < (1u << w); ++x) out[x] = orc_perm(seed, layer, stream, pid, w, x);
}

/* ------------------------------------------------------------------------ */
/* Synthetic Hessian for the sketched HVP operator v -> S HVP(S^T v) of      */
/* Sec. 2 (sketching the Hessian-vector product) and Sec. 4 ("Scaling        */
/* eigenvalue estimation").  It stands in for the model's HVP:               */
/*   H = shift I + sum_{j < r} lambda_j v_j v_j^T                            */
/* on the concatenated parameters (N_tot = sum of the layers' element        */
/* counts), v_j = s_j / sqrt(N_tot), s_j a Rademacher vector.  Coordinate e  */
/* of layer l takes, for vector j, bit (e mod 32) of word ((e / 32) mod 4)   */
/* of the Philox block with counter (e / 128, (l << 6) | j, ST_HVP); bit 1   */
/* means -1.  The scaling by lambda_j / N_tot is left to the caller.         */
/* ------------------------------------------------------------------------ */
enum { ST_HVP = 10 };

int orc_hvp_sign(uint64_t seed, uint32_t layer, uint32_t j, uint64_t e) {
  uint32_t w[4];
  block(seed, (layer << 6) | j, ST_HVP, e >> 7, w);
  return ((w[(e >> 5) & 3] >> (e & 31)) & 1u) ? -1 : 1;
}

void orc_hvp_signs(uint64_t seed, uint32_t layer, uint32_t j, uint64_t start, uint64_t count, int8_t *out) {
  for (uint64_t i = 0; i < count; ++i) out[i] = (int8_t)orc_hvp_sign(seed, layer, j, start + i);
}

/* t[j] += sum_e s_j(e) x[e] over the n coordinates of one layer, j < r. */
void orc_hvp_dots(uint64_t seed, uint32_t layer, int r, uint64_t n, const double *x, double *t) {
#pragma omp parallel for schedule(static)
  for (int j = 0; j < r; ++j) {
    double acc = 0.0;
    for (uint64_t e = 0; e < n; ++e) acc += orc_hvp_sign(seed, layer, (uint32_t)j, e) * x[e];
    t[j] += acc;
  }
}

/* y[e] = shift x[e] + sum_j coef[j] s_j(e) over the n coordinates of one layer. */
void orc_hvp_combine(uint64_t seed, uint32_t layer, int r, uint64_t n, double shift, const double *coef,
                     const double *x, double *y) {
#pragma omp parallel for schedule(static)
  for (int64_t e = 0; e < (int64_t)n; ++e) {
    double acc = shift * x[e];
    for (int j = 0; j < r; ++j) acc += coef[j] * orc_hvp_sign(seed, layer, (uint32_t)j, (uint64_t)e);
    y[e] = acc;
  }
}
