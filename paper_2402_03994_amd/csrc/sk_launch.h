// sk_launch.h -- host-side launchers of the sketch kernels (one per kernel).
#pragma once

#include "sk_internal.h"

namespace sk {

// Generic in-place normalised Walsh-Hadamard transform of V contiguous
// vectors of length 2^lgn, as a sequence of LDS-tiled passes.
void fwht_inplace(float *data, int64_t V, int lgn, hipStream_t st);
// The passes of fwht_inplace from index bit lo0 on (the first pass of fwht_inplace covers bits
// [0, min(lgn, 13)), so lo0 = min(lgn, 13) continues after a fused first pass).
void fwht_inplace_from(float *data, int64_t V, int lgn, int lo0, hipStream_t st);
// The same passes except the last one.
void fwht_inplace_from_but_last(float *data, int64_t V, int lgn, int lo0, hipStream_t st);
// The passes fwht_inplace_from(lgn, lo0) makes: n passes over index bits [los[k], los[k] + ws[k]) with
// 2^lgcss[k] columns per tile (arrays of at least 64 entries).
int fwht_pass_plan(int lgn, int lo0, int *los, int *ws, int *lgcss);
// FJL forward, the last transform pass of layers with N' > 2^13 fused with the sample gather
// (sample lists sorted by the pass's blocks at creation).
bool fjl_last_signed_ok(const sk_sketch *s, int layer, int lo0);
void launch_fjl_last_signed(const sk_sketch *s, int layer, const float *w, int lo0, int64_t b_begin, int64_t bc,
                            void *out, int out_dtype, const float *theta0, float oscale, hipStream_t st);
void launch_fjl_last_gather(const sk_sketch *s, int layer, const float *w, int64_t b_begin, int64_t bc, float *out,
                            bool accumulate, hipStream_t st);
// FJL forward: signed load fused with the transform over index bits [0, lgw) (lgw = min(log2 N', 13)).
void launch_fjl_pass0(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc, float *w,
                      int lgw, hipStream_t st);

void launch_fill_zero(float *p, int64_t n, hipStream_t st);

// ---- QKH / AFJLQ (random-orthogonal Kronecker pre-conditioner) ----
constexpr int kQhMaxLead = 64;  // AFFDQ: slabs of one layer (N' <= 2^26)
constexpr int kQhSecond = 8;   // AFFDQ: stream factor index of the second set's digit 0
// Float offsets of a layer's factors in the factor block (per kind).
struct QhLayout {
  int64_t a, at, qt, qtt, w;                 // restricted set: A, A^T, Qt, Qt^T, w
  int64_t q1m, q1mt, q1l, q1lt, c, m;        // AFFDQ first set, c (P x P), M (P x b_m x 1024)
  int64_t total;
};
int qh_plan_layer(LayerDesc &ld, int64_t D, int kind);
QhLayout qh_layout(const LayerDesc &ld, int kind);
int64_t qh_layer_floats(const LayerDesc &ld, int kind);
void qh_generate_factors(const sk_sketch *s, std::vector<float> &host);
int64_t qh_bytes_per_vector(const sk_sketch *s, int layer, bool transpose);
// Layers whose live rows are fewer than D / 1024 (P = 1): forward in groups.
bool qh_small_layer(const sk_sketch *s, int layer);
int64_t qh_small_bytes_per_vector(const sk_sketch *s, int l0, int l1);
int qh_small_group_count(const sk_sketch *s, int l0, int l1);
void run_qh_small_group(const sk_sketch *s, int l0, int l1, int gi, const void *const *x, int dtype,
                        int64_t b_begin, int64_t bc, float *ws, float *out, bool accumulate, int phases,
                        hipStream_t st);
void run_qh_apply(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc, float *ws,
                  float *out, bool accumulate, int phases, hipStream_t st);
void run_qh_apply_T(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, float *ws, void *out,
                    int out_dtype, const float *theta0, hipStream_t st);
void launch_affdq_mtab(const sk_sketch *s, int layer, hipStream_t st);
void run_affdq_apply(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc, float *ws,
                     float *out, bool accumulate, int phases, hipStream_t st);
void run_affdq_apply_T(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, float *ws,
                       void *out, int out_dtype, const float *theta0, hipStream_t st);

// ---- AFJLF (Fourier pre-conditioner) ----
// layers with N' = D and at most 16384 entries (one kernel per direction)
bool afjlf_small_layer(const sk_sketch *s, int layer);
// whether the two-pass kernels take a layer of N' = 2^lgnp at D = 2^lgD (D^2 / (4 N') <= 16384 outputs per residue)
bool afjlf_two_pass_ok(int lgnp, int lgD);
int64_t afjlf_bytes_per_vector(const sk_sketch *s, int l0, int l1, bool transpose);
// exp(-2 pi i m / S), S = max(D, 4096), as (cos, sin) pairs, computed in double
void afjlf_twiddles(int64_t D, std::vector<float> &host, int &lgS);
// Kernel timing classes: SK_PROF_FF_ROWS brackets the launches that read the
// gradients (pass 1, small layers), SK_PROF_FF_RES the residue passes and the
// layer sum (forward); the transpose uses SK_PROF_FF_RES for pass 2 and
// SK_PROF_GATHER for the kernels that write the outputs.
void run_afjlf_fwd(sk_sketch *s, int l0, int l1, const void *const *grads, int dtype, int64_t b_begin,
                   int64_t bc, float *ws, int64_t ws_floats, float *out, bool accumulate, hipStream_t st);
void run_afjlf_T(sk_sketch *s, int l0, int l1, const float *z, int64_t b_begin, int64_t bc, float *ws,
                 int64_t ws_floats, void *const *outs, int out_dtype, const void *const *theta0, hipStream_t st);

// ---- AFJL ----
void launch_afjl_fold(const sk_sketch *s, const PtrPack &ptrs, int first_layer, int dtype, bool vec, int64_t batch,
                      int64_t b_begin, int64_t bc, int item_begin, int item_end, float *part, hipStream_t st);
void launch_afjl_tail(const sk_sketch *s, int l_begin, int l_end, int item_begin, const float *part, int64_t bc,
                      int64_t b_begin, int64_t batch, float *out, bool accumulate, hipStream_t st);
// AFJL transpose over a group of up to kMaxPtrs consecutive layers: g_l . z
// for all of them into w ([layer][vector][D]), then (after the transform of
// all ng * bc vectors) every output row of the group in one launch.
constexpr int kAfjlTRows = 32;  // source rows per workgroup of the AFJL transpose output kernel
struct AfjlTGroup {
  int32_t layer[kMaxPtrs];
  int64_t tile0[kMaxPtrs + 1];  // first tile of kAfjlTRows rows of each layer in the launch grid (+ total)
  void *out[kMaxPtrs];
  const float *th[kMaxPtrs];
};
void launch_afjl_T_prep(const sk_sketch *s, int l_first, int ng, const float *z, int64_t b_begin, int64_t bc,
                        float *w, hipStream_t st);
void launch_afjl_T_out(const sk_sketch *s, const AfjlTGroup &g, int ng, const float *w, int64_t b_begin, int64_t bc,
                       int out_dtype, hipStream_t st);

// ---- AFFD ----
// AFFD specialised for D > 1024, last digit 1024 and at most 64 top-digit values.
bool affd_fast_path(const sk_sketch *s, int layer);
int64_t affd_fast_bytes_per_vector(const sk_sketch *s, int layer);
int64_t affd_live_bytes_per_vector(const sk_sketch *s, int layer);
int64_t affd_tile_bytes();
void run_affd_fast(const sk_sketch *s, int layer, const void *x, int dtype, bool vec, int64_t b_begin, int64_t bc,
                   float *out, bool accumulate, hipStream_t st);
// AFFD for layers whose second-to-last digit is 1024 wide (slabs stored transposed).
// Small layers (N' = D, two digits, at most kSmallRows source rows of 1024):
// phases of up to kMaxPtrs such layers run as one launch each.
constexpr int kSmallRows = 8;
constexpr int kSmallMaxDk1 = 512;
struct SmallGroup {
  int32_t layer[kMaxPtrs];
  const void *x[kMaxPtrs];
  const float *gt[kMaxPtrs];  // stored G of the layer over [0, D), or null
};
// stored G rows of the small-path layers: g[j] = gauss(j) of the layer, j < D
void launch_affd_small_gtab(const sk_sketch *s, int layer, float *g, hipStream_t st);
bool affd_small_path(const sk_sketch *s, int layer);
// workspace bytes per (layer, vector) of a group: W and F, D floats each
int64_t affd_small_bytes_per_vector(const sk_sketch *s);
// phases: bit 0 = the row kernel (reads the gradients), bit 1 = the rest
void run_affd_small(const sk_sketch *s, const SmallGroup &g, int nslots, int dtype, int64_t b_begin, int64_t bc,
                    int phases, float *out, bool accumulate, hipStream_t st);
bool affd_transposed_path(const sk_sketch *s, int layer);
// Vectors per call (0 = no preference), live slabs per group, and whether W^T
// is stored compactly per group (stored M tables) or at the slab's own index.
struct AffdTPlan {
  int64_t tile;
  int gsl;
  bool compact;
};
AffdTPlan affd_transposed_plan(const sk_sketch *s, int layer);
int affd_transposed_nlive(const sk_sketch *s, int layer);
int64_t affd_transposed_group_elems(const sk_sketch *s, int layer, int s_first, int nsl);
// One slab group of a call: live slabs s_first .. s_first + nsl - 1; W^T
// holds vslabs slabs per vector when compact; F is carried in facc between
// groups (fmode bit 0: read facc first, bit 1: last group).
struct AffdTGroup {
  int s_first, nsl, vslabs;
  bool compact;
  float *facc;
  int fmode;
};
// Phases A-C of the transposed path for vectors b_begin .. b_begin + bc - 1,
// writing G^T of vector b_begin + v at gbuf + v D; the W^T workspace is s->ws.
// M[t'][l][p] = (H_TT (signs . g[., p, l]))[t'] for a transposed-path layer
void launch_affd_mtab(const sk_sketch *s, int layer, float *m, hipStream_t st);
// phases: bit 0 = A (the row kernel, reads the gradients), bit 1 = B and C
void run_affd_transposed(const sk_sketch *s, int layer, const void *x, int dtype, bool vec, int64_t b_begin,
                         int64_t bc, float *gbuf, int phases, const AffdTGroup &grp, hipStream_t st);
// Phase E of up to kMaxPtrs layers in one launch: G^T of layer j for vector
// v at g[j] + v gstride; out (+)= sum_j scale[j] (contribution of layer j).
struct OutLayers {
  int32_t n;
  int32_t layer[kMaxPtrs];
  float scale[kMaxPtrs];
  const float *g[kMaxPtrs];
};
void run_affd_transposed_outm(const sk_sketch *s, const OutLayers &ol, int64_t gstride, int64_t b_begin,
                              int64_t gb, float *out, bool accumulate, hipStream_t st);
float affd_transposed_out_scale(const sk_sketch *s, int layer);
void launch_affd_prolog(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc,
                        float *w, hipStream_t st);
void launch_affd_fold(const sk_sketch *s, int layer, const float *w, int64_t bc, float *f, hipStream_t st);
void launch_affd_gather(const sk_sketch *s, int layer, const float *f, int64_t b_begin, int64_t bc, float *out,
                        bool accumulate, hipStream_t st);
void launch_affd_T_scatter(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, float *w,
                           hipStream_t st);
void launch_mul_gauss(const sk_sketch *s, int layer, float *w, int64_t bc, hipStream_t st);
void launch_affd_T_out(const sk_sketch *s, int layer, const float *w, int64_t b_begin, int64_t bc, void *out,
                       int out_dtype, const float *theta0, hipStream_t st);

// ---- FJL ----
void launch_fjl_gather(const sk_sketch *s, int layer, const float *w, int64_t b_begin, int64_t bc, float *out,
                       bool accumulate, hipStream_t st);
void launch_fjl_T_pass0(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, float *w, int lgw,
                        hipStream_t st);
void launch_signed_out(const sk_sketch *s, int layer, const float *w, int64_t b_begin, int64_t bc, void *out,
                       int out_dtype, const float *theta0, float scale, hipStream_t st);

// One-pass FJL transpose for 2^14 <= N' <= 2^21 (tables built at creation).
bool fjl_onepass_T_ok(int lgnp, int64_t D);
void launch_fjl_T_onepass(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, void *out,
                          int out_dtype, const float *theta0, hipStream_t st);
// One-pass FJL forward for the same layers: 2^(lgnp - 13) partial slots of
// bc x D floats at part, summed afterwards by launch_reduce_partials.
void launch_fjl_fwd_onepass(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc,
                            float *part, hipStream_t st);

// ---- FFD ----
int64_t ffd_live_blocks(const sk_sketch *s, int layer);
// Small D (<= 2^13): the layer's block tables (g, Pi, signs) are made per call
// by launch_ffd_tables into ffd_small_table_floats floats of the workspace,
// which the block kernels then read.
int64_t ffd_small_table_floats(const sk_sketch *s, int layer);
void launch_ffd_tables(const sk_sketch *s, int layer, float *tab, hipStream_t st);
void launch_ffd_small_fwd(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc,
                          float *part, int64_t slot0, int64_t groups, const float *tab, hipStream_t st);
int64_t ffd_small_groups(const sk_sketch *s, int layer);
void launch_reduce_partials(const float *part, int64_t nslots, int64_t bc, int64_t D, int64_t b_begin, float *out,
                            bool accumulate, hipStream_t st);
void launch_ffd_small_T(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, void *out,
                        int out_dtype, const float *theta0, const float *tab, hipStream_t st);
void launch_ffd_copy_blocks(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc,
                            float *w, hipStream_t st);
void launch_ffd_gperm_fwd(const sk_sketch *s, int layer, const float *w, int64_t bc, float *w2, hipStream_t st);
void launch_ffd_sum_signed(const sk_sketch *s, int layer, const float *w2, int64_t b_begin, int64_t bc, float *out,
                           bool accumulate, hipStream_t st);
void launch_ffd_expand_z(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, float *w,
                         hipStream_t st);
void launch_ffd_permg_T(const sk_sketch *s, int layer, const float *w, int64_t bc, float *w2, hipStream_t st);
void launch_ffd_T_out(const sk_sketch *s, int layer, const float *w2, int64_t b_begin, int64_t bc, void *out,
                      int out_dtype, const float *theta0, hipStream_t st);

// ---- tables / debug ----
void launch_gauss_table(const sk_sketch *s, float *gtab, hipStream_t st);
void launch_debug_stream(const sk_sketch *s, int layer, int stream_id, uint64_t start, uint64_t count, uint64_t aux,
                         void *dout, hipStream_t st);

// FFD with D = 2^20: rows/cols kernels over transposed intermediates.
// phases: bit 0 = the kernel that reads the input, bit 1 = the rest.
bool ffd_large_path(const sk_sketch *s);
// Bucket offsets of the permutations of a layer's live blocks: uint16
// [block][direction][source group s < 128][destination chunk q < 128] = the
// start of group s's run inside chunk q's bucket of 8192 (direction 0: d =
// pi(k), 1: d = pi^{-1}(k)).
constexpr int64_t kFfdBucketTab = 2 * 128 * 128;
void launch_ffd_bucket_tab(const sk_sketch *s, int layer, uint16_t *tab, hipStream_t st);
void run_ffd_large_fwd(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc,
                       float *out, bool accumulate, int phases, hipStream_t st);
void run_ffd_large_T(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, void *out,
                     int out_dtype, const float *theta0, int phases, hipStream_t st);

// ---- QK ----
void launch_qk_factors(const sk_sketch *s, hipStream_t st);
// stages: bit 0 = T = X B^T (reads the gradients), bit 1 = out (+)= A T
void launch_qk_apply(const sk_sketch *s, int layer, const void *x, int dtype, int64_t b_begin, int64_t bc,
                     float *t_ws, int stages, float *out, bool accumulate, hipStream_t st);
int64_t qk_workspace_elems(const sk_sketch *s, int layer, int64_t bc);
void launch_qk_apply_T(const sk_sketch *s, int layer, const float *z, int64_t b_begin, int64_t bc, float *t_ws,
                       void *out, int out_dtype, const float *theta0, hipStream_t st);

}  // namespace sk
