// sk_internal.h -- plan records and kernel launchers of the sketch library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/sketch.h"
#include "sk_device.h"

namespace sk {

constexpr int kMaxDigits = 4;  // N' <= 2^40
constexpr int kMaxPtrs = 64;   // layers per launch (pointer pack in kernel arguments)
constexpr int kFfdSmallMax = 13;  // log2 D up to which an FFD block lives in LDS

// Per-layer plan record, mirrored on the device.
struct LayerDesc {
  int64_t n;          // elements rows*cols
  int64_t np;         // padded length N' (FWHT kinds)
  int32_t lgnp, K;    // log2 N', number of Kronecker digits
  int32_t lg[kMaxDigits];  // digit widths, digit 0 most significant
  int32_t L, lgL;     // size of the last digit (row length)
  int32_t dk1, lgdk1; // size of the second-to-last digit (1 if K < 2)
  int64_t rows_live;  // ceil(n / L)
  int32_t poff[2][2][kMaxDigits];  // digit-permutation tables [pi1, pi2][fwd, inv][digit]
  int32_t layer_id;   // RNG layer id (index in the list)
  int32_t rslot_off;  // AFJL: offset of this layer's R (first item, chunk count) pairs
  int32_t item_off;   // AFJL: first fold item of this layer
  int32_t n_items;    // AFJL: fold items of this layer
  int32_t rmaxch;     // AFJL: most fold items of one destination row
  int32_t m, nc, da, db;  // QK shape and block
  int64_t qk_col;     // QK: first output column of the block
  int64_t fa_off, fb_off;  // QK: element offsets of A (da x m, fp32) and B (db x nc, bf16 hi/lo pairs)
  int32_t lo_len_lg;  // AFFD: log2 of the low block spanned by c < D
  uint32_t hstar;     // AFFD: top-digit index of pi2 at the all-zero low part
  int32_t qbm, qdm;   // QKH/AFJLQ: size of factor K-2 and its rows kept (D / 1024)
  int64_t qP;         // QKH/AFJLQ: slabs of qbm x 1024 (product of the leading factors)
  int64_t qoff;       // QKH/AFJLQ: float offset of the layer's A, A^T, Qt, Qt^T, w
};

// AFJL fold work item: rows t in [t0, t1) of destination row r of a layer.
struct FoldItem {
  int32_t layer;  // index into the layer table
  int32_t r;
  int32_t t0, t1;
};

constexpr int kFoldRowsPerItem = 256;  // AFJL: source rows of one fold work item
constexpr int kTailGroups = 16;  // AFJL tail: parallel layer groups
struct TailGroups {
  int32_t bound[kTailGroups + 1];
};

struct PtrPack {
  const void *p[kMaxPtrs];
};
struct OutPack {
  void *p[kMaxPtrs];
};

const char *set_error(int code, const std::string &msg);

}  // namespace sk

struct sk_sketch {
  int kind = 0;
  int device = 0;
  int64_t D = 0;
  uint64_t seed = 0;
  sk::Key key{};
  std::vector<sk::LayerDesc> layers;
  sk::LayerDesc *d_layers = nullptr;
  uint16_t *d_ptab = nullptr;  // digit permutation tables (values < 1024)
  std::vector<uint16_t> h_ptab;  // host copy
  float *d_gtab = nullptr;     // FJL/AFJL: per-layer G over [0, D)
  // AFJL
  int R = 1, Lw = 0;
  std::vector<sk::FoldItem> items;
  sk::FoldItem *d_items = nullptr;
  int2 *d_rslot = nullptr;     // per layer, per destination row: (first item, chunks)
  int32_t *d_rfirst = nullptr; // per layer, per destination row: first item, -1 if none
  // FJL transpose: samples sorted by position, per layer
  std::vector<int64_t> fjl_off;  // per layer: offset into the sorted arrays (n_layers+1)
  std::vector<int64_t> fjl_uoff; // per layer: offset into the unique-position arrays
  uint32_t *d_fjl_pos = nullptr;   // unique positions
  uint32_t *d_fjl_seg = nullptr;   // segment starts into d_fjl_smp (per unique position, +1 sentinel per layer)
  uint32_t *d_fjl_smp = nullptr;   // sample ids sorted by (position, id)
  std::vector<int64_t> fjl_toff_at; // per layer: offset of its tile table in d_fjl_toff
  uint32_t *d_fjl_toff = nullptr;  // per layer and tile of 2^min(lg N', 13) positions: first unique index (+1 end)
  // FJL forward with N' > 2^13: per layer, the D samples sorted by the block of the last transform pass that
  // holds their position (ids and positions, D each) and the blocks' first entries (+ end)
  uint32_t *d_fjl_lsmp = nullptr, *d_fjl_lpos = nullptr, *d_fjl_loff = nullptr;
  std::vector<int64_t> fjl_loff_at;
  // one-pass FJL transpose (2^14 <= N' <= 2^21): per layer, the samples sorted by tile cell
  // (top bits, low bits), entry (id << 8) | middle bits, with 2^13 + 1 cell offsets
  uint32_t *d_fjlb_off = nullptr, *d_fjlb_ent = nullptr;
  std::vector<int64_t> fjlb_off_at, fjlb_ent_at;
  // and for the one-pass forward, each sample's (cell << 8) | middle bits, by id
  uint32_t *d_fjlb_pos = nullptr;
  std::vector<int64_t> fjlb_pos_at;
  // QK
  float *d_qka = nullptr;       // A factors, fp32
  uint16_t *d_qkah = nullptr;   // A factors as bf16 hi terms, then bf16 lo terms (A-first contraction)
  float *d_qkbf = nullptr;      // B factors, fp32 (second stage of the A-first contraction)
  uint16_t *d_qkb = nullptr;    // B factors as bf16 hi terms, then bf16 lo terms (hi + lo ~ fp32 B)
  int64_t qk_a_elems = 0, qk_b_elems = 0;
  // AFFD: precomputed M = H_TT (signs . G) per transposed-path layer
  float *d_mtab = nullptr;
  std::vector<int64_t> mtab_off;  // per layer: float offset into d_mtab, -1 if none
  // AFFD: G over [0, D) of each small-path layer (N' = D)
  float *d_gsmall = nullptr;
  std::vector<int64_t> gsmall_off;  // per layer: float offset into d_gsmall, -1 if none
  // FFD, D = 2^20: per block and direction, where each 8-column source group's
  // run starts in the bucket of each 8-row destination chunk (uint16 [2][128][128])
  uint16_t *d_ffdb = nullptr;
  std::vector<int64_t> ffdb_off;  // per layer: offset into d_ffdb, -1 if none
  // QKH / AFJLQ: per layer A, A^T, Qt, Qt^T, w (fp32)
  float *d_qh = nullptr;
  // AFJLF: twiddle table exp(-2 pi i m / 2^ftw_lg), m < 2^ftw_lg (complex fp32)
  float *d_ftw = nullptr;
  int ftw_lg = 0;
  // kernel timing
  struct ProfRec {
    int cls;
    int ev;
    int64_t bytes;
  };
  uint32_t prof_mask = 0;  // classes whose launch groups are timed
  std::vector<hipEvent_t> evpool;
  int evnext = 0;
  std::vector<ProfRec> recs;
  // workspace
  float *ws = nullptr;
  int64_t ws_bytes = 0;
  int64_t total_numel = 0, total_padded = 0;
};

namespace sk {

// Brackets a group of launches with a pair of pooled events when profiling.
struct ProfScope {
  sk_sketch *s;
  int idx = -1;
  hipStream_t st;
  ProfScope(sk_sketch *s_, int cls, int64_t bytes, hipStream_t st_) : s(s_), st(st_) {
    if (!((s->prof_mask >> cls) & 1u) || s->evnext + 2 > (int)s->evpool.size()) return;
    idx = s->evnext;
    s->evnext += 2;
    s->recs.push_back(sk_sketch::ProfRec{cls, idx, bytes});
    (void)hipEventRecord(s->evpool[idx], st);
  }
  ~ProfScope() {
    if (idx >= 0) (void)hipEventRecord(s->evpool[idx + 1], st);
  }
};
#define SK_PROF(cls, bytes, ...)          \
  do {                                    \
    ProfScope ps_(s, (cls), (bytes), st); \
    __VA_ARGS__;                          \
  } while (0)

}  // namespace sk
