// sk_api.hip -- C ABI of the sketch library: validation, planning (per-layer
// digit structure, permutation tables, AFJL work items, FJL transpose lists,
// QK factors), workspace ownership and dispatch of the kernels in sk_fwht.hip
// and sk_qk.hip onto the caller's stream.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "sk_launch.h"

using namespace sk;

namespace {

thread_local std::string g_err;

int fail(int code, const std::string &msg) {
  g_err = msg;
  return code;
}

#define SK_HIP(call)                                                                              \
  do {                                                                                            \
    hipError_t e_ = (call);                                                                       \
    if (e_ != hipSuccess) return fail(SK_EHIP, std::string(#call) + ": " + hipGetErrorString(e_)); \
  } while (0)

int ilog2(int64_t v) {
  int l = 0;
  while ((1ll << l) < v) ++l;
  return l;
}

bool is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }

int64_t workspace_budget() {
  const char *e = std::getenv("SK_WORKSPACE_MB");
  int64_t mb = e ? std::atoll(e) : 4096;
  if (mb < 16) mb = 16;
  return mb << 20;
}

// Restores the caller's current device on scope exit.
struct DeviceGuard {
  int prev = -1;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != dev) (void)hipSetDevice(dev);
  }
  ~DeviceGuard() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

void free_all(sk_sketch *s) {
  auto f = [](void *p) {
    if (p) (void)hipFree(p);
  };
  f(s->d_layers);
  f(s->d_ptab);
  f(s->d_gtab);
  f(s->d_items);
  f(s->d_rslot);
  f(s->d_rfirst);
  f(s->d_fjl_pos);
  f(s->d_fjl_seg);
  f(s->d_fjl_smp);
  f(s->d_fjl_toff);
  f(s->d_fjl_lsmp);
  f(s->d_fjl_lpos);
  f(s->d_fjl_loff);
  f(s->d_fjlb_off);
  f(s->d_fjlb_ent);
  f(s->d_fjlb_pos);
  f(s->d_qka);
  f(s->d_qkb);
  f(s->d_qkah);
  f(s->d_qkbf);
  f(s->d_mtab);
  f(s->d_gsmall);
  f(s->d_ffdb);
  f(s->d_qh);
  f(s->d_ftw);
  f(s->ws);
  for (hipEvent_t e : s->evpool) (void)hipEventDestroy(e);
  s->evpool.clear();
}

bool fwht_kind(int k) { return k == SK_FJL || k == SK_FFD || k == SK_AFFD || k == SK_AFJL; }
bool q_kind(int k) { return k == SK_QKH || k == SK_AFJLQ || k == SK_AFFDQ; }
// kinds on the padded per-layer length N' with its Kronecker digits
bool padded_kind(int k) { return fwht_kind(k) || q_kind(k) || k == SK_AFJLF; }
// kinds whose kernels need D >= 2048
bool big_d_kind(int k) { return q_kind(k) || k == SK_AFJLF; }


// Bytes of workspace one vector needs for one call over layers [l0, l1).
int64_t per_vector_bytes(const sk_sketch *s, int l0, int l1, bool transpose) {
  int64_t need = 0;
  for (int l = l0; l < l1; ++l) {
    const LayerDesc &ld = s->layers[l];
    int64_t b = 0;
    switch (s->kind) {
      case SK_AFJL:
        if (transpose) b = s->D * 4;
        break;
      case SK_AFFD:
        b = transpose ? ld.np * 4 : (ld.np + (1ll << ld.lo_len_lg) + s->D) * 4;
        break;
      case SK_FJL:
        b = ld.np * 4;
        break;
      case SK_FFD:
        if (ilog2(s->D) <= kFfdSmallMax)  // partial sums (forward), then the call's block tables
          b = ((transpose ? 0 : ffd_small_groups(s, l) * s->D) + ffd_small_table_floats(s, l)) * 4;
        else  // two intermediates, plus a uint16 bucket index per position and group of four vectors
          b = 2 * ffd_live_blocks(s, l) * s->D * 4 + ffd_live_blocks(s, l) * s->D / 2;
        break;
      case SK_QKH:
      case SK_AFJLQ:
      case SK_AFFDQ:
        b = qh_bytes_per_vector(s, l, transpose);
        break;
      case SK_AFJLF:  // the whole range at once below
        break;
      case SK_QK:  // T = X B^T (m x dB) or, A first, U = A X (dA x n)
        b = std::max((int64_t)ld.m * ld.db, (int64_t)ld.da * ld.nc) * 4;
        break;
    }
    need = std::max(need, b);
  }
  if ((s->kind == SK_QKH || s->kind == SK_AFJLQ) && !transpose)
    need = std::max(need, qh_small_bytes_per_vector(s, l0, l1));
  if (s->kind == SK_AFJLF) need = afjlf_bytes_per_vector(s, l0, l1, transpose);
  if (s->kind == SK_AFJL && !transpose) {
    // fold partials of every item of the call, plus the tail's per-group sums
    const int64_t items = s->layers[l1 - 1].item_off + s->layers[l1 - 1].n_items - s->layers[l0].item_off;
    need = std::max(need, items * s->Lw * 4 + (int64_t)kTailGroups * s->D * 4);
  }
  return need;
}

}  // namespace

// ---------------------------------------------------------------------------
// Allocation-free forward sketch.  The per-call scratch (fold partials, FJL
// and FFD intermediates, QK first-stage products) lives in `scratch`, a
// file-scope device array of kStaticScratchBytes that every device the library
// runs on holds until the process ends.  Host code never uses the array's
// name as an address (on the host it is only a stand-in for the symbol): the
// device address of each device's copy is looked up once per device with
// hipGetSymbolAddress, with that device current, and kept in g_scratch_ptr.
// ---------------------------------------------------------------------------
constexpr int64_t kStaticScratchBytes = SK_STATIC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];
namespace {
constexpr int kMaxScratchDevices = 64;
void *g_scratch_ptr[kMaxScratchDevices] = {};
std::mutex g_scratch_mu;

// Device address of `device`'s copy of scratch (the device must be current).
int scratch_ptr(int device, void **ptr) {
  if (device < 0 || device >= kMaxScratchDevices) return fail(SK_EUNSUPPORTED, "device index beyond 63");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[device]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(SK_EHIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    g_scratch_ptr[device] = p;
  }
  *ptr = g_scratch_ptr[device];
  return SK_OK;
}

// Points the handle's workspace at other memory for one call.
struct WorkspaceSwap {
  sk_sketch *s;
  float *ws;
  int64_t bytes;
  WorkspaceSwap(sk_sketch *s_, void *p, int64_t b) : s(s_), ws(s_->ws), bytes(s_->ws_bytes) {
    s->ws = (float *)p;
    s->ws_bytes = b;
  }
  ~WorkspaceSwap() {
    s->ws = ws;
    s->ws_bytes = bytes;
  }
};
}  // namespace

namespace sk {
const char *set_error(int code, const std::string &msg) {
  (void)code;
  g_err = msg;
  return g_err.c_str();
}
}  // namespace sk

extern "C" {

const char *sketch_last_error(void) { return g_err.c_str(); }

const char *sketch_status_string(int code) {
  switch (code) {
    case SK_OK: return "ok";
    case SK_EINVAL: return "invalid argument";
    case SK_EDTYPE: return "invalid dtype";
    case SK_ENOMEM: return "out of device memory";
    case SK_EHIP: return "HIP runtime error";
    case SK_EUNSUPPORTED: return "unsupported configuration";
    default: return "unknown status";
  }
}

int sketch_create(sk_kind kind, const sk_layer_shape *shapes, int32_t n_layers, int64_t D, uint64_t seed,
                  uint32_t flags, int32_t device, sk_sketch **out) {
  if (!out) return fail(SK_EINVAL, "out is NULL");
  *out = nullptr;
  if ((int)kind < 0 || (int)kind > 8) return fail(SK_EINVAL, "unknown sketch kind");
  if (!shapes || n_layers < 1) return fail(SK_EINVAL, "need at least one layer shape");
  if (flags & ~SK_FLAG_AFFD_NO_MTAB) return fail(SK_EINVAL, "unknown flags");
  for (int l = 0; l < n_layers; ++l) {
    if (shapes[l].rows < 1 || shapes[l].cols < 1)
      return fail(SK_EINVAL, "layer " + std::to_string(l) + ": rows and cols must be >= 1");
    if (shapes[l].rows > (1ll << 40) / shapes[l].cols)
      return fail(SK_EUNSUPPORTED, "layer " + std::to_string(l) + " too large");
  }
  if (padded_kind(kind)) {
    if (!is_pow2(D)) return fail(SK_EINVAL, "D must be a power of two");
    if (D < (big_d_kind(kind) ? 2048 : 16))
      return fail(SK_EUNSUPPORTED, std::string("D < ") + (big_d_kind(kind) ? "2048" : "16") + " is not supported by the kernels");
    if (D > (1ll << 20)) return fail(SK_EUNSUPPORTED, "D > 2^20 is not supported by the kernels");
    if (kind == SK_AFFDQ)
      for (int l = 0; l < n_layers; ++l)
        if (shapes[l].rows * shapes[l].cols > (1ll << 26))
          return fail(SK_EUNSUPPORTED, "AFFDQ: layer " + std::to_string(l) + " pads beyond 2^26 elements");
    // AFJLF: one-kernel layers (N' = D, at most 16384 entries) or two passes
    // with at most 16384 outputs per residue
    if (kind == SK_AFJLF)
      for (int l = 0; l < n_layers; ++l) {
        const int64_t n = shapes[l].rows * shapes[l].cols;
        int lgn = 0;
        while ((1ll << lgn) < std::max(n, D)) ++lgn;
        const bool small = lgn == ilog2(D) && n <= 16384;
        if (!small && !afjlf_two_pass_ok(lgn, ilog2(D)))
          return fail(SK_EUNSUPPORTED, "AFJLF: layer " + std::to_string(l) +
                                           ": more than 16384 outputs per residue (D^2/(4 N') with N' < 256 D/2; "
                                           "or N' = D with more than 16384 entries)");
      }
    // FJL sample positions are one 32-bit Philox word masked to N' - 1, uniform
    // only while N' <= 2^32
    if (kind == SK_FJL)
      for (int l = 0; l < n_layers; ++l)
        if (shapes[l].rows * shapes[l].cols > (1ll << 32))
          return fail(SK_EUNSUPPORTED, "FJL: layer " + std::to_string(l) + " pads beyond 2^32 elements");
  } else {
    int64_t tot = 0;
    for (int l = 0; l < n_layers; ++l) {
      const sk_layer_shape &sh = shapes[l];
      if (sh.qk_da < 1 || sh.qk_db < 1 || sh.qk_da > sh.rows || sh.qk_db > sh.cols)
        return fail(SK_EINVAL, "layer " + std::to_string(l) + ": need 1 <= qk_da <= rows and 1 <= qk_db <= cols");
      if (sh.rows > (1ll << 31) || sh.cols > (1ll << 31))
        return fail(SK_EUNSUPPORTED, "QK matrix dimension above 2^31");
      tot += (int64_t)sh.qk_da * sh.qk_db;
    }
    if (tot != D) return fail(SK_EINVAL, "QK: sum of qk_da*qk_db must equal D");
  }
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) return fail(SK_EHIP, "no HIP device available");
  if (device < 0 || device >= ndev) return fail(SK_EINVAL, "device index out of range");

  sk_sketch *s = new (std::nothrow) sk_sketch();
  if (!s) return fail(SK_ENOMEM, "host allocation failed");
  s->kind = kind;
  s->device = device;
  s->D = D;
  s->seed = seed;
  s->key = make_key(seed);
  s->layers.resize(n_layers);

  std::vector<uint16_t> ptab;
  const bool need_pi1 = kind == SK_AFFD || kind == SK_AFJL;
  const bool need_pi2 = kind == SK_AFFD;
  int64_t qk_col = 0, fac_a = 0, fac_b = 0;
  for (int l = 0; l < n_layers; ++l) {
    LayerDesc &ld = s->layers[l];
    std::memset(&ld, 0, sizeof(ld));
    ld.n = shapes[l].rows * shapes[l].cols;
    ld.layer_id = l;
    s->total_numel += ld.n;
    if (padded_kind(kind)) {
      ld.np = 1;
      while (ld.np < std::max(ld.n, D)) ld.np <<= 1;
      ld.lgnp = ilog2(ld.np);
      int lg[8];
      ld.K = kron_shapes_log2(ld.lgnp, lg);
      if (ld.K > kMaxDigits) {
        free_all(s);
        delete s;
        return fail(SK_EUNSUPPORTED, "layer too large (more than 4 Kronecker digits)");
      }
      for (int k = 0; k < ld.K; ++k) ld.lg[k] = lg[k];
      ld.lgL = ld.lg[ld.K - 1];
      ld.L = 1 << ld.lgL;
      ld.lgdk1 = ld.K >= 2 ? ld.lg[ld.K - 2] : 0;
      ld.dk1 = 1 << ld.lgdk1;
      ld.rows_live = (ld.n + ld.L - 1) / ld.L;
      s->total_padded += ld.np;
      for (int si = 0; si < 2; ++si) {
        if ((si == 0 && !need_pi1) || (si == 1 && !need_pi2)) continue;
        const uint32_t stream = si == 0 ? ST_PI1 : ST_PI2;
        for (int k = 0; k < ld.K; ++k) {
          const int w = ld.lg[k];
          const PermKey pk = perm_key((uint32_t)l, stream, (uint32_t)k, (uint32_t)w, s->key);
          ld.poff[si][0][k] = (int32_t)ptab.size();
          ld.poff[si][1][k] = (int32_t)ptab.size() + (1 << w);
          ptab.resize(ptab.size() + 2 * (size_t)(1 << w));
          uint16_t *fw = ptab.data() + ld.poff[si][0][k];
          uint16_t *iv = ptab.data() + ld.poff[si][1][k];
          for (uint32_t x = 0; x < (1u << w); ++x) {
            const uint32_t y = perm_fwd(pk, x);
            fw[x] = (uint16_t)y;
            iv[y] = (uint16_t)x;
          }
        }
      }
      if (kind == SK_AFFD) {
        // low block: the digits spanned by c < D
        const int nlow = D > ld.L ? 2 : 1;
        ld.lo_len_lg = ld.lgL + (nlow == 2 ? ld.lgdk1 : 0);
        uint32_t hstar = 0;
        int shift = 0;
        for (int k = ld.K - 1 - nlow; k >= 0; --k) {
          hstar |= (uint32_t)ptab[ld.poff[1][0][k] + 0] << shift;
          shift += ld.lg[k];
        }
        ld.hstar = hstar;
      }
    } else {
      ld.m = (int32_t)shapes[l].rows;
      ld.nc = (int32_t)shapes[l].cols;
      ld.da = shapes[l].qk_da;
      ld.db = shapes[l].qk_db;
      ld.qk_col = qk_col;
      qk_col += (int64_t)ld.da * ld.db;
      ld.fa_off = fac_a;
      fac_a += (int64_t)ld.da * ld.m;
      ld.fb_off = fac_b;
      fac_b += (int64_t)ld.db * ld.nc;
    }
  }
  s->qk_a_elems = fac_a;
  s->qk_b_elems = fac_b;
  int64_t qh_floats = 0;
  if (q_kind(kind)) {
    for (int l = 0; l < n_layers; ++l) {
      LayerDesc &ld = s->layers[l];
      if (qh_plan_layer(ld, D, kind) != SK_OK) {
        free_all(s);
        delete s;
        return fail(SK_EUNSUPPORTED, "layer " + std::to_string(l) + ": Kronecker shape not supported");
      }
      ld.qoff = qh_floats;
      qh_floats += (qh_layer_floats(ld, kind) + 3) & ~3ll;  // 16-byte aligned blocks
    }
  }

  // AFJL work items: destination rows r of an R x Lw accumulator.
  std::vector<int2> rslot;
  if (kind == SK_AFJL) {
    s->Lw = (int)std::min<int64_t>(D, 1024);
    s->R = (int)(D / s->Lw);
    const int R = s->R;
    const int64_t rows_per_item = kFoldRowsPerItem;
    for (int l = 0; l < n_layers; ++l) {
      LayerDesc &ld = s->layers[l];
      ld.rslot_off = (int32_t)rslot.size();
      ld.item_off = (int32_t)s->items.size();
      if (R == 1) {
        const int64_t T = ld.rows_live;
        const int first = (int)s->items.size();
        for (int64_t t0 = 0; t0 < T; t0 += rows_per_item)
          s->items.push_back(FoldItem{l, 0, (int32_t)t0, (int32_t)std::min(T, t0 + rows_per_item)});
        rslot.push_back(int2{first, (int)(s->items.size() - first)});
      } else {
        const int nk = ld.dk1 / R;
        const int64_t ntop_live = (ld.rows_live + ld.dk1 - 1) / ld.dk1;
        const int64_t T = ntop_live * nk;
        const uint16_t *inv = ptab.data() + ld.poff[0][1][ld.K - 2];
        for (int r = 0; r < R; ++r) {
          // live rows mapped to r, to skip destination rows that receive nothing
          int64_t live = 0;
          for (int64_t t = 0; t < T && live == 0; ++t) {
            const int64_t htop = t / nk, k = t % nk;
            if (htop * ld.dk1 + inv[r + k * R] < ld.rows_live) live = 1;
          }
          const int first = (int)s->items.size();
          if (live)
            for (int64_t t0 = 0; t0 < T; t0 += rows_per_item)
              s->items.push_back(FoldItem{l, r, (int32_t)t0, (int32_t)std::min(T, t0 + rows_per_item)});
          rslot.push_back(int2{first, (int)(s->items.size() - first)});
        }
      }
      ld.n_items = (int32_t)s->items.size() - ld.item_off;
      ld.rmaxch = 0;
      for (size_t i = ld.rslot_off; i < rslot.size(); ++i) ld.rmaxch = std::max(ld.rmaxch, rslot[i].y);
    }
  }

  // FJL transpose: samples grouped by position (deterministic order).
  std::vector<uint32_t> fpos, fseg, fsmp, ftoff, flsmp, flpos, floff, fboff, fbent, fbpos;
  if (kind == SK_FJL) {
    s->fjlb_pos_at.assign(n_layers, -1);
    s->fjlb_off_at.assign(n_layers, -1);
    s->fjlb_ent_at.assign(n_layers, -1);
    s->fjl_uoff.assign(n_layers + 1, 0);
    s->fjl_toff_at.assign(n_layers, 0);
    s->fjl_loff_at.assign(n_layers, 0);
    flsmp.assign((size_t)n_layers * D, 0);
    flpos.assign((size_t)n_layers * D, 0);
    std::vector<std::pair<uint32_t, uint32_t>> v(D);
    for (int l = 0; l < n_layers; ++l) {
      const LayerDesc &ld = s->layers[l];
      for (int64_t i = 0; i < D; ++i) v[i] = {sample_index((uint64_t)i, (uint32_t)l, s->key, (uint64_t)ld.np), (uint32_t)i};
      std::sort(v.begin(), v.end());
      const uint32_t base = (uint32_t)fsmp.size();
      for (int64_t i = 0; i < D; ++i) {
        if (i == 0 || v[i].first != v[i - 1].first) {
          fpos.push_back(v[i].first);
          fseg.push_back(base + (uint32_t)i);
        }
        fsmp.push_back(v[i].second);
      }
      fseg.push_back(base + (uint32_t)D);  // sentinel
      s->fjl_uoff[l + 1] = (int64_t)fpos.size();
      // tile table of the fused transpose pass: the layer's unique positions in tile t are
      // [ftoff[at + t], ftoff[at + t + 1]) (indices relative to the layer's first one)
      const int lgw = std::min(ld.lgnp, 13);
      const int64_t tiles = ld.np >> lgw, u0 = s->fjl_uoff[l];
      s->fjl_toff_at[l] = (int64_t)ftoff.size();
      int64_t u = u0;
      for (int64_t t = 0; t <= tiles; ++t) {
        while (u < s->fjl_uoff[l + 1] && ((int64_t)fpos[u] >> lgw) < t) ++u;
        ftoff.push_back((uint32_t)(u - u0));
      }
      // forward: the samples by block of the last transform pass (positions whose low `lo` bits fall in
      // [cb 2^lgcs, (cb + 1) 2^lgcs)), ids ascending within a block
      s->fjl_loff_at[l] = (int64_t)floff.size();
      if (ld.lgnp > 13) {
        int los[64], wsp[64], lgcss[64];
        const int np = fwht_pass_plan(ld.lgnp, 13, los, wsp, lgcss);
        const int lo = los[np - 1], lgcs = lgcss[np - 1];
        const int64_t nblk = 1ll << (lo - lgcs);
        std::vector<std::pair<uint32_t, uint32_t>> bs(D);
        for (int64_t i = 0; i < D; ++i) {
          const uint32_t p = sample_index((uint64_t)i, (uint32_t)l, s->key, (uint64_t)ld.np);
          bs[i] = {(uint32_t)((p & ((1u << lo) - 1)) >> lgcs), (uint32_t)i};
        }
        std::sort(bs.begin(), bs.end());
        int64_t k = 0;
        for (int64_t b = 0; b <= nblk; ++b) {
          while (k < D && (int64_t)bs[k].first < b) ++k;
          floff.push_back((uint32_t)k);
        }
        for (int64_t i = 0; i < D; ++i) {
          flsmp[(size_t)l * D + i] = bs[i].second;
          flpos[(size_t)l * D + i] = sample_index((uint64_t)bs[i].second, (uint32_t)l, s->key, (uint64_t)ld.np);
        }
      }
      if (fjl_onepass_T_ok(ld.lgnp, D)) {
        // cell (p_h, p_c) = (p >> 13, low B = 26 - lgnp bits) of the one-pass transpose's tile; entries of a
        // cell by id, each (id << 8) | the H = lgnp - 13 middle bits
        const int Hb = ld.lgnp - 13, Bb = 13 - Hb;
        std::vector<std::pair<uint32_t, uint32_t>> cs(D);
        for (int64_t i = 0; i < D; ++i) {
          const uint32_t p = sample_index((uint64_t)i, (uint32_t)l, s->key, (uint64_t)ld.np);
          const uint32_t cell = ((p >> 13) << Bb) | (p & ((1u << Bb) - 1));
          cs[i] = {cell, ((uint32_t)i << 8) | ((p >> Bb) & ((1u << Hb) - 1))};
        }
        s->fjlb_pos_at[l] = (int64_t)fbpos.size();
        for (int64_t i = 0; i < D; ++i) fbpos.push_back((cs[i].first << 8) | (cs[i].second & 255u));
        std::sort(cs.begin(), cs.end());
        s->fjlb_off_at[l] = (int64_t)fboff.size();
        s->fjlb_ent_at[l] = (int64_t)fbent.size();
        int64_t k = 0;
        for (uint32_t c = 0; c <= 8192; ++c) {
          while (k < D && cs[k].first < c) ++k;
          fboff.push_back((uint32_t)k);
        }
        for (int64_t i = 0; i < D; ++i) fbent.push_back(cs[i].second);
      }
    }
  }

  DeviceGuard guard(device);
  auto alloc = [&](void **p, size_t bytes) -> int {
    if (bytes == 0) return SK_OK;
    if (hipMalloc(p, bytes) != hipSuccess) {
      (void)hipGetLastError();
      return fail(SK_ENOMEM, "hipMalloc of " + std::to_string(bytes) + " bytes failed");
    }
    return SK_OK;
  };
  auto h2d_sync = [&](void *d, const void *h, size_t bytes) -> int {
    if (bytes == 0) return SK_OK;
    if (hipMemcpy(d, h, bytes, hipMemcpyHostToDevice) != hipSuccess)
      return fail(SK_EHIP, std::string("hipMemcpy: ") + hipGetErrorString(hipGetLastError()));
    return SK_OK;
  };
  int rc = SK_OK;
#define SK_TRY(expr)      \
  do {                    \
    rc = (expr);          \
    if (rc != SK_OK) {    \
      free_all(s);        \
      delete s;           \
      return rc;          \
    }                     \
  } while (0)
  SK_TRY(alloc((void **)&s->d_layers, sizeof(LayerDesc) * n_layers));
  SK_TRY(alloc((void **)&s->d_ptab, sizeof(uint16_t) * ptab.size()));
  s->h_ptab = ptab;
  if (kind == SK_AFJL || kind == SK_FJL || kind == SK_AFJLQ || kind == SK_AFJLF)
    SK_TRY(alloc((void **)&s->d_gtab, sizeof(float) * n_layers * D));
  if (kind == SK_AFJLF) {
    std::vector<float> tw;
    afjlf_twiddles(D, tw, s->ftw_lg);
    SK_TRY(alloc((void **)&s->d_ftw, sizeof(float) * tw.size()));
    SK_TRY(h2d_sync(s->d_ftw, tw.data(), sizeof(float) * tw.size()));
  }
  if (qh_floats > 0) {
    SK_TRY(alloc((void **)&s->d_qh, sizeof(float) * qh_floats));
    std::vector<float> host((size_t)qh_floats, 0.0f);
    qh_generate_factors(s, host);
    if (hipMemcpy(s->d_qh, host.data(), sizeof(float) * qh_floats, hipMemcpyHostToDevice) != hipSuccess) {
      free_all(s);
      delete s;
      return fail(SK_EHIP, std::string("hipMemcpy: ") + hipGetErrorString(hipGetLastError()));
    }
    if (kind == SK_AFFDQ)
      for (int l = 0; l < n_layers; ++l) launch_affdq_mtab(s, l, nullptr);
  }
  SK_TRY(alloc((void **)&s->d_items, sizeof(FoldItem) * s->items.size()));
  SK_TRY(alloc((void **)&s->d_rslot, sizeof(int2) * rslot.size()));
  std::vector<int32_t> rfirst(rslot.size());
  for (size_t i = 0; i < rslot.size(); ++i) rfirst[i] = rslot[i].y > 0 ? rslot[i].x : -1;
  SK_TRY(alloc((void **)&s->d_rfirst, sizeof(int32_t) * rfirst.size()));
  SK_TRY(alloc((void **)&s->d_fjl_pos, sizeof(uint32_t) * fpos.size()));
  SK_TRY(alloc((void **)&s->d_fjl_seg, sizeof(uint32_t) * fseg.size()));
  SK_TRY(alloc((void **)&s->d_fjl_smp, sizeof(uint32_t) * fsmp.size()));
  SK_TRY(alloc((void **)&s->d_fjl_toff, sizeof(uint32_t) * ftoff.size()));
  SK_TRY(alloc((void **)&s->d_fjl_lsmp, sizeof(uint32_t) * flsmp.size()));
  SK_TRY(alloc((void **)&s->d_fjl_lpos, sizeof(uint32_t) * flpos.size()));
  SK_TRY(alloc((void **)&s->d_fjl_loff, sizeof(uint32_t) * floff.size()));
  if (!fboff.empty()) {
    SK_TRY(alloc((void **)&s->d_fjlb_off, sizeof(uint32_t) * fboff.size()));
    SK_TRY(alloc((void **)&s->d_fjlb_ent, sizeof(uint32_t) * fbent.size()));
    SK_TRY(alloc((void **)&s->d_fjlb_pos, sizeof(uint32_t) * fbpos.size()));
  }
  SK_TRY(alloc((void **)&s->d_qka, sizeof(float) * fac_a));
  SK_TRY(alloc((void **)&s->d_qkb, sizeof(uint16_t) * 2 * fac_b));
  SK_TRY(alloc((void **)&s->d_qkah, sizeof(uint16_t) * 2 * fac_a));
  SK_TRY(alloc((void **)&s->d_qkbf, sizeof(float) * fac_b));

  auto h2d = [&](void *d, const void *h, size_t bytes) -> int {
    if (bytes == 0) return SK_OK;
    if (hipMemcpy(d, h, bytes, hipMemcpyHostToDevice) != hipSuccess)
      return fail(SK_EHIP, std::string("hipMemcpy: ") + hipGetErrorString(hipGetLastError()));
    return SK_OK;
  };
  SK_TRY(h2d(s->d_layers, s->layers.data(), sizeof(LayerDesc) * n_layers));
  SK_TRY(h2d(s->d_ptab, ptab.data(), sizeof(uint16_t) * ptab.size()));
  SK_TRY(h2d(s->d_items, s->items.data(), sizeof(FoldItem) * s->items.size()));
  SK_TRY(h2d(s->d_rslot, rslot.data(), sizeof(int2) * rslot.size()));
  SK_TRY(h2d(s->d_rfirst, rfirst.data(), sizeof(int32_t) * rfirst.size()));
  SK_TRY(h2d(s->d_fjl_pos, fpos.data(), sizeof(uint32_t) * fpos.size()));
  SK_TRY(h2d(s->d_fjl_seg, fseg.data(), sizeof(uint32_t) * fseg.size()));
  SK_TRY(h2d(s->d_fjl_smp, fsmp.data(), sizeof(uint32_t) * fsmp.size()));
  SK_TRY(h2d(s->d_fjl_toff, ftoff.data(), sizeof(uint32_t) * ftoff.size()));
  SK_TRY(h2d(s->d_fjl_lsmp, flsmp.data(), sizeof(uint32_t) * flsmp.size()));
  SK_TRY(h2d(s->d_fjl_lpos, flpos.data(), sizeof(uint32_t) * flpos.size()));
  SK_TRY(h2d(s->d_fjl_loff, floff.data(), sizeof(uint32_t) * floff.size()));
  if (!fboff.empty()) {
    SK_TRY(h2d(s->d_fjlb_off, fboff.data(), sizeof(uint32_t) * fboff.size()));
    SK_TRY(h2d(s->d_fjlb_ent, fbent.data(), sizeof(uint32_t) * fbent.size()));
    SK_TRY(h2d(s->d_fjlb_pos, fbpos.data(), sizeof(uint32_t) * fbpos.size()));
  }

  // workspace: room for up to 256 vectors of the largest per-vector need
  const int64_t pv = std::max(per_vector_bytes(s, 0, n_layers, false), per_vector_bytes(s, 0, n_layers, true));
  const int64_t budget = workspace_budget();
  if (pv > budget) {
    free_all(s);
    delete s;
    return fail(SK_EUNSUPPORTED, "one vector needs " + std::to_string(pv) + " bytes of workspace, above the budget");
  }
  s->ws_bytes = std::min<int64_t>(budget, pv * 256);
  if (s->ws_bytes > 0) SK_TRY(alloc((void **)&s->ws, (size_t)s->ws_bytes));

  if (kind == SK_AFFD && !(flags & SK_FLAG_AFFD_NO_MTAB)) {
    // M tables of the transposed-path layers, when they fit the budget
    int64_t total = 0;
    s->mtab_off.assign(n_layers, -1);
    for (int l = 0; l < n_layers; ++l)
      if (affd_transposed_path(s, l)) {
        s->mtab_off[l] = total;
        total += s->layers[l].np;
      }
    const char *e = std::getenv("SK_AFFD_MTAB_MB");
    const int64_t mb = e ? std::atoll(e) : 8192;
    if (total > 0 && total * 4 <= (mb << 20)) {
      SK_TRY(alloc((void **)&s->d_mtab, (size_t)total * 4));
      for (int l = 0; l < n_layers; ++l)
        if (s->mtab_off[l] >= 0) launch_affd_mtab(s, l, s->d_mtab + s->mtab_off[l], nullptr);
    } else {
      s->mtab_off.assign(n_layers, -1);
    }
  }
  if (kind == SK_AFFD) {
    // G of the small-path layers (N' = D floats each)
    int64_t total = 0;
    s->gsmall_off.assign(n_layers, -1);
    for (int l = 0; l < n_layers; ++l)
      if (affd_small_path(s, l)) {
        s->gsmall_off[l] = total;
        total += D;
      }
    if (total > 0) {
      SK_TRY(alloc((void **)&s->d_gsmall, (size_t)total * 4));
      for (int l = 0; l < n_layers; ++l)
        if (s->gsmall_off[l] >= 0) launch_affd_small_gtab(s, l, s->d_gsmall + s->gsmall_off[l], nullptr);
    }
  }
  if (kind == SK_FFD && ffd_large_path(s)) {
    // bucket offsets of the permutation of every live block (64 KB per block),
    // when they fit SK_FFD_BUCKET_MB MiB
    int64_t total = 0;
    s->ffdb_off.assign(n_layers, -1);
    for (int l = 0; l < n_layers; ++l) {
      s->ffdb_off[l] = total;
      total += ffd_live_blocks(s, l) * kFfdBucketTab;
    }
    const char *e = std::getenv("SK_FFD_BUCKET_MB");
    const int64_t mb = e ? std::atoll(e) : 1024;
    if (total * 2 <= (mb << 20)) {
      SK_TRY(alloc((void **)&s->d_ffdb, (size_t)total * 2));
      for (int l = 0; l < n_layers; ++l) launch_ffd_bucket_tab(s, l, s->d_ffdb + s->ffdb_off[l], nullptr);
    } else {
      s->ffdb_off.assign(n_layers, -1);
    }
  }
  if (s->d_gtab) launch_gauss_table(s, s->d_gtab, nullptr);
  if (kind == SK_QK) launch_qk_factors(s, nullptr);
  if (hipDeviceSynchronize() != hipSuccess) {
    const std::string m = hipGetErrorString(hipGetLastError());
    free_all(s);
    delete s;
    return fail(SK_EHIP, "table generation failed: " + m);
  }
#undef SK_TRY
  *out = s;
  return SK_OK;
}

void sketch_destroy(sk_sketch *s) {
  if (!s) return;
  {
    DeviceGuard guard(s->device);
    (void)hipDeviceSynchronize();
    free_all(s);
  }
  delete s;
}

int sketch_query(const sk_sketch *s, sk_info *info) {
  if (!s || !info) return fail(SK_EINVAL, "NULL argument");
  info->kind = s->kind;
  info->n_layers = (int32_t)s->layers.size();
  info->D = s->D;
  info->seed = s->seed;
  info->total_numel = s->total_numel;
  info->total_padded = s->total_padded;
  info->workspace_bytes = s->ws_bytes;
  info->rng_version = kRngVersion;
  info->device = s->device;
  return SK_OK;
}

static int check_range(const sk_sketch *s, int32_t first_layer, int32_t n_layers) {
  if (first_layer < 0 || n_layers < 1 || (int64_t)first_layer + n_layers > (int64_t)s->layers.size())
    return fail(SK_EINVAL, "layer range out of bounds");
  return SK_OK;
}

int sketch_apply(sk_sketch *s, const void *const *grads, sk_dtype dtype, int64_t batch, float *out,
                 int32_t first_layer, int32_t n_layers, int32_t accumulate, void *stream) {
  if (!s) return fail(SK_EINVAL, "sketch is NULL");
  if (dtype != SK_F32 && dtype != SK_BF16) return fail(SK_EDTYPE, "dtype must be SK_F32 or SK_BF16");
  if (batch < 0) return fail(SK_EINVAL, "batch must be >= 0");
  if (int rc = check_range(s, first_layer, n_layers)) return rc;
  if (batch == 0) return SK_OK;
  if (!grads || !out) return fail(SK_EINVAL, "grads and out must be non-NULL");
  for (int i = 0; i < n_layers; ++i)
    if (!grads[i]) return fail(SK_EINVAL, "grads[" + std::to_string(i) + "] is NULL");
  const int l0 = first_layer, l1 = first_layer + n_layers;
  hipStream_t st = (hipStream_t)stream;
  DeviceGuard guard(s->device);
  const int64_t pv = per_vector_bytes(s, l0, l1, false);
  int64_t bcmax = pv > 0 ? s->ws_bytes / pv : batch;
  if (bcmax < 1) return fail(SK_EUNSUPPORTED, "workspace too small for one vector");
  // AFJLF kernels place every work item of a vector on XCD (vector mod 8): chunks of a
  // multiple of 8 vectors keep the eight XCDs equally loaded
  if (s->kind == SK_AFJLF && bcmax > 8 && batch > bcmax) bcmax &= ~7ll;
  const int esz = dtype == SK_BF16 ? 2 : 4;
  if (s->kind == SK_AFFD) {
    bool all_fast = true;
    for (int l = l0; l < l1; ++l) all_fast = all_fast && affd_fast_path(s, l);
    if (all_fast) bcmax = batch;  // the fast path tiles the batch per layer
  }

  for (int64_t b0 = 0; b0 < batch; b0 += bcmax) {
    const int64_t bc = std::min(bcmax, batch - b0);
    switch (s->kind) {
      case SK_AFJL: {
        // fold launches of at most kMaxPtrs layers, then one tail over all layers
        const int it_base = s->layers[l0].item_off;
        int64_t in_bytes = 0;
        for (int g0 = l0; g0 < l1; g0 += kMaxPtrs) {
          const int g1 = std::min(l1, g0 + kMaxPtrs);
          PtrPack pp{};
          bool vec = true;
          int64_t gb = 0;
          for (int l = g0; l < g1; ++l) {
            pp.p[l - g0] = grads[l - l0];
            gb += bc * s->layers[l].n * esz;
            // vector loads: 4 fp32 or 8 bf16 elements (16 bytes) per thread
            if ((s->layers[l].n & (dtype == SK_BF16 ? 7 : 3)) || ((uintptr_t)grads[l - l0] & 15)) vec = false;
          }
          in_bytes += gb;
          const int it0 = s->layers[g0].item_off;
          const int it1 = s->layers[g1 - 1].item_off + s->layers[g1 - 1].n_items;
          float *part = s->ws + (int64_t)(it0 - it_base) * bc * s->Lw;
          SK_PROF(SK_PROF_AFJL_FOLD, gb,
                  launch_afjl_fold(s, pp, g0, dtype, vec, batch, b0, bc, it0, it1, part, st));
        }
        SK_PROF(SK_PROF_AFJL_TAIL, bc * s->D * 4,
                launch_afjl_tail(s, l0, l1, it_base, s->ws, bc, b0, batch, out, accumulate != 0, st));
        (void)in_bytes;
        break;
      }
      case SK_AFFD: {
        bool acc_now = accumulate != 0;  // false until the first layer has written out
        std::vector<int> small;
        // Transposed-path layers: the W^T region of the largest tile of the
        // call at the start of the workspace, then one G^T slot (bc x D
        // floats) per layer waiting for the shared output pass, which runs
        // when the slots are full, before any other kind of layer uses the
        // workspace, and at the end.
        const int64_t ws_f = s->ws_bytes / 4;
        struct TPlan {
          int64_t tile, wt_pv, fa_pv;
          int gsl, ngroups, nlive;
          bool compact;
        };
        auto tplan = [&](int l) {
          const LayerDesc &ld = s->layers[l];
          const AffdTPlan pl = affd_transposed_plan(s, l);
          TPlan t{};
          t.tile = pl.tile ? pl.tile
                           : std::max<int64_t>(1, affd_tile_bytes() / std::max<int64_t>(affd_live_bytes_per_vector(s, l), 1));
          t.nlive = affd_transposed_nlive(s, l);
          t.gsl = pl.gsl;
          t.ngroups = (t.nlive + pl.gsl - 1) / pl.gsl;
          t.compact = pl.compact;
          t.wt_pv = pl.compact ? ((int64_t)pl.gsl << 20) : ld.np;
          t.fa_pv = t.ngroups > 1 ? (1ll << 20) : 0;
          t.tile = std::min({t.tile, bc, std::max<int64_t>(1, ws_f / (t.wt_pv + t.fa_pv + s->D))});
          return t;
        };
        int64_t wt_region = 0;
        for (int l = l0; l < l1; ++l)
          if (!affd_small_path(s, l) && affd_fast_path(s, l) && affd_transposed_path(s, l)) {
            const TPlan t = tplan(l);
            wt_region = std::max(wt_region, t.tile * (t.wt_pv + t.fa_pv));
          }
        const int64_t gslot = bc * s->D;
        const int64_t nslots = std::min<int64_t>(kMaxPtrs, (ws_f - wt_region) / gslot);
        OutLayers ol{};
        auto flush = [&]() {
          if (!ol.n) return;
          SK_PROF(SK_PROF_GATHER, bc * s->D * 4, run_affd_transposed_outm(s, ol, s->D, b0, bc, out, acc_now, st));
          acc_now = true;
          ol.n = 0;
        };
        // rows and top kernels of one transposed layer for vectors g0 .. g0 + gb - 1,
        // G^T of vector g0 + v at gbuf + v D
        auto run_t = [&](int l, const TPlan &t, int64_t g0, int64_t gb, float *gbuf) {
          const LayerDesc &ld = s->layers[l];
          const bool vec = !(ld.n & 3) && !((uintptr_t)grads[l - l0] & 15);
          float *facc = s->ws + t.tile * t.wt_pv;
          for (int64_t t0 = g0; t0 < g0 + gb; t0 += t.tile) {
            const int64_t tb = std::min(t.tile, g0 + gb - t0);
            float *gt = gbuf + (t0 - g0) * s->D;
            for (int gi = 0; gi < t.ngroups; ++gi) {
              AffdTGroup grp{gi * t.gsl, std::min(t.gsl, t.nlive - gi * t.gsl), t.gsl, t.compact, facc,
                             (gi > 0 ? 1 : 0) | (gi == t.ngroups - 1 ? 2 : 0)};
              const int64_t gel = t.ngroups > 1 ? affd_transposed_group_elems(s, l, grp.s_first, grp.nsl) : ld.n;
              SK_PROF(SK_PROF_AFFD_ROWS, tb * gel * esz,
                      run_affd_transposed(s, l, grads[l - l0], dtype, vec, t0, tb, gt, 1, grp, st));
              SK_PROF(SK_PROF_AFFD_FOLD, 0,
                      run_affd_transposed(s, l, grads[l - l0], dtype, vec, t0, tb, gt, 2, grp, st));
            }
          }
        };
        for (int l = l0; l < l1; ++l) {
          const LayerDesc &ld = s->layers[l];
          if (affd_small_path(s, l)) {
            small.push_back(l);
            continue;
          }
          if (affd_fast_path(s, l) && affd_transposed_path(s, l)) {
            const TPlan t = tplan(l);
            if (nslots >= 1) {
              if (ol.n == nslots) flush();
              float *gbuf = s->ws + wt_region + ol.n * gslot;
              run_t(l, t, b0, bc, gbuf);
              ol.layer[ol.n] = l;
              ol.scale[ol.n] = affd_transposed_out_scale(s, l);
              ol.g[ol.n] = gbuf;
              ++ol.n;
              continue;
            }
            // small workspace: G^T of up to gmax vectors after this layer's W^T tile
            const int64_t gmax = std::max(t.tile, (ws_f - t.tile * (t.wt_pv + t.fa_pv)) / s->D / t.tile * t.tile);
            float *gbuf = s->ws + t.tile * (t.wt_pv + t.fa_pv);
            for (int64_t g0 = b0; g0 < b0 + bc; g0 += gmax) {
              const int64_t gb = std::min(gmax, b0 + bc - g0);
              run_t(l, t, g0, gb, gbuf);
              OutLayers one{};
              one.n = 1;
              one.layer[0] = l;
              one.scale[0] = affd_transposed_out_scale(s, l);
              one.g[0] = gbuf;
              SK_PROF(SK_PROF_GATHER, gb * s->D * 4, run_affd_transposed_outm(s, one, s->D, g0, gb, out, acc_now, st));
            }
            acc_now = true;
            continue;
          }
          flush();  // the other paths use the workspace from its start
          if (affd_fast_path(s, l)) {
            // batch tile sized so the layer's intermediate stays cache-resident between phases
            const int64_t live = affd_live_bytes_per_vector(s, l);
            int64_t tile = std::max<int64_t>(1, affd_tile_bytes() / std::max<int64_t>(live, 1));
            const bool vec = !(ld.n & 3) && !((uintptr_t)grads[l - l0] & 15);
            tile = std::min(tile, std::max<int64_t>(1, s->ws_bytes / affd_fast_bytes_per_vector(s, l)));
            for (int64_t t0 = b0; t0 < b0 + bc; t0 += tile) {
              const int64_t tb = std::min(tile, b0 + bc - t0);
              SK_PROF(SK_PROF_AFFD_FOLD, tb * ld.n * esz + (l == l1 - 1 ? tb * s->D * 4 : 0),
                      run_affd_fast(s, l, grads[l - l0], dtype, vec, t0, tb, out, acc_now, st));
            }
            acc_now = true;
            continue;
          }
          float *w = s->ws;
          float *f = s->ws + bc * ld.np;
          SK_PROF(SK_PROF_PROLOG, bc * ld.n * esz, launch_affd_prolog(s, l, grads[l - l0], dtype, b0, bc, w, st));
          SK_PROF(SK_PROF_FWHT, 0, fwht_inplace(w, bc, ld.lgnp, st));
          SK_PROF(SK_PROF_AFFD_FOLD, 0, launch_affd_fold(s, l, w, bc, f, st));
          SK_PROF(SK_PROF_FWHT, 0, fwht_inplace(f, bc, ld.lo_len_lg, st));
          SK_PROF(SK_PROF_GATHER, (l == l1 - 1 ? bc * s->D * 4 : 0),
                  launch_affd_gather(s, l, f, b0, bc, out, acc_now, st));
          acc_now = true;
        }
        flush();
        if (!small.empty()) {
          // groups of up to kMaxPtrs small layers; vectors tiled so that W and F
          // of every slot fit the workspace
          const int64_t per = affd_small_bytes_per_vector(s);
          const int64_t vt = std::min<int64_t>(bc, std::max<int64_t>(1, s->ws_bytes / per));
          const int S = (int)std::min<int64_t>(kMaxPtrs, std::max<int64_t>(1, s->ws_bytes / (vt * per)));
          for (size_t i0 = 0; i0 < small.size(); i0 += S) {
            const int ns = (int)std::min<size_t>(S, small.size() - i0);
            SmallGroup g{};
            int64_t nsum = 0;
            for (int j = 0; j < ns; ++j) {
              g.layer[j] = small[i0 + j];
              g.x[j] = grads[small[i0 + j] - l0];
              g.gt[j] = s->d_gsmall ? s->d_gsmall + s->gsmall_off[small[i0 + j]] : nullptr;
              nsum += s->layers[small[i0 + j]].n;
            }
            for (int64_t t0 = b0; t0 < b0 + bc; t0 += vt) {
              const int64_t tb = std::min(vt, b0 + bc - t0);
              SK_PROF(SK_PROF_PROLOG, tb * nsum * esz, run_affd_small(s, g, ns, dtype, t0, tb, 1, out, acc_now, st));
              SK_PROF(SK_PROF_AFFD_FOLD, 0, run_affd_small(s, g, ns, dtype, t0, tb, 2, out, acc_now, st));
            }
            acc_now = true;
          }
        }
        break;
      }
      case SK_FJL:
        for (int l = l0; l < l1; ++l) {
          const LayerDesc &ld = s->layers[l];
          if (s->fjlb_pos_at[l] >= 0) {
            // one pass into 2^(lgnp - 13) partial slots, then their sum
            SK_PROF(SK_PROF_PROLOG, bc * ld.n * esz,
                    launch_fjl_fwd_onepass(s, l, grads[l - l0], dtype, b0, bc, s->ws, st));
            SK_PROF(SK_PROF_GATHER, (l == l1 - 1 ? bc * s->D * 4 : 0),
                    launch_reduce_partials(s->ws, 1ll << (ld.lgnp - 13), bc, s->D, b0, out, accumulate || l > l0, st));
            continue;
          }
          const int lgw = std::min(ld.lgnp, 13);  // fwht_inplace's first pass, fused with the signed load
          SK_PROF(SK_PROF_PROLOG, bc * ld.n * esz, launch_fjl_pass0(s, l, grads[l - l0], dtype, b0, bc, s->ws, lgw, st));
          if (ld.lgnp > 13) {
            // the middle passes, then the last one fused with the sample gather
            SK_PROF(SK_PROF_FWHT, 0, fwht_inplace_from_but_last(s->ws, bc, ld.lgnp, lgw, st));
            SK_PROF(SK_PROF_GATHER, (l == l1 - 1 ? bc * s->D * 4 : 0),
                    launch_fjl_last_gather(s, l, s->ws, b0, bc, out, accumulate || l > l0, st));
          } else {
            SK_PROF(SK_PROF_GATHER, (l == l1 - 1 ? bc * s->D * 4 : 0),
                    launch_fjl_gather(s, l, s->ws, b0, bc, out, accumulate || l > l0, st));
          }
        }
        break;
      case SK_FFD: {
        const int lgD = ilog2(s->D);
        for (int l = l0; l < l1; ++l) {
          if (lgD <= kFfdSmallMax) {
            const int64_t groups = ffd_small_groups(s, l);
            float *tab = s->ws + bc * groups * s->D;  // after the partial sums
            SK_PROF(SK_PROF_PROLOG, 0, launch_ffd_tables(s, l, tab, st));
            SK_PROF(SK_PROF_FFD, bc * s->layers[l].n * esz,
                    launch_ffd_small_fwd(s, l, grads[l - l0], dtype, b0, bc, s->ws, 0, groups, tab, st));
            SK_PROF(SK_PROF_GATHER, (l == l1 - 1 ? bc * s->D * 4 : 0),
                    launch_reduce_partials(s->ws, groups, bc, s->D, b0, out, accumulate || l > l0, st));
          } else if (ffd_large_path(s)) {
            SK_PROF(SK_PROF_PROLOG, bc * s->layers[l].n * esz,
                    run_ffd_large_fwd(s, l, grads[l - l0], dtype, b0, bc, out, accumulate || l > l0, 1, st));
            SK_PROF(SK_PROF_FFD, 0,
                    run_ffd_large_fwd(s, l, grads[l - l0], dtype, b0, bc, out, accumulate || l > l0, 2, st));
          } else {
            const int64_t nlive = ffd_live_blocks(s, l);
            float *w = s->ws, *w2 = s->ws + bc * nlive * s->D;
            SK_PROF(SK_PROF_PROLOG, bc * s->layers[l].n * esz,
                    launch_ffd_copy_blocks(s, l, grads[l - l0], dtype, b0, bc, w, st));
            SK_PROF(SK_PROF_FWHT, 0, fwht_inplace(w, bc * nlive, lgD, st));
            SK_PROF(SK_PROF_FFD, 0, launch_ffd_gperm_fwd(s, l, w, bc, w2, st));
            SK_PROF(SK_PROF_FWHT, 0, fwht_inplace(w2, bc * nlive, lgD, st));
            SK_PROF(SK_PROF_GATHER, (l == l1 - 1 ? bc * s->D * 4 : 0),
                    launch_ffd_sum_signed(s, l, w2, b0, bc, out, accumulate || l > l0, st));
          }
        }
        break;
      }
      case SK_QKH:
      case SK_AFJLQ: {
        // the Qt-first layers in groups (one launch per phase and group), then the others
        bool acc = accumulate != 0;
        const int ngr = qh_small_group_count(s, l0, l1);
        for (int gi = 0; gi < ngr; ++gi) {
          int64_t gb = 0;
          for (int l = l0; l < l1; ++l)
            if (qh_small_layer(s, l)) gb += bc * s->layers[l].n * esz;  // reported with the first group
          SK_PROF(SK_PROF_QH_FIRST, gi == 0 ? gb : 0,
                  run_qh_small_group(s, l0, l1, gi, grads, dtype, b0, bc, s->ws, out, acc, 1, st));
          SK_PROF(SK_PROF_QH_SECOND, 0, run_qh_small_group(s, l0, l1, gi, grads, dtype, b0, bc, s->ws, out, acc, 2, st));
          acc = true;
        }
        int last = -1;
        for (int l = l0; l < l1; ++l)
          if (!qh_small_layer(s, l)) last = l;
        for (int l = l0; l < l1; ++l) {
          if (qh_small_layer(s, l)) continue;
          SK_PROF(SK_PROF_QH_FIRST, bc * s->layers[l].n * esz,
                  run_qh_apply(s, l, grads[l - l0], dtype, b0, bc, s->ws, out, acc, 1, st));
          SK_PROF(SK_PROF_QH_SECOND, (l == last ? bc * s->D * 4 : 0),
                  run_qh_apply(s, l, grads[l - l0], dtype, b0, bc, s->ws, out, acc, 2, st));
          acc = true;
        }
        break;
      }
      case SK_AFJLF:
        run_afjlf_fwd(s, l0, l1, grads, dtype, b0, bc, s->ws, s->ws_bytes / 4, out, accumulate != 0, st);
        break;
      case SK_AFFDQ:
        for (int l = l0; l < l1; ++l) {
          const bool acc = accumulate || l > l0;
          SK_PROF(SK_PROF_QH_FIRST, bc * s->layers[l].n * esz,
                  run_affdq_apply(s, l, grads[l - l0], dtype, b0, bc, s->ws, out, acc, 1, st));
          SK_PROF(SK_PROF_QH_SECOND, (l == l1 - 1 ? bc * s->D * 4 : 0),
                  run_affdq_apply(s, l, grads[l - l0], dtype, b0, bc, s->ws, out, acc, 2, st));
        }
        break;
      case SK_QK:
        for (int l = l0; l < l1; ++l) {
          SK_PROF(SK_PROF_QK_XB, bc * s->layers[l].n * esz,
                  launch_qk_apply(s, l, grads[l - l0], dtype, b0, bc, s->ws, 1, out, accumulate != 0, st));
          SK_PROF(SK_PROF_QK, bc * s->layers[l].da * s->layers[l].db * 4,
                  launch_qk_apply(s, l, grads[l - l0], dtype, b0, bc, s->ws, 2, out, accumulate != 0, st));
        }
        break;
    }
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(SK_EHIP, std::string("kernel launch failed: ") + hipGetErrorString(e));
  return SK_OK;
}

// Allocation-free forward sketch: sketch_apply with the per-call scratch in
// the static device array below instead of the handle's workspace.
int sketch_apply_noalloc(sk_sketch *s, const void *const *grads, sk_dtype dtype, int64_t batch, float *out,
                         int32_t first_layer, int32_t n_layers, int32_t accumulate, void *stream) {
  if (!s) return fail(SK_EINVAL, "sketch is NULL");
  if (dtype != SK_F32 && dtype != SK_BF16) return fail(SK_EDTYPE, "dtype must be SK_F32 or SK_BF16");
  if (batch < 0) return fail(SK_EINVAL, "batch must be >= 0");
  if (int rc = check_range(s, first_layer, n_layers)) return rc;
  const int64_t pv = per_vector_bytes(s, first_layer, first_layer + n_layers, false);
  if (pv > kStaticScratchBytes)
    return fail(SK_EUNSUPPORTED, "one vector of these layers needs " + std::to_string(pv) +
                                     " bytes of scratch; the static scratch holds " +
                                     std::to_string(kStaticScratchBytes));
  DeviceGuard guard(s->device);
  void *p = nullptr;
  if (int rc = scratch_ptr(s->device, &p)) return rc;
  WorkspaceSwap swap(s, p, kStaticScratchBytes);
  return sketch_apply(s, grads, dtype, batch, out, first_layer, n_layers, accumulate, stream);
}

int sketch_apply_T(sk_sketch *s, const float *z, int64_t batch, void *const *out, sk_dtype out_dtype,
                   const void *const *theta0, int32_t first_layer, int32_t n_layers, void *stream) {
  if (!s) return fail(SK_EINVAL, "sketch is NULL");
  if (out_dtype != SK_F32 && out_dtype != SK_BF16) return fail(SK_EDTYPE, "out_dtype must be SK_F32 or SK_BF16");
  if (batch < 0) return fail(SK_EINVAL, "batch must be >= 0");
  if (int rc = check_range(s, first_layer, n_layers)) return rc;
  if (batch == 0) return SK_OK;
  if (!z || !out) return fail(SK_EINVAL, "z and out must be non-NULL");
  for (int i = 0; i < n_layers; ++i)
    if (!out[i]) return fail(SK_EINVAL, "out[" + std::to_string(i) + "] is NULL");
  const int l0 = first_layer, l1 = first_layer + n_layers;
  hipStream_t st = (hipStream_t)stream;
  DeviceGuard guard(s->device);
  const int64_t pv = per_vector_bytes(s, l0, l1, true);
  int64_t bcmax = pv > 0 ? s->ws_bytes / pv : batch;
  if (bcmax < 1) return fail(SK_EUNSUPPORTED, "workspace too small for one vector");
  if (s->kind == SK_AFJLF && bcmax > 8 && batch > bcmax) bcmax &= ~7ll;
  const int lgD = ilog2(s->D);
  const int osz = out_dtype == SK_BF16 ? 2 : 4;
  for (int64_t b0 = 0; b0 < batch; b0 += bcmax) {
    const int64_t bc = std::min(bcmax, batch - b0);
    if (s->kind == SK_AFJL) {
      // layer groups: as many layers per launch as the workspace holds (bc * D floats each)
      const int gmax = (int)std::max<int64_t>(1, std::min<int64_t>(kMaxPtrs, s->ws_bytes / (bc * s->D * 4)));
      for (int la = l0; la < l1; la += gmax) {
        const int ng = std::min(gmax, l1 - la);
        AfjlTGroup g{};
        int64_t obytes = 0;
        g.tile0[0] = 0;
        for (int i = 0; i < ng; ++i) {
          const LayerDesc &ld = s->layers[la + i];
          g.layer[i] = la + i;
          g.out[i] = out[la + i - l0];
          g.th[i] = theta0 ? (const float *)theta0[la + i - l0] : nullptr;
          g.tile0[i + 1] = g.tile0[i] + (ld.rows_live + kAfjlTRows - 1) / kAfjlTRows;
          obytes += bc * ld.n * osz + (g.th[i] ? ld.n * 4 : 0);
        }
        SK_PROF(SK_PROF_PROLOG, bc * s->D * 4, launch_afjl_T_prep(s, la, ng, z, b0, bc, s->ws, st));
        SK_PROF(SK_PROF_FWHT, 0, fwht_inplace(s->ws, (int64_t)ng * bc, lgD, st));
        SK_PROF(SK_PROF_GATHER, obytes, launch_afjl_T_out(s, g, ng, s->ws, b0, bc, out_dtype, st));
      }
      continue;
    }
    if (s->kind == SK_AFJLF) {
      run_afjlf_T(s, l0, l1, z, b0, bc, s->ws, s->ws_bytes / 4, out, out_dtype, theta0, st);
      continue;
    }
    for (int l = l0; l < l1; ++l) {
      const LayerDesc &ld = s->layers[l];
      void *o = out[l - l0];
      const float *th = theta0 ? (const float *)theta0[l - l0] : nullptr;
      const int64_t obytes = bc * ld.n * osz + (th ? ld.n * 4 : 0);  // output written, theta0 read
      switch (s->kind) {
        case SK_AFJL:  // grouped above
          break;
        case SK_AFFD:
          SK_PROF(SK_PROF_PROLOG, bc * s->D * 4, {
            launch_fill_zero(s->ws, bc * ld.np, st);
            launch_affd_T_scatter(s, l, z, b0, bc, s->ws, st);
          });
          SK_PROF(SK_PROF_FWHT, 0, fwht_inplace(s->ws, bc, ld.lgnp, st));
          SK_PROF(SK_PROF_OTHER, 0, launch_mul_gauss(s, l, s->ws, bc, st));
          SK_PROF(SK_PROF_FWHT, 0, fwht_inplace(s->ws, bc, ld.lgnp, st));
          SK_PROF(SK_PROF_GATHER, obytes, launch_affd_T_out(s, l, s->ws, b0, bc, o, out_dtype, th, st));
          break;
        case SK_FJL: {
          if (s->fjlb_off_at[l] >= 0) {
            SK_PROF(SK_PROF_FJL_T, obytes + bc * s->D * 4,
                    launch_fjl_T_onepass(s, l, z, b0, bc, o, out_dtype, th, st));
            break;
          }
          const int lgw = std::min(ld.lgnp, 13);  // fwht_inplace's first pass, fused with the scatter
          const float oscale = (float)std::sqrt((double)ld.np / (double)s->D);
          SK_PROF(SK_PROF_PROLOG, bc * s->D * 4, launch_fjl_T_pass0(s, l, z, b0, bc, s->ws, lgw, st));
          if (fjl_last_signed_ok(s, l, lgw)) {
            // the remaining passes, the last one writing the signed output
            SK_PROF(SK_PROF_FWHT, 0, fwht_inplace_from_but_last(s->ws, bc, ld.lgnp, lgw, st));
            SK_PROF(SK_PROF_GATHER, obytes,
                    launch_fjl_last_signed(s, l, s->ws, lgw, b0, bc, o, out_dtype, th, oscale, st));
          } else {
            SK_PROF(SK_PROF_FWHT, 0, fwht_inplace_from(s->ws, bc, ld.lgnp, lgw, st));
            SK_PROF(SK_PROF_GATHER, obytes, launch_signed_out(s, l, s->ws, b0, bc, o, out_dtype, th, oscale, st));
          }
          break;
        }
        case SK_FFD:
          if (lgD <= kFfdSmallMax) {
            SK_PROF(SK_PROF_PROLOG, 0, launch_ffd_tables(s, l, s->ws, st));
            SK_PROF(SK_PROF_FFD_T, obytes + bc * s->D * 4,
                    launch_ffd_small_T(s, l, z, b0, bc, o, out_dtype, th, s->ws, st));
          } else if (ffd_large_path(s)) {
            SK_PROF(SK_PROF_FFD, 0, run_ffd_large_T(s, l, z, b0, bc, o, out_dtype, th, 1, st));
            SK_PROF(SK_PROF_GATHER, obytes + bc * s->D * 4, run_ffd_large_T(s, l, z, b0, bc, o, out_dtype, th, 2, st));
          } else {
            const int64_t nlive = ffd_live_blocks(s, l);
            float *w = s->ws, *w2 = s->ws + bc * nlive * s->D;
            SK_PROF(SK_PROF_PROLOG, bc * s->D * 4, launch_ffd_expand_z(s, l, z, b0, bc, w, st));
            SK_PROF(SK_PROF_FWHT, 0, fwht_inplace(w, bc * nlive, lgD, st));
            SK_PROF(SK_PROF_FFD, 0, launch_ffd_permg_T(s, l, w, bc, w2, st));
            SK_PROF(SK_PROF_FWHT, 0, fwht_inplace(w2, bc * nlive, lgD, st));
            SK_PROF(SK_PROF_GATHER, obytes, launch_ffd_T_out(s, l, w2, b0, bc, o, out_dtype, th, st));
          }
          break;
        case SK_QKH:
        case SK_AFJLQ:
          SK_PROF(SK_PROF_QH_T, obytes, run_qh_apply_T(s, l, z, b0, bc, s->ws, o, out_dtype, th, st));
          break;
        case SK_AFFDQ:
          SK_PROF(SK_PROF_QH_T, obytes, run_affdq_apply_T(s, l, z, b0, bc, s->ws, o, out_dtype, th, st));
          break;
        case SK_QK:
          SK_PROF(SK_PROF_QK, obytes + bc * ld.da * ld.db * 4,
                  launch_qk_apply_T(s, l, z, b0, bc, s->ws, o, out_dtype, th, st));
          break;
      }
    }
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(SK_EHIP, std::string("kernel launch failed: ") + hipGetErrorString(e));
  return SK_OK;
}

int sketch_profile(sk_sketch *s, uint32_t classes) {
  if (!s) return fail(SK_EINVAL, "sketch is NULL");
  if (classes & ~(uint32_t)SK_PROF_ALL) return fail(SK_EINVAL, "unknown kernel class in profiling mask");
  DeviceGuard guard(s->device);
  if (classes) {
    if (s->evpool.empty()) {
      s->evpool.resize(2 * 16384);
      for (auto &e : s->evpool) SK_HIP(hipEventCreate(&e));
    }
    s->evnext = 0;
    s->recs.clear();
  }
  s->prof_mask = classes;
  return SK_OK;
}

int sketch_profile_read(sk_sketch *s, double *ms, int64_t *count, int64_t *bytes) {
  if (!s || !ms || !count || !bytes) return fail(SK_EINVAL, "NULL argument");
  DeviceGuard guard(s->device);
  for (int c = 0; c < SK_PROF_CLASSES; ++c) {
    ms[c] = 0.0;
    count[c] = 0;
    bytes[c] = 0;
  }
  for (const auto &r : s->recs) {
    SK_HIP(hipEventSynchronize(s->evpool[r.ev + 1]));
    float t = 0.0f;
    SK_HIP(hipEventElapsedTime(&t, s->evpool[r.ev], s->evpool[r.ev + 1]));
    ms[r.cls] += t;
    count[r.cls] += 1;
    bytes[r.cls] += r.bytes;
  }
  s->recs.clear();
  s->evnext = 0;
  return SK_OK;
}

int sketch_debug_stream(sk_sketch *s, int32_t layer, int32_t stream_id, uint64_t start, uint64_t count, uint64_t aux,
                        void *host_out) {
  if (!s || !host_out) return fail(SK_EINVAL, "NULL argument");
  if (layer < 0 || layer >= (int32_t)s->layers.size()) return fail(SK_EINVAL, "layer out of range");
  if (count == 0) return SK_OK;
  const LayerDesc &ld = s->layers[layer];
  size_t esz = 4;
  uint64_t limit = ~0ull;
  switch (stream_id) {
    case SK_STREAM_SIGN:
      esz = 1;
      limit = fwht_kind(s->kind) ? (uint64_t)ld.np : ~0ull;
      break;
    case SK_STREAM_GAUSS:
    case SK_STREAM_QKA:
    case SK_STREAM_QKB:
      break;
    case SK_STREAM_INDEX:
      if (!fwht_kind(s->kind)) return fail(SK_EINVAL, "index stream needs an FWHT kind");
      limit = (uint64_t)s->D;
      break;
    case SK_STREAM_PI1:
    case SK_STREAM_PI2:
      if (!(s->kind == SK_AFJL || s->kind == SK_AFFD) || (stream_id == SK_STREAM_PI2 && s->kind != SK_AFFD))
        return fail(SK_EINVAL, "this sketch has no such permutation");
      limit = (uint64_t)ld.np;
      break;
    case SK_STREAM_FFDPERM:
      if (s->kind != SK_FFD) return fail(SK_EINVAL, "FFD permutations need an FFD sketch");
      limit = (uint64_t)s->D;
      break;
    default:
      return fail(SK_EINVAL, "unknown stream id");
  }
  if (start > limit || count > limit - start) return fail(SK_EINVAL, "index range out of bounds");
  DeviceGuard guard(s->device);
  void *d = nullptr;
  SK_HIP(hipMalloc(&d, count * esz));
  launch_debug_stream(s, layer, stream_id, start, count, aux, d, nullptr);
  hipError_t e = hipMemcpy(host_out, d, count * esz, hipMemcpyDeviceToHost);
  (void)hipFree(d);
  if (e != hipSuccess) return fail(SK_EHIP, std::string("debug stream: ") + hipGetErrorString(e));
  return SK_OK;
}

}  // extern "C"
