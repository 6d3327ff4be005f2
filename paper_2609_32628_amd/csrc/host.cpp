// Host side of libda2: argument validation, buffer sizes and offsets, the region
// layout and the four stream-ordered entry points. Validation never touches the
// GPU, so every error path can be exercised on a machine without one.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <vector>

#include "../../include/da2.h"
#include "launch.hpp"

namespace {

constexpr int64_t kAlign = 256;
inline int64_t align_up(int64_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Dims {
  int64_t B, H, d, T, Hg, Wg, N, R, Npad, BH;
  int64_t Rf;  // blocks per frame
  int32_t partition;
};

int32_t derive(const da2_problem* p, Dims* o) {
  if (!p) return DA2_ERR_INVALID_ARG;
  if (p->B <= 0 || p->H <= 0 || p->T <= 0 || p->Hg <= 0 || p->Wg <= 0 || p->d <= 0) return DA2_ERR_INVALID_ARG;
  if (p->partition != DA2_PART_TILES8 && p->partition != DA2_PART_RAGGED) return DA2_ERR_INVALID_ARG;
  if (p->d != 64 && p->d != 128) return DA2_ERR_UNSUPPORTED;  // a valid head dim the kernels do not implement
  Dims d{};
  d.B = p->B;
  d.H = p->H;
  d.d = p->d;
  d.T = p->T;
  d.Hg = p->Hg;
  d.Wg = p->Wg;
  d.N = d.T * d.Hg * d.Wg;
  d.partition = p->partition;
  d.Rf = d.partition == DA2_PART_TILES8 ? ((d.Hg + 7) / 8) * ((d.Wg + 7) / 8) : (d.Hg * d.Wg + 63) / 64;
  d.R = d.T * d.Rf;
  d.Npad = 64 * d.R;
  d.BH = d.B * d.H;
  // launch grids put R and 2*B*H in 16-bit grid dimensions
  if (d.R > 65535 || d.BH > 32767 || d.N > (1ll << 31) - 1 || d.BH * d.R > (1ll << 31) - 1)
    return DA2_ERR_INVALID_ARG;
  *o = d;
  return DA2_OK;
}

// MXFP4 section bytes per block: d/32 data fragments and one scale fragment of 1 KB.
inline int64_t mx_block_bytes(const Dims& d) { return 1024 * (d.d / 32 + 1); }

constexpr int kSections = 16;

// Byte size of each ops section (the index numbering of da2_ops_offsets).
void section_sizes(const Dims& d, int64_t* sz) {
  const int64_t e = d.BH * d.Npad * d.d;                       // values per operand
  const int64_t nv = da2::nv_block_bytes((int)d.d) * d.BH * d.R;  // packed NVFP4 operand
  const int64_t mx = mx_block_bytes(d) * d.BH * d.R;
  const int64_t v[kSections] = {nv, nv, nv, e, e, e, 4 * d.BH * d.R, 4 * d.BH * d.R, 4 * d.BH * d.d, 16 * d.BH,
                                2 * e, 2 * e, 2 * e, mx, mx, mx};
  for (int i = 0; i < kSections; ++i) sz[i] = v[i];
}

// Offsets of the sections a run with (fmt4, with16) writes and reads, -1 for
// the others: the 8-bit operands and all scales [3..9] first, then the 4-bit
// encoding in use ([0..2] NVFP4 or [13..15] MXFP4), then the 16-bit operands
// [10..12] when with16, so that no offset but the 16-bit ones depends on
// with16. Returns the total size.
int64_t ops_offsets(const Dims& d, int32_t fmt4, int32_t with16, int64_t* off) {
  int64_t sz[kSections];
  section_sizes(d, sz);
  for (int i = 0; i < kSections; ++i) off[i] = -1;
  const int nv[] = {3, 4, 5, 6, 7, 8, 9, 0, 1, 2, 10, 11, 12};
  const int mx[] = {3, 4, 5, 6, 7, 8, 9, 13, 14, 15, 10, 11, 12};
  const int* order = fmt4 == DA2_FMT4_MXFP4 ? mx : nv;
  const int n = with16 ? 13 : 10;
  int64_t o = 0;
  for (int k = 0; k < n; ++k) {
    off[order[k]] = o;
    o += align_up(sz[order[k]]);
  }
  return o;
}

void sizes_of(const Dims& d, int32_t scope, int32_t fmt4, int32_t with16, da2_sizes_t* s) {
  std::memset(s, 0, sizeof(*s));
  s->R = (int32_t)d.R;
  s->Npad = (int32_t)d.Npad;
  s->layout_bytes = 4 * (d.R + d.Npad + d.N);
  s->A_bytes = 4 * d.BH * d.R * d.R;
  s->cls_bytes = d.BH * d.R * d.R;
  s->stats_bytes = 4 * d.BH * (4 + d.d);
  s->lists_bytes = align_up(2 * d.BH * d.R * d.R) + align_up(16 * d.BH * d.R) + align_up(4 * d.BH * d.R) + kAlign;
  int64_t off[kSections];
  s->ops_bytes = ops_offsets(d, fmt4, with16, off);
  s->ws_draft_bytes = 4 * align_up(8 * d.BH * d.R * d.d) + 2 * align_up(8 * d.BH * d.R * d.R) + align_up(8 * d.BH * d.R);
  int64_t thr = scope == DA2_SCOPE_ROW ? 8 * da2::kCuts * d.BH * d.R : 8 * da2::kCuts * d.BH;
  s->ws_rank_bytes = align_up(4 * d.BH * da2::kCuts * 2048) + align_up(thr) + align_up(8 * da2::kCuts * d.BH) +
                     align_up(8 * da2::kCuts * d.BH) + align_up(4 * d.BH * d.R) +
                     align_up(8 * d.BH * da2::kCuts * da2::kRankCand) + align_up(4 * d.BH * da2::kCuts);
  s->ws_prep_bytes = 0;
}

bool fmt_ok(int32_t fmt4, int32_t with16) {
  return (fmt4 == DA2_FMT4_NVFP4 || fmt4 == DA2_FMT4_MXFP4) && (with16 == 0 || with16 == 1);
}

void lists_offsets(const Dims& d, int64_t* off) {
  off[0] = 0;
  off[1] = align_up(2 * d.BH * d.R * d.R);
  off[2] = off[1] + align_up(16 * d.BH * d.R);
  off[3] = off[2] + align_up(4 * d.BH * d.R);
}

void draft_offsets(const Dims& d, int64_t* off) {
  const int64_t pooled = align_up(8 * d.BH * d.R * d.d), logits = align_up(8 * d.BH * d.R * d.R);
  for (int i = 0; i < 4; ++i) off[i] = i * pooled;
  off[4] = 4 * pooled;
  off[5] = 4 * pooled + logits;
  off[6] = 4 * pooled + 2 * logits;
}

int32_t check_tensor(const da2_tensor* t, const Dims& d, bool out) {
  if (!t) return DA2_ERR_INVALID_ARG;
  if (t->dtype != DA2_BF16 && t->dtype != DA2_FP32) return DA2_ERR_INVALID_ARG;
  if (t->stride_b <= 0 || t->stride_h <= 0 || t->stride_n <= 0) return DA2_ERR_INVALID_ARG;
  if (t->stride_n < d.d) return DA2_ERR_INVALID_ARG;
  if (!out) {  // inputs are read in 16-byte vectors
    const int64_t per = t->dtype == DA2_BF16 ? 8 : 4;
    if (t->stride_b % per || t->stride_h % per || t->stride_n % per) return DA2_ERR_INVALID_ARG;
  }
  return DA2_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// gfx950 check, cached per device ordinal (0 unknown, 1 ok, 2 unsupported).
std::atomic<int8_t> g_arch_ok[64];

int32_t check_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return DA2_ERR_UNSUPPORTED;
  if (dev < 64) {
    int8_t c = g_arch_ok[dev].load(std::memory_order_relaxed);
    if (c == 1) return DA2_OK;
    if (c == 2) return DA2_ERR_UNSUPPORTED;
  }
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return DA2_ERR_HIP;
  const bool ok = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
  if (dev < 64) g_arch_ok[dev].store(ok ? 1 : 2, std::memory_order_relaxed);
  return ok ? DA2_OK : DA2_ERR_UNSUPPORTED;
}

int32_t hip_status(hipError_t e) { return e == hipSuccess ? DA2_OK : DA2_ERR_HIP; }

// Ragged partition of one H x W frame (the candidate family documented in
// da2.h): the label of every cell, row-major.
std::vector<int32_t> ragged_frame_labels(int64_t H, int64_t W) {
  constexpr int64_t C = 64;
  const int64_t Rf = (H * W + C - 1) / C;
  std::vector<int32_t> best, cand(H * W);
  int64_t best_key[3] = {0, 0, 0};
  for (int orient = 0; orient < 2; ++orient) {
    // bands split the first axis of the (h, w) view; orient 1 is the transposed frame
    const int64_t h = orient == 0 ? H : W, w = orient == 0 ? W : H;
    for (int64_t nb = 1; nb <= h; ++nb) {
      int64_t runs = 0;
      for (int64_t i = 0; i < nb; ++i) runs += ((h / nb + (i < h % nb ? 1 : 0)) * w + C - 1) / C;
      if (runs != Rf) continue;
      int64_t y0 = 0, label = 0;
      for (int64_t i = 0; i < nb; ++i) {
        const int64_t hb = h / nb + (i < h % nb ? 1 : 0), n = hb * w, r = (n + C - 1) / C;
        int64_t k = 0, used = 0, size = n / r + (0 < n % r ? 1 : 0);
        for (int64_t c = 0; c < w; ++c)
          for (int64_t q = 0; q < hb; ++q) {
            const int64_t yy = y0 + (c % 2 == 0 ? q : hb - 1 - q);  // snake down / up the column
            const int64_t idx = orient == 0 ? yy * W + c : c * W + yy;
            cand[idx] = (int32_t)(label + k);
            if (++used == size && k + 1 < r) {
              ++k;
              used = 0;
              size = n / r + (k < n % r ? 1 : 0);
            }
          }
        y0 += hb;
        label += r;
      }
      int64_t cut = 0;
      for (int64_t y = 0; y < H; ++y)
        for (int64_t x = 0; x < W; ++x) {
          if (x + 1 < W && cand[y * W + x] != cand[y * W + x + 1]) ++cut;
          if (y + 1 < H && cand[y * W + x] != cand[(y + 1) * W + x]) ++cut;
        }
      const int64_t key[3] = {cut, orient, nb};
      if (best.empty() || std::lexicographical_compare(key, key + 3, best_key, best_key + 3)) {
        best = cand;
        std::copy(key, key + 3, best_key);
      }
    }
  }
  return best;
}

}  // namespace

extern "C" {

const char* da2_status_string(int32_t s) {
  switch (s) {
    case DA2_OK: return "DA2_OK";
    case DA2_ERR_INVALID_ARG: return "DA2_ERR_INVALID_ARG: invalid argument";
    case DA2_ERR_UNSUPPORTED: return "DA2_ERR_UNSUPPORTED: unsupported request or device (gfx950 required)";
    case DA2_ERR_WORKSPACE: return "DA2_ERR_WORKSPACE: workspace too small";
    case DA2_ERR_HIP: return "DA2_ERR_HIP: HIP runtime error";
    default: return "DA2 unknown status";
  }
}

int32_t da2_sizes(const da2_problem* p, int32_t scope, int32_t fmt4, int32_t with16, da2_sizes_t* out) {
  Dims d;
  int32_t st = derive(p, &d);
  if (st) return st;
  if (!out || (scope != DA2_SCOPE_HEAD && scope != DA2_SCOPE_ROW) || !fmt_ok(fmt4, with16)) return DA2_ERR_INVALID_ARG;
  sizes_of(d, scope, fmt4, with16, out);
  return DA2_OK;
}

int32_t da2_ops_layout_version(void) { return DA2_OPS_LAYOUT_VERSION; }

int32_t da2_ws_draft_offsets(const da2_problem* p, int64_t* off) {
  Dims d;
  int32_t st = derive(p, &d);
  if (st) return st;
  if (!off) return DA2_ERR_INVALID_ARG;
  draft_offsets(d, off);
  return DA2_OK;
}

int32_t da2_lists_offsets(const da2_problem* p, int64_t* off) {
  Dims d;
  int32_t st = derive(p, &d);
  if (st) return st;
  if (!off) return DA2_ERR_INVALID_ARG;
  lists_offsets(d, off);
  return DA2_OK;
}

int32_t da2_ops_offsets(const da2_problem* p, int32_t fmt4, int32_t with16, int64_t* off) {
  Dims d;
  int32_t st = derive(p, &d);
  if (st) return st;
  if (!off || !fmt_ok(fmt4, with16)) return DA2_ERR_INVALID_ARG;
  ops_offsets(d, fmt4, with16, off);
  return DA2_OK;
}

int32_t da2_layout_build(const da2_problem* p, int32_t* L, int64_t n_ints) {
  Dims d;
  int32_t st = derive(p, &d);
  if (st) return st;
  if (!L || n_ints < d.R + d.Npad + d.N) return DA2_ERR_INVALID_ARG;
  // region label of every cell of a frame
  std::vector<int32_t> lab;
  if (d.partition == DA2_PART_TILES8) {
    const int64_t nJ = (d.Wg + 7) / 8;
    lab.resize(d.Hg * d.Wg);
    for (int64_t y = 0; y < d.Hg; ++y)
      for (int64_t x = 0; x < d.Wg; ++x) lab[y * d.Wg + x] = (int32_t)((y / 8) * nJ + x / 8);
  } else {
    lab = ragged_frame_labels(d.Hg, d.Wg);
  }
  int32_t* n_a = L;
  int32_t* s2t = L + d.R;
  int32_t* t2s = L + d.R + d.Npad;
  for (int64_t i = 0; i < d.Npad; ++i) s2t[i] = -1;
  for (int64_t a = 0; a < d.R; ++a) n_a[a] = 0;
  for (int64_t t = 0; t < d.T; ++t)
    for (int64_t y = 0; y < d.Hg; ++y)  // row-major, so each block's slots come out row-major
      for (int64_t x = 0; x < d.Wg; ++x) {
        const int64_t a = t * d.Rf + lab[y * d.Wg + x];
        const int64_t tok = t * d.Hg * d.Wg + y * d.Wg + x;
        const int64_t slot = a * 64 + n_a[a]++;
        s2t[slot] = (int32_t)tok;
        t2s[tok] = (int32_t)slot;
      }
  return DA2_OK;
}

int32_t da2_draft_map(const void* Q, const void* K, const da2_tensor* qk, const int32_t* layout,
                      const da2_problem* p, double lambda, float* A, void* stats, void* ws, int64_t ws_bytes,
                      void* stream) {
  Dims d;
  int32_t st = derive(p, &d);
  if (st) return st;
  if ((st = check_tensor(qk, d, false))) return st;
  if (!Q || !K || !layout || !A || !stats || !ws) return DA2_ERR_INVALID_ARG;
  if (!aligned16(Q) || !aligned16(K)) return DA2_ERR_INVALID_ARG;
  if (!(lambda >= 0.0 && lambda <= 1.0)) return DA2_ERR_INVALID_ARG;
  da2_sizes_t sz;
  sizes_of(d, DA2_SCOPE_HEAD, DA2_FMT4_NVFP4, 0, &sz);
  if (ws_bytes < sz.ws_draft_bytes) return DA2_ERR_WORKSPACE;
  if ((st = check_device())) return st;
  int64_t off[7];
  draft_offsets(d, off);
  char* w = static_cast<char*>(ws);
  da2::DraftArgs a{};
  a.Q = Q;
  a.K = K;
  a.sb = qk->stride_b;
  a.sh = qk->stride_h;
  a.sn = qk->stride_n;
  a.dtype = qk->dtype;
  a.B = (int)d.B;
  a.H = (int)d.H;
  a.d = (int)d.d;
  a.R = (int)d.R;
  a.Npad = (int)d.Npad;
  a.layout = layout;
  a.lambda = lambda;
  a.A = A;
  a.stats = static_cast<uint32_t*>(stats);
  a.Qbar = reinterpret_cast<double*>(w + off[0]);
  a.Qmax = reinterpret_cast<double*>(w + off[1]);
  a.Kbar = reinterpret_cast<double*>(w + off[2]);
  a.Kmax = reinterpret_cast<double*>(w + off[3]);
  a.S1 = reinterpret_cast<double*>(w + off[4]);
  a.S2 = reinterpret_cast<double*>(w + off[5]);
  a.blkmax = reinterpret_cast<float*>(w + off[6]);
  return hip_status(da2::launch_draft(a, static_cast<hipStream_t>(stream)));
}

}  // extern "C"

namespace {

// Validation shared by both ranking entry points (everything but the workspace).
int32_t rank_check(const float* A, const da2_problem* p, int32_t num16, int32_t num8, int32_t num4, int32_t den,
                   int32_t scope, const uint8_t* cls, const void* lists, Dims* d) {
  int32_t st = derive(p, d);
  if (st) return st;
  if (!A || !cls || !lists) return DA2_ERR_INVALID_ARG;
  if (den <= 0 || num16 < 0 || num8 < 0 || num4 < 0 || (int64_t)num16 + num8 + num4 > den)
    return DA2_ERR_INVALID_ARG;
  if (scope != DA2_SCOPE_HEAD && scope != DA2_SCOPE_ROW) return DA2_ERR_INVALID_ARG;
  if (scope == DA2_SCOPE_HEAD && d->R * d->R >= (1ll << 22)) return DA2_ERR_INVALID_ARG;
  if (scope == DA2_SCOPE_ROW && d->R > 8192) return DA2_ERR_UNSUPPORTED;
  return DA2_OK;
}

// The ranking launch on a validated problem with workspace ws (at least
// ws_rank_bytes, 256-byte aligned).
int32_t rank_launch(const float* A, const Dims& d, int32_t num16, int32_t num8, int32_t num4, int32_t den,
                    int32_t scope, uint8_t* cls, void* lists, void* ws, void* stream) {
  const int64_t M = scope == DA2_SCOPE_HEAD ? d.R * d.R : d.R;
  // cumulative quotas, rounded half up: ranks [0, cut0) -> 16, [cut0, cut1) -> 8, [cut1, cut2) -> 4
  auto half_up = [&](int64_t num) { return (2 * num * M + den) / (2 * (int64_t)den); };
  int64_t lo[4];
  lists_offsets(d, lo);
  char* lb = static_cast<char*>(lists);
  char* w = static_cast<char*>(ws);
  int64_t thr = scope == DA2_SCOPE_ROW ? 8 * da2::kCuts * d.BH * d.R : 8 * da2::kCuts * d.BH;
  da2::RankArgs a{};
  a.A = A;
  a.B = (int)d.B;
  a.H = (int)d.H;
  a.R = (int)d.R;
  a.scope = scope;
  a.cut[0] = half_up(num16);
  a.cut[1] = half_up((int64_t)num16 + num8);
  a.cut[2] = half_up((int64_t)num16 + num8 + num4);
  a.cls = cls;
  a.keys = reinterpret_cast<uint16_t*>(lb + lo[0]);
  a.counts = reinterpret_cast<int32_t*>(lb + lo[1]);
  a.order = reinterpret_cast<int32_t*>(lb + lo[2]);
  a.meta = reinterpret_cast<int32_t*>(lb + lo[3]);
  int64_t o = 0;
  a.hist = reinterpret_cast<uint32_t*>(w + o);
  o += align_up(4 * d.BH * da2::kCuts * 2048);
  a.thr = reinterpret_cast<uint64_t*>(w + o);
  o += align_up(thr);
  a.prefix = reinterpret_cast<uint64_t*>(w + o);
  o += align_up(8 * da2::kCuts * d.BH);
  a.kleft = reinterpret_cast<int64_t*>(w + o);
  o += align_up(8 * da2::kCuts * d.BH);
  a.cost = reinterpret_cast<int32_t*>(w + o);
  o += align_up(4 * d.BH * d.R);
  a.cand = reinterpret_cast<uint64_t*>(w + o);
  o += align_up(8 * d.BH * da2::kCuts * da2::kRankCand);
  a.ccount = reinterpret_cast<uint32_t*>(w + o);
  return hip_status(da2::launch_rank(a, static_cast<hipStream_t>(stream)));
}

}  // namespace

extern "C" {

int32_t da2_rank_assign(const float* A, const da2_problem* p, int32_t num16, int32_t num8, int32_t num4,
                        int32_t den, int32_t scope, uint8_t* cls, void* lists, void* ws, int64_t ws_bytes,
                        void* stream) {
  Dims d;
  int32_t st = rank_check(A, p, num16, num8, num4, den, scope, cls, lists, &d);
  if (st) return st;
  if (!ws) return DA2_ERR_INVALID_ARG;
  da2_sizes_t sz;
  sizes_of(d, scope, DA2_FMT4_NVFP4, 0, &sz);
  if (ws_bytes < sz.ws_rank_bytes) return DA2_ERR_WORKSPACE;
  if ((st = check_device())) return st;
  return rank_launch(A, d, num16, num8, num4, den, scope, cls, lists, ws, stream);
}

int32_t da2_rank_assign_noalloc(const float* A, const da2_problem* p, int32_t num16, int32_t num8, int32_t num4,
                                int32_t den, int32_t scope, uint8_t* cls, void* lists, void* stream) {
  Dims d;
  int32_t st = rank_check(A, p, num16, num8, num4, den, scope, cls, lists, &d);
  if (st) return st;
  da2_sizes_t sz;
  sizes_of(d, scope, DA2_FMT4_NVFP4, 0, &sz);
  static_assert(da2::kRankScratchBytes == DA2_RANK_NOALLOC_MAX_BYTES, "header limit and scratch size agree");
  if (sz.ws_rank_bytes > da2::kRankScratchBytes) return DA2_ERR_WORKSPACE;
  if ((st = check_device())) return st;
  void* ws = nullptr;
  if (da2::rank_scratch_address(&ws) != hipSuccess) return DA2_ERR_HIP;
  return rank_launch(A, d, num16, num8, num4, den, scope, cls, lists, ws, stream);
}

int32_t da2_prep_operands(const void* Q, const void* K, const void* V, const da2_tensor* qkv, const int32_t* layout,
                          const da2_problem* p, int32_t with16, int32_t fmt4, void* stats, void* ops,
                          int64_t ops_bytes, void* ws, int64_t ws_bytes, void* stream) {
  Dims d;
  int32_t st = derive(p, &d);
  if (st) return st;
  if ((st = check_tensor(qkv, d, false))) return st;
  if (!Q || !K || !V || !layout || !stats || !ops) return DA2_ERR_INVALID_ARG;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V)) return DA2_ERR_INVALID_ARG;
  if (!fmt_ok(fmt4, with16)) return DA2_ERR_INVALID_ARG;
  (void)ws;
  if (ws_bytes < 0) return DA2_ERR_WORKSPACE;
  int64_t off[kSections];
  if (ops_bytes < ops_offsets(d, fmt4, with16, off)) return DA2_ERR_INVALID_ARG;
  if ((st = check_device())) return st;
  char* ob = static_cast<char*>(ops);
  // sections this run does not write get no pointer (the kernels skip them)
  auto sec = [&](int i) -> char* { return off[i] < 0 ? nullptr : ob + off[i]; };
  da2::PrepArgs a{};
  a.with16 = with16;
  a.fmt4 = fmt4;
  a.Q = Q;
  a.K = K;
  a.V = V;
  a.sb = qkv->stride_b;
  a.sh = qkv->stride_h;
  a.sn = qkv->stride_n;
  a.dtype = qkv->dtype;
  a.B = (int)d.B;
  a.H = (int)d.H;
  a.d = (int)d.d;
  a.R = (int)d.R;
  a.Npad = (int)d.Npad;
  a.N = (int)d.N;
  a.layout = layout;
  a.stats = static_cast<uint32_t*>(stats);
  a.Q4 = reinterpret_cast<uint8_t*>(sec(0));
  a.K4 = reinterpret_cast<uint8_t*>(sec(1));
  a.V4 = reinterpret_cast<uint8_t*>(sec(2));
  a.Q8 = reinterpret_cast<int8_t*>(sec(3));
  a.K8 = reinterpret_cast<int8_t*>(sec(4));
  a.V8 = reinterpret_cast<uint8_t*>(sec(5));
  a.dQ = reinterpret_cast<float*>(sec(6));
  a.dK = reinterpret_cast<float*>(sec(7));
  a.dV = reinterpret_cast<float*>(sec(8));
  a.g = reinterpret_cast<float*>(sec(9));
  a.Q16 = reinterpret_cast<_Float16*>(sec(10));
  a.K16 = reinterpret_cast<_Float16*>(sec(11));
  a.V16 = reinterpret_cast<_Float16*>(sec(12));
  a.Q4mx = reinterpret_cast<uint8_t*>(sec(13));
  a.K4mx = reinterpret_cast<uint8_t*>(sec(14));
  a.V4mx = reinterpret_cast<uint8_t*>(sec(15));
  a.tag = da2::ops_tag(fmt4, with16);
  return hip_status(da2::launch_prep(a, static_cast<hipStream_t>(stream)));
}

int32_t da2_mixed_attn(const void* ops, int64_t ops_bytes, const void* lists, const int32_t* layout,
                       const da2_problem* p, int32_t fmt4, const da2_tensor* out, void* O, void* stream) {
  Dims d;
  int32_t st = derive(p, &d);
  if (st) return st;
  if ((st = check_tensor(out, d, true))) return st;
  if (!ops || !lists || !layout || !O) return DA2_ERR_INVALID_ARG;
  if (fmt4 != DA2_FMT4_NVFP4 && fmt4 != DA2_FMT4_MXFP4) return DA2_ERR_INVALID_ARG;
  int64_t off[kSections], lo[4];
  // at least the sections of a run without the 16-bit path; the 16-bit
  // sections are read only when the buffer holds them too
  if (ops_bytes < ops_offsets(d, fmt4, 0, off)) return DA2_ERR_INVALID_ARG;
  const bool has16 = ops_bytes >= ops_offsets(d, fmt4, 1, off);
  if ((st = check_device())) return st;
  // the 16-bit sections come last, so the other offsets do not depend on
  // with16; the kernel reads the 16-bit ones only when a row holds 16-bit
  // blocks and the operands' tag says they were written
  ops_offsets(d, fmt4, 1, off);
  lists_offsets(d, lo);
  const char* ob = static_cast<const char*>(ops);
  auto sec = [&](int i) -> const char* { return off[i] < 0 ? nullptr : ob + off[i]; };
  const char* lb = static_cast<const char*>(lists);
  da2::AttnArgs a{};
  a.Q4 = reinterpret_cast<const uint8_t*>(sec(0));
  a.K4 = reinterpret_cast<const uint8_t*>(sec(1));
  a.V4 = reinterpret_cast<const uint8_t*>(sec(2));
  a.Q8 = reinterpret_cast<const int8_t*>(sec(3));
  a.K8 = reinterpret_cast<const int8_t*>(sec(4));
  a.V8 = reinterpret_cast<const uint8_t*>(sec(5));
  a.dQ = reinterpret_cast<const float*>(sec(6));
  a.dK = reinterpret_cast<const float*>(sec(7));
  a.dV = reinterpret_cast<const float*>(sec(8));
  a.g = reinterpret_cast<const float*>(sec(9));
  a.Q16 = reinterpret_cast<const _Float16*>(sec(10));
  a.K16 = reinterpret_cast<const _Float16*>(sec(11));
  a.V16 = reinterpret_cast<const _Float16*>(sec(12));
  a.Q4mx = reinterpret_cast<const uint8_t*>(sec(13));
  a.K4mx = reinterpret_cast<const uint8_t*>(sec(14));
  a.V4mx = reinterpret_cast<const uint8_t*>(sec(15));
  a.tag = da2::ops_tag(fmt4, 0);
  a.has16 = has16 ? 1 : 0;
  a.meta = reinterpret_cast<int32_t*>(const_cast<char*>(lb) + lo[3]);
  a.fmt4 = fmt4;
  a.keys = reinterpret_cast<const uint16_t*>(lb + lo[0]);
  a.counts = reinterpret_cast<const int32_t*>(lb + lo[1]);
  a.order = reinterpret_cast<const int32_t*>(lb + lo[2]);
  a.layout = layout;
  a.B = (int)d.B;
  a.H = (int)d.H;
  a.d = (int)d.d;
  a.R = (int)d.R;
  a.Npad = (int)d.Npad;
  a.O = O;
  a.ob = out->stride_b;
  a.oh = out->stride_h;
  a.on = out->stride_n;
  a.odtype = out->dtype;
  return hip_status(da2::launch_attn(a, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
