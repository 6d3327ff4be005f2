// Shared ranking kernels (Algorithm 1; routing appendix).
//
// Every region pair gets a unique 54-bit key: the order-preserving image of its
// float32 score in bits 53..22 and (2^22 - 1 - index) in bits 21..0, so that a
// larger key means "ranked earlier" under (score descending, index ascending).
// With the cumulative quotas cut0 = T16, cut1 = T16 + T8, cut2 = T16 + T8 + T4,
// the pairs of class 16 are exactly those with key >= key of rank cut0, class
// 8 those below it with key >= key of rank cut1, and class 4 those below that
// with key >= key of rank cut2 (1-based ranks; an empty cut matches nothing).
//
// Head scope finds the three threshold keys with a 5-pass most-significant-digit
// radix select (11,11,11,11,10 bits) over all R^2 keys of a head: a histogram
// kernel spread over many workgroups, then a one-workgroup scan per head that
// fixes the next digit. The third pass also collects the keys that match a
// cut's 22-bit prefix (the threshold is one of them); when there are at most
// kRankCand of them, its scan sorts them and reads the threshold key directly.
// A cut with more (ties, or a dense bin) takes the last two passes inside that
// scan's workgroup, over the head's scores with an LDS histogram, so the host
// launches three histogram passes in every case. Row scope sorts each row's R
// keys in LDS (bitonic).
#include <mutex>

#include "common.hpp"
#include "launch.hpp"

namespace da2 {

constexpr int kBins = 2048;
constexpr int kPasses = 5;
__constant__ int kShift[kPasses] = {43, 32, 21, 10, 0};
__constant__ int kWidth[kPasses] = {11, 11, 11, 11, 10};
constexpr int kHistChunk = 8192;
constexpr uint64_t kNone = ~0ull;
constexpr int kCollectPass = 2;   // the pass that collects candidate keys
constexpr int kLocalCand = 256;   // candidates one histogram workgroup stages per cut

__device__ inline uint64_t rank_key(float a, uint32_t idx) {
  if (a == 0.0f) a = 0.0f;  // -0 ranks like +0
  uint32_t u = __float_as_uint(a);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (static_cast<uint64_t>(u) << 22) | static_cast<uint64_t>((1u << 22) - 1u - idx);
}

__global__ void rank_init_kernel(RankArgs args) {
  const int bh = blockIdx.x;
  for (int i = threadIdx.x; i < kCuts * kBins; i += blockDim.x) args.hist[(int64_t)bh * kCuts * kBins + i] = 0u;
  if (threadIdx.x < kCuts) {
    const int t = threadIdx.x;
    args.prefix[bh * kCuts + t] = 0ull;
    args.kleft[bh * kCuts + t] = args.cut[t];
    args.ccount[bh * kCuts + t] = 0u;
  }
}

// Histogram slot of each cut in the pass whose digit ends at bit hi: -1 for a
// finished cut, else the first active cut with the same prefix (cuts with
// equal prefixes, such as all of them in the first pass, count the same
// elements into one histogram). prefix and kleft: the head's cuts, in global
// memory or LDS.
__device__ inline void slots_of(const uint64_t* prefix, const int64_t* kleft, int hi, int (&slot)[kCuts],
                                uint64_t (&pre)[kCuts]) {
  for (int t = 0; t < kCuts; ++t) {
    pre[t] = prefix[t] >> hi;
    slot[t] = kleft[t] > 0 ? t : -1;
    for (int u = 0; u < t && slot[t] == t; ++u)
      if (slot[u] == u && pre[u] == pre[t]) slot[t] = u;
  }
}

__global__ __launch_bounds__(256) void rank_hist_kernel(RankArgs args, int pass) {
  __shared__ uint32_t lh[kCuts][kBins];
  __shared__ uint64_t lc[kCuts][kLocalCand];  // staged candidates (collecting pass)
  __shared__ uint32_t lcnt[kCuts], lbase[kCuts];
  const int bh = blockIdx.y;
  const bool collect = pass == kCollectPass;
  const int64_t M = (int64_t)args.R * args.R;
  const int sh = kShift[pass], hi = sh + kWidth[pass];
  const uint64_t mask = (1ull << kWidth[pass]) - 1ull;
  for (int i = threadIdx.x; i < kCuts * kBins; i += 256) (&lh[0][0])[i] = 0u;
  int slot[kCuts];
  uint64_t pre[kCuts];
  slots_of(args.prefix + bh * kCuts, args.kleft + bh * kCuts, hi, slot, pre);
  bool own[kCuts], any = false;
  for (int t = 0; t < kCuts; ++t) {
    own[t] = slot[t] == t;
    any = any || own[t];
  }
  if (threadIdx.x < kCuts) lcnt[threadIdx.x] = 0u;
  __syncthreads();
  if (any) {
    const float* A = args.A + (int64_t)bh * M;
    const int64_t e0 = (int64_t)blockIdx.x * kHistChunk;
    const int64_t e1 = e0 + kHistChunk < M ? e0 + kHistChunk : M;
    constexpr int U = 8;  // loads in flight per thread
    for (int64_t eb = e0 + threadIdx.x; eb < e1; eb += 256 * U) {
      float v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = eb + u * 256 < e1 ? A[eb + u * 256] : 0.0f;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t e = eb + u * 256;
        if (e >= e1) break;
        const uint64_t key = rank_key(v[u], static_cast<uint32_t>(e));
        const uint32_t dig = static_cast<uint32_t>((key >> sh) & mask);
#pragma unroll
        for (int t = 0; t < kCuts; ++t)
          if (own[t] && (key >> hi) == pre[t]) {
            atomicAdd(&lh[t][dig], 1u);
            if (collect) {
              const uint32_t pos = atomicAdd(&lcnt[t], 1u);
              if (pos < kLocalCand) lc[t][pos] = key;
            }
          }
      }
    }
  }
  __syncthreads();
  uint32_t* gh = args.hist + (int64_t)bh * kCuts * kBins;
  for (int t = 0; t < kCuts; ++t) {
    if (!own[t]) continue;  // uniform across the block
    for (int i = threadIdx.x; i < kBins; i += 256) {
      const uint32_t v = lh[t][i];
      if (v) atomicAdd(gh + t * kBins + i, v);
    }
  }
  if (collect) {
    // reserve room in the head's candidate list; a workgroup with more than
    // kLocalCand candidates marks the list as too long (count > kRankCand)
    if (threadIdx.x < kCuts) {
      const int t = threadIdx.x;
      const uint32_t c = lcnt[t];
      uint32_t base = kRankCand;
      if (own[t] && c > 0)
        base = atomicAdd(args.ccount + bh * kCuts + t, c <= (uint32_t)kLocalCand ? c : (uint32_t)kRankCand + 1u);
      lbase[t] = base;
    }
    __syncthreads();
    for (int t = 0; t < kCuts; ++t) {
      const uint32_t c = lcnt[t], base = lbase[t];
      if (!own[t] || c == 0 || c > (uint32_t)kLocalCand || base + c > (uint32_t)kRankCand) continue;  // uniform
      uint64_t* dst = args.cand + ((int64_t)bh * kCuts + t) * kRankCand + base;
      for (uint32_t i = threadIdx.x; i < c; i += 256) dst[i] = lc[t][i];
    }
  }
}

// Descending bitonic sort of n (a power of two, <= kRankCand) keys in LDS by a
// 256-thread block.
__device__ inline void block_sort_desc(uint64_t* sk, int n) {
  for (int k = 2; k <= n; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = threadIdx.x; i < n; i += 256) {
        const int l = i ^ j;
        if (l > i) {
          const bool desc = (i & k) == 0;
          const uint64_t x = sk[i], y = sk[l];
          if (desc ? (x < y) : (x > y)) {
            sk[i] = y;
            sk[l] = x;
          }
        }
      }
      __syncthreads();
    }
  }
}

// Exclusive prefix sum over a 256-thread block.
__device__ inline uint32_t block_exscan_256(uint32_t v, uint32_t* sh, uint32_t* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint32_t x = v;
  for (int o = 1; o < 64; o <<= 1) {
    uint32_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) sh[w] = x;
  __syncthreads();
  uint32_t base = 0;
  for (int q = 0; q < w; ++q) base += sh[q];
  *total = sh[0] + sh[1] + sh[2] + sh[3];
  __syncthreads();
  return base + x - v;
}

// Fixes the next digit of cut t from a histogram h of the digit (2048 bins,
// global or LDS) in which the cut's keys are counted: thread i owns bins
// [2047-8i-7, 2047-8i], visited from the top, and the thread whose run holds
// rank k appends the digit to the cut's prefix and keeps the rank left inside
// that bin. Called by all 256 threads; returns after a barrier.
__device__ inline void scan_digit(const uint32_t* h, int s, int64_t k, uint64_t& prefix, int64_t& kleft,
                                  uint32_t* sh) {
  uint32_t c[8], local = 0;
  for (int q = 0; q < 8; ++q) {
    c[q] = h[kBins - 1 - 8 * threadIdx.x - q];
    local += c[q];
  }
  uint32_t total;
  const uint32_t before = block_exscan_256(local, sh, &total);
  if ((int64_t)before < k && k <= (int64_t)before + local) {
    uint32_t run = before;
    for (int q = 0; q < 8; ++q) {
      if (k <= (int64_t)run + c[q]) {
        const uint64_t dig = kBins - 1 - 8 * threadIdx.x - q;
        prefix |= dig << s;
        kleft = k - run;
        break;
      }
      run += c[q];
    }
  }
  __syncthreads();
}

// One workgroup per head: fixes this pass's digit of every cut from the
// global histogram. The cuts' prefixes and ranks left are held in LDS while
// the workgroup works and written back at the end. The collecting pass first
// resolves each cut whose candidate list is complete by sorting it; a cut still
// open after that (its 22-bit prefix is shared by more keys than the list
// holds: ties or a dense bin) takes the remaining passes here, over the head's
// scores with an LDS histogram, so the host launches no further passes.
__global__ __launch_bounds__(256) void rank_scan_kernel(RankArgs args, int pass) {
  __shared__ uint32_t sh[4];
  // candidate keys; in the remaining passes, the cuts' digit histograms
  constexpr int kSkWords = kRankCand > kCuts * kBins / 2 ? kRankCand : kCuts * kBins / 2;
  __shared__ uint64_t sk[kSkWords];
  __shared__ uint64_t s_prefix[kCuts];
  __shared__ int64_t s_kleft[kCuts];
  const int bh = blockIdx.x;
  const int s = kShift[pass];
  uint32_t* gh = args.hist + (int64_t)bh * kCuts * kBins;
  if (threadIdx.x < kCuts) {
    s_prefix[threadIdx.x] = args.prefix[bh * kCuts + threadIdx.x];
    s_kleft[threadIdx.x] = args.kleft[bh * kCuts + threadIdx.x];
  }
  __syncthreads();
  // the histogram slots of this pass, fixed before any cut's prefix changes
  int slot[kCuts];
  uint64_t pre[kCuts];
  slots_of(s_prefix, s_kleft, s + kWidth[pass], slot, pre);
  uint32_t ncand[kCuts];
  for (int t = 0; t < kCuts; ++t)
    ncand[t] = pass == kCollectPass && slot[t] >= 0 ? args.ccount[bh * kCuts + slot[t]] : (uint32_t)kRankCand + 1u;
  __syncthreads();  // every thread has read the prefixes and ranks before any changes
  for (int t = 0; t < kCuts; ++t) {
    const int64_t k = s_kleft[t];
    if (k <= 0) continue;  // uniform across the block
    if (ncand[t] >= 1u && ncand[t] <= (uint32_t)kRankCand && k <= (int64_t)ncand[t]) {
      // the collected keys are exactly those with this cut's prefix, and the
      // threshold is the k-th largest of them (1 <= k <= ncand always holds
      // here; anything else takes the histogram path below)
      const int n = (int)ncand[t];
      int np = 1;
      while (np < n) np <<= 1;
      const uint64_t* src = args.cand + ((int64_t)bh * kCuts + slot[t]) * kRankCand;
      for (int i = threadIdx.x; i < np; i += 256) sk[i] = i < n ? src[i] : 0ull;
      __syncthreads();
      block_sort_desc(sk, np);
      if (threadIdx.x == 0) {
        s_prefix[t] = sk[k - 1];
        s_kleft[t] = 0;
      }
      __syncthreads();
      continue;
    }
    scan_digit(gh + slot[t] * kBins, s, k, s_prefix[t], s_kleft[t], sh);
  }
  for (int i = threadIdx.x; i < kCuts * kBins; i += 256) gh[i] = 0u;
  if (pass == kCollectPass) {
    // remaining passes for the cuts still open, in this workgroup (the
    // candidate sorts are done with sk, whose LDS now holds the histograms)
    uint32_t* lh = reinterpret_cast<uint32_t*>(sk);
    static_assert(kCuts * kBins * sizeof(uint32_t) <= sizeof(sk), "histograms fit");
    const int64_t M = (int64_t)args.R * args.R;
    const float* A = args.A + (int64_t)bh * M;
    for (int q = kCollectPass + 1; q < kPasses; ++q) {
      bool open = false;
      for (int t = 0; t < kCuts; ++t) open = open || s_kleft[t] > 0;
      if (!open) break;  // uniform: every thread reads the same LDS values
      const int sq = kShift[q], hi = sq + kWidth[q];
      const uint64_t mask = (1ull << kWidth[q]) - 1ull;
      slots_of(s_prefix, s_kleft, hi, slot, pre);
      bool own[kCuts];
      for (int t = 0; t < kCuts; ++t) own[t] = slot[t] == t;
      for (int i = threadIdx.x; i < kCuts * kBins; i += 256) lh[i] = 0u;
      __syncthreads();
      for (int64_t e = threadIdx.x; e < M; e += 256) {
        const uint64_t key = rank_key(A[e], static_cast<uint32_t>(e));
        const uint32_t dig = static_cast<uint32_t>((key >> sq) & mask);
        for (int t = 0; t < kCuts; ++t)
          if (own[t] && (key >> hi) == pre[t]) atomicAdd(&lh[t * kBins + dig], 1u);
      }
      __syncthreads();
      for (int t = 0; t < kCuts; ++t) {
        const int64_t k = s_kleft[t];
        if (k <= 0) continue;  // uniform
        scan_digit(lh + slot[t] * kBins, sq, k, s_prefix[t], s_kleft[t], sh);
      }
    }
  }
  __syncthreads();
  if (threadIdx.x < kCuts) {
    const int t = threadIdx.x;
    args.prefix[bh * kCuts + t] = s_prefix[t];
    args.kleft[bh * kCuts + t] = s_kleft[t];
    if (pass == kCollectPass) args.thr[bh * kCuts + t] = args.cut[t] > 0 ? s_prefix[t] : kNone;
  }
}

// Row scope: sort each row's keys descending in LDS, read the threshold keys.
__global__ __launch_bounds__(256) void rank_row_select_kernel(RankArgs args, int P) {
  extern __shared__ uint64_t sk[];
  const int a = blockIdx.x, bh = blockIdx.y, R = args.R;
  const float* A = args.A + ((int64_t)bh * R + a) * R;
  for (int i = threadIdx.x; i < P; i += 256) sk[i] = i < R ? rank_key(A[i], i) : 0ull;
  __syncthreads();
  for (int k = 2; k <= P; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = threadIdx.x; i < P; i += 256) {
        const int l = i ^ j;
        if (l > i) {
          const bool desc = (i & k) == 0;
          const uint64_t x = sk[i], y = sk[l];
          if (desc ? (x < y) : (x > y)) {
            sk[i] = y;
            sk[l] = x;
          }
        }
      }
      __syncthreads();
    }
  }
  if (threadIdx.x < kCuts) {
    const int t = threadIdx.x;
    const int64_t want = args.cut[t];
    args.thr[((int64_t)bh * R + a) * kCuts + t] = want > 0 ? sk[want - 1] : kNone;
  }
}

// Exclusive prefix sum of 64-bit values over an NT-thread block (NT = 64: one
// wave, no LDS; NT = 256: four waves through LDS).
template <int NT>
__device__ inline uint64_t block_exscan_u64(uint64_t v, uint64_t* sh, uint64_t* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint64_t x = v;
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if constexpr (NT == 64) {
    *total = __shfl(x, 63, 64);
    return x - v;
  } else {
    if (lane == 63) sh[w] = x;
    __syncthreads();
    uint64_t base = 0;
    for (int q = 0; q < w; ++q) base += sh[q];
    *total = sh[0] + sh[1] + sh[2] + sh[3];
    __syncthreads();
    return base + x - v;
  }
}

// Classes, ascending per-row lists (4-bit, then 8-bit, then 16-bit: the phase
// order of the attention), counts and row cost; one NT-thread workgroup per
// row (NT = 64 for rows of up to 1024 blocks, 256 beyond). The row's scores are
// staged in LDS (R floats, dynamic) with coalesced loads; thread i then owns
// the contiguous run of key blocks [i E, (i + 1) E), E = ceil(R / NT): it
// classifies its run, a block-wide scan of the packed per-class counts (21
// bits each) gives every class's write offset, and a second walk over the run
// writes the lists.
template <int NT>
__global__ __launch_bounds__(NT) void rank_classify_kernel(RankArgs args) {
  extern __shared__ float srow[];
  __shared__ uint64_t sh[4];
  const int a = blockIdx.x, bh = blockIdx.y, R = args.R, tid = threadIdx.x;
  const int64_t row = (int64_t)bh * R + a;
  const float* A = args.A + row * R;
  // eight loads in flight per thread (indices past the row read its last entry)
  for (int b0 = tid; b0 < R; b0 += NT * 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = A[min(b0 + NT * u, R - 1)];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (b0 + NT * u < R) srow[b0 + NT * u] = v[u];
  }
  __syncthreads();
  const bool head = args.scope == DA2_SCOPE_HEAD;
  const uint64_t* thr = head ? args.thr + (int64_t)bh * kCuts : args.thr + row * kCuts;
  const uint64_t t16 = thr[0], t8 = thr[1], t4 = thr[2];
  uint8_t* cls = args.cls + row * R;
  uint16_t* keys = args.keys + row * R;
  auto class_of = [&](int b) -> int {
    const uint64_t key =
        head ? rank_key(srow[b], static_cast<uint32_t>(a * R + b)) : rank_key(srow[b], static_cast<uint32_t>(b));
    return key >= t16 ? 16 : (key >= t8 ? 8 : (key >= t4 ? 4 : 0));
  };
  constexpr int kF = 21;
  constexpr uint64_t kM = (1ull << kF) - 1ull;
  auto field = [](int c) -> uint64_t {
    return c == 4 ? 1ull : (c == 8 ? (1ull << kF) : (c == 16 ? (1ull << (2 * kF)) : 0ull));
  };
  const int E = (R + NT - 1) / NT;
  const int b0 = min(R, tid * E), b1 = min(R, b0 + E);
  uint64_t cnt = 0;
  for (int b = b0; b < b1; ++b) {
    const int c = class_of(b);
    cls[b] = static_cast<uint8_t>(c);
    cnt += field(c);
  }
  uint64_t tot;
  const uint64_t before = block_exscan_u64<NT>(cnt, sh, &tot);
  const uint32_t n4 = static_cast<uint32_t>(tot & kM), n8 = static_cast<uint32_t>((tot >> kF) & kM),
                 n16 = static_cast<uint32_t>((tot >> (2 * kF)) & kM);
  uint32_t p4 = static_cast<uint32_t>(before & kM);
  uint32_t p8 = n4 + static_cast<uint32_t>((before >> kF) & kM);
  uint32_t p16 = n4 + n8 + static_cast<uint32_t>((before >> (2 * kF)) & kM);
  for (int b = b0; b < b1; ++b) {
    const int c = class_of(b);
    if (c == 4)
      keys[p4++] = static_cast<uint16_t>(b);
    else if (c == 8)
      keys[p8++] = static_cast<uint16_t>(b);
    else if (c == 16)
      keys[p16++] = static_cast<uint16_t>(b);
  }
  if (tid == 0) {
    args.counts[row * 4 + 0] = n4;
    args.counts[row * 4 + 1] = n8;
    args.counts[row * 4 + 2] = n16;
    args.counts[row * 4 + 3] = 0;
    // attention cost of the row in units of the measured per-tile times
    // (a 4-bit NVFP4 or 16-bit tile costs about 1.5 INT8 tiles)
    args.cost[row] = 3 * n4 + 2 * n8 + 3 * n16;
  }
}

// One workgroup: counting sort of the rows into the attention work order.
// Rows are grouped by head and, inside a head, by row parity (two half-heads
// with near-equal cost); each group is sorted most expensive first. The
// attention launch hands workgroup b the entry (b mod 8) * ceil(n/8) + b div 8,
// and workgroups are dispatched round-robin over the 8 XCDs, so each XCD walks
// one contiguous segment (about n/8 rows of one or two heads, whose K/V then
// share that XCD's L2) longest-first.
constexpr int kOrderBins = 8192;
// Bin of row i (cost c) in the work order. 32-bit arithmetic: rows number
// fewer than 2^31 and R <= 65535 (both checked on the host), so c (n4 + n8 +
// n16 <= R blocks at most 3 each) times the bins per group (<= 4096) and the
// rescaled key (< 2^16 x 8192) stay below 2^32.
__device__ inline uint32_t order_key(const RankArgs& args, uint32_t i, int32_t c) {
  const uint32_t R = static_cast<uint32_t>(args.R), BH = static_cast<uint32_t>(args.B * args.H);
  const uint32_t cmax = 3u * R;  // cost of a row with R 4-bit or 16-bit blocks
  const uint32_t groups = 2u * BH;
  const uint32_t nbh = groups < kOrderBins ? kOrderBins / groups : 1u;  // cost bins per group
  const uint32_t bh = i / R, half = (i - bh * R) & 1u;
  const uint32_t bin = static_cast<uint32_t>(c) * (nbh - 1u) / cmax;
  uint32_t key = (2u * bh + half) * nbh + (nbh - 1u - bin);
  if (groups * nbh > kOrderBins) key = key * kOrderBins / (groups * nbh);
  return key;
}

__global__ __launch_bounds__(1024) void rank_order_kernel(RankArgs args) {
  __shared__ uint32_t hist[kOrderBins];
  __shared__ uint32_t part[1024];
  constexpr int U = 8;  // row costs in flight per thread
  const uint32_t n = static_cast<uint32_t>(args.B * args.H) * static_cast<uint32_t>(args.R);
  for (int i = threadIdx.x; i < kOrderBins; i += 1024) hist[i] = 0u;
  __syncthreads();
  for (uint32_t i0 = threadIdx.x; i0 < n; i0 += 1024u * U) {
    int32_t c[U];
#pragma unroll
    for (int u = 0; u < U; ++u) c[u] = args.cost[min(i0 + 1024u * u, n - 1u)];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (i0 + 1024u * u < n) atomicAdd(&hist[order_key(args, i0 + 1024u * u, c[u])], 1u);
  }
  __syncthreads();
  constexpr int per = kOrderBins / 1024;
  uint32_t s = 0;
  for (int q = 0; q < per; ++q) s += hist[threadIdx.x * per + q];
  // exclusive scan of the 1024 per-thread sums: within each wave, then over
  // the 16 wave totals
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint32_t x = s;
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) part[w] = x;
  __syncthreads();
  uint32_t run = x - s;
  for (int q = 0; q < w; ++q) run += part[q];
  for (int q = 0; q < per; ++q) {
    uint32_t v = hist[threadIdx.x * per + q];
    hist[threadIdx.x * per + q] = run;
    run += v;
  }
  __syncthreads();
  for (uint32_t i0 = threadIdx.x; i0 < n; i0 += 1024u * U) {
    int32_t c[U];
#pragma unroll
    for (int u = 0; u < U; ++u) c[u] = args.cost[min(i0 + 1024u * u, n - 1u)];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = i0 + 1024u * u;
      if (i < n) {
        const uint32_t pos = atomicAdd(&hist[order_key(args, i, c[u])], 1u);
        args.order[pos] = static_cast<int32_t>(i);
      }
    }
  }
  if (threadIdx.x == 0) {
    args.meta[0] = static_cast<int32_t>(n);
    args.meta[1] = 0;  // error flags of da2_mixed_attn calls on these lists
  }
}

// Fixed device scratch for callers that cannot allocate (da2_rank_assign_noalloc):
// every workspace array of the ranking lives here instead of in a caller
// buffer. Each device holds its own copy for the life of the process; calls
// on one device share it, so such calls must not overlap on that device. The
// kernels clear what must start at zero (rank_init_kernel), so no state from
// an earlier call is read.
static __device__ __align__(256) uint8_t scratch[kRankScratchBytes];

// Device address of this device's copy of the scratch array, looked up once
// per device with that device current and then reused. In host code the
// array's name is only a stand-in for the symbol, never a device address.
hipError_t rank_scratch_address(void** out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *out = addr[dev];
  return hipSuccess;
}

hipError_t launch_rank(const RankArgs& args, hipStream_t stream) {
  const int BH = args.B * args.H;
  if (args.scope == DA2_SCOPE_HEAD) {
    const int64_t M = (int64_t)args.R * args.R;
    const int chunks = (int)((M + kHistChunk - 1) / kHistChunk);
    hipLaunchKernelGGL(rank_init_kernel, dim3(BH), dim3(256), 0, stream, args);
    // passes after the collecting one run inside its scan (see rank_scan_kernel)
    for (int p = 0; p <= kCollectPass; ++p) {
      hipLaunchKernelGGL(rank_hist_kernel, dim3(chunks, BH), dim3(256), 0, stream, args, p);
      hipLaunchKernelGGL(rank_scan_kernel, dim3(BH), dim3(256), 0, stream, args, p);
    }
  } else {
    int P = 1;
    while (P < args.R) P <<= 1;
    hipLaunchKernelGGL(rank_row_select_kernel, dim3(args.R, BH), dim3(256), P * sizeof(uint64_t), stream, args, P);
  }
  if (args.R <= 1024)
    hipLaunchKernelGGL(rank_classify_kernel<64>, dim3(args.R, BH), dim3(64), args.R * sizeof(float), stream, args);
  else
    hipLaunchKernelGGL(rank_classify_kernel<256>, dim3(args.R, BH), dim3(256), args.R * sizeof(float), stream, args);
  hipLaunchKernelGGL(rank_order_kernel, dim3(1), dim3(1024), 0, stream, args);
  return hipGetLastError();
}

}  // namespace da2
