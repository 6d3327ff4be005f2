// Shared ranking kernels (Algorithm 1 without the 16-bit quota; routing appendix).
//
// Every region pair gets a unique 54-bit key: the order-preserving image of its
// float32 score in bits 53..22 and (2^22 - 1 - index) in bits 21..0, so that a
// larger key means "ranked earlier" under (score descending, index ascending).
// The pairs of class 8 are exactly those with key >= key of rank T8, and the
// retained pairs those with key >= key of rank T8+T4 (1-based ranks).
//
// Head scope finds both threshold keys with a 5-pass most-significant-digit
// radix select (11,11,11,11,10 bits) over all R^2 keys of a head: a histogram
// kernel spread over many workgroups, then a one-workgroup scan per head that
// fixes the next digit. Row scope sorts each row's R keys in LDS (bitonic).
#include "common.hpp"
#include "launch.hpp"

namespace da2 {

constexpr int kBins = 2048;
constexpr int kPasses = 5;
__constant__ int kShift[kPasses] = {43, 32, 21, 10, 0};
__constant__ int kWidth[kPasses] = {11, 11, 11, 11, 10};
constexpr int kHistChunk = 8192;
constexpr uint64_t kNone = ~0ull;

__device__ inline uint64_t rank_key(float a, uint32_t idx) {
  if (a == 0.0f) a = 0.0f;  // -0 ranks like +0
  uint32_t u = __float_as_uint(a);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (static_cast<uint64_t>(u) << 22) | static_cast<uint64_t>((1u << 22) - 1u - idx);
}

__global__ void rank_init_kernel(RankArgs args) {
  const int bh = blockIdx.x;
  for (int i = threadIdx.x; i < 2 * kBins; i += blockDim.x) args.hist[(int64_t)bh * 2 * kBins + i] = 0u;
  if (threadIdx.x < 2) {
    const int t = threadIdx.x;
    args.prefix[bh * 2 + t] = 0ull;
    args.kleft[bh * 2 + t] = t == 0 ? args.T8 : args.T8 + args.T4;
  }
}

__global__ __launch_bounds__(256) void rank_hist_kernel(RankArgs args, int pass) {
  __shared__ uint32_t lh[2][kBins];
  const int bh = blockIdx.y;
  const int64_t M = (int64_t)args.R * args.R;
  const int sh = kShift[pass], hi = sh + kWidth[pass];
  const uint64_t mask = (1ull << kWidth[pass]) - 1ull;
  for (int i = threadIdx.x; i < 2 * kBins; i += 256) (&lh[0][0])[i] = 0u;
  bool act[2];
  uint64_t pre[2];
  for (int t = 0; t < 2; ++t) {
    act[t] = args.kleft[bh * 2 + t] > 0;
    pre[t] = args.prefix[bh * 2 + t] >> hi;
  }
  __syncthreads();
  if (act[0] || act[1]) {
    const float* A = args.A + (int64_t)bh * M;
    const int64_t e0 = (int64_t)blockIdx.x * kHistChunk;
    const int64_t e1 = e0 + kHistChunk < M ? e0 + kHistChunk : M;
    for (int64_t e = e0 + threadIdx.x; e < e1; e += 256) {
      const uint64_t key = rank_key(A[e], static_cast<uint32_t>(e));
      const uint32_t dig = static_cast<uint32_t>((key >> sh) & mask);
      if (act[0] && (key >> hi) == pre[0]) atomicAdd(&lh[0][dig], 1u);
      if (act[1] && (key >> hi) == pre[1]) atomicAdd(&lh[1][dig], 1u);
    }
  }
  __syncthreads();
  uint32_t* gh = args.hist + (int64_t)bh * 2 * kBins;
  for (int i = threadIdx.x; i < 2 * kBins; i += 256) {
    uint32_t v = (&lh[0][0])[i];
    if (v) atomicAdd(gh + i, v);
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

__global__ __launch_bounds__(256) void rank_scan_kernel(RankArgs args, int pass) {
  __shared__ uint32_t sh[4];
  const int bh = blockIdx.x;
  const int s = kShift[pass];
  uint32_t* gh = args.hist + (int64_t)bh * 2 * kBins;
  for (int t = 0; t < 2; ++t) {
    const int64_t k = args.kleft[bh * 2 + t];
    if (k <= 0) continue;  // uniform across the block
    // thread i owns bins [2047-8i-7, 2047-8i], visited from the top
    uint32_t c[8], local = 0;
    for (int q = 0; q < 8; ++q) {
      c[q] = gh[t * kBins + (kBins - 1 - 8 * threadIdx.x - q)];
      local += c[q];
    }
    uint32_t total;
    uint32_t before = block_exscan_256(local, sh, &total);
    if ((int64_t)before < k && k <= (int64_t)before + local) {
      uint32_t run = before;
      for (int q = 0; q < 8; ++q) {
        if (k <= (int64_t)run + c[q]) {
          const uint64_t dig = kBins - 1 - 8 * threadIdx.x - q;
          args.prefix[bh * 2 + t] |= dig << s;
          args.kleft[bh * 2 + t] = k - run;
          break;
        }
        run += c[q];
      }
    }
    __syncthreads();
  }
  for (int i = threadIdx.x; i < 2 * kBins; i += 256) gh[i] = 0u;
  if (pass == kPasses - 1 && threadIdx.x < 2) {
    const int t = threadIdx.x;
    const int64_t want = t == 0 ? args.T8 : args.T8 + args.T4;
    args.thr[bh * 2 + t] = want > 0 ? args.prefix[bh * 2 + t] : kNone;
  }
}

// Row scope: sort each row's keys descending in LDS, read the two threshold keys.
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
  if (threadIdx.x < 2) {
    const int t = threadIdx.x;
    const int64_t want = t == 0 ? args.T8 : args.T8 + args.T4;
    args.thr[((int64_t)bh * R + a) * 2 + t] = want > 0 ? sk[want - 1] : kNone;
  }
}

// Classes, ascending per-row lists (4-bit then 8-bit), counts and row cost.
__global__ __launch_bounds__(256) void rank_classify_kernel(RankArgs args) {
  __shared__ uint32_t sh[4];
  const int a = blockIdx.x, bh = blockIdx.y, R = args.R;
  const int64_t row = (int64_t)bh * R + a;
  const float* A = args.A + row * R;
  const uint64_t* thr = args.scope == DA2_SCOPE_HEAD ? args.thr + (int64_t)bh * 2 : args.thr + row * 2;
  const uint64_t t8 = thr[0], t84 = thr[1];
  uint8_t* cls = args.cls + row * R;
  uint16_t* keys = args.keys + row * R;
  const int lane = threadIdx.x & 63;
  uint32_t n4 = 0, n8 = 0;
  for (int want = 4; want <= 8; want += 4) {
    uint32_t base = want == 4 ? 0u : n4;
    for (int c0 = 0; c0 < R; c0 += 256) {
      const int b = c0 + threadIdx.x;
      int c = 0;
      if (b < R) {
        const uint64_t key = args.scope == DA2_SCOPE_HEAD ? rank_key(A[b], static_cast<uint32_t>(a * R + b))
                                                          : rank_key(A[b], static_cast<uint32_t>(b));
        c = key >= t8 ? 8 : (key >= t84 ? 4 : 0);
        if (want == 4) cls[b] = static_cast<uint8_t>(c);
      }
      const bool f = c == want;
      const uint64_t m = __ballot(f);
      const uint32_t in_wave = __popcll(m & ((1ull << lane) - 1ull));
      uint32_t tot;
      const uint32_t wave_base = block_exscan_256(lane == 0 ? (uint32_t)__popcll(m) : 0u, sh, &tot);
      const uint32_t wb = __shfl(wave_base, 0, 64);
      if (f) keys[base + wb + in_wave] = static_cast<uint16_t>(b);
      base += tot;
    }
    if (want == 4)
      n4 = base;
    else
      n8 = base - n4;
  }
  if (threadIdx.x == 0) {
    args.counts[row * 2 + 0] = n4;
    args.counts[row * 2 + 1] = n8;
    args.cost[row] = 5 * n4 + 4 * n8;
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
__device__ inline int order_key(const RankArgs& args, int64_t i) {
  const int BH = args.B * args.H;
  const int64_t cmax = 5ll * args.R;
  const int groups = 2 * BH;
  const int nbh = groups < kOrderBins ? kOrderBins / groups : 1;  // cost bins per group
  const int bh = (int)(i / args.R), half = (int)(i % args.R) & 1;
  const int bin = (int)((int64_t)args.cost[i] * (nbh - 1) / (cmax > 0 ? cmax : 1));
  int64_t key = (int64_t)(2 * bh + half) * nbh + (nbh - 1 - bin);
  if ((int64_t)groups * nbh > kOrderBins) key = key * kOrderBins / ((int64_t)groups * nbh);
  return (int)key;
}

__global__ __launch_bounds__(1024) void rank_order_kernel(RankArgs args) {
  __shared__ uint32_t hist[kOrderBins];
  __shared__ uint32_t part[1024];
  const int64_t n = (int64_t)args.B * args.H * args.R;
  for (int i = threadIdx.x; i < kOrderBins; i += 1024) hist[i] = 0u;
  __syncthreads();
  for (int64_t i = threadIdx.x; i < n; i += 1024) atomicAdd(&hist[order_key(args, i)], 1u);
  __syncthreads();
  constexpr int per = kOrderBins / 1024;
  uint32_t s = 0;
  for (int q = 0; q < per; ++q) s += hist[threadIdx.x * per + q];
  part[threadIdx.x] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t run = 0;
    for (int q = 0; q < 1024; ++q) {
      uint32_t v = part[q];
      part[q] = run;
      run += v;
    }
  }
  __syncthreads();
  uint32_t run = part[threadIdx.x];
  for (int q = 0; q < per; ++q) {
    uint32_t v = hist[threadIdx.x * per + q];
    hist[threadIdx.x * per + q] = run;
    run += v;
  }
  __syncthreads();
  for (int64_t i = threadIdx.x; i < n; i += 1024) {
    const uint32_t pos = atomicAdd(&hist[order_key(args, i)], 1u);
    args.order[pos] = (int32_t)i;
  }
  if (threadIdx.x == 0) args.meta[0] = (int32_t)n;
}

hipError_t launch_rank(const RankArgs& args, hipStream_t stream) {
  const int BH = args.B * args.H;
  if (args.scope == DA2_SCOPE_HEAD) {
    const int64_t M = (int64_t)args.R * args.R;
    const int chunks = (int)((M + kHistChunk - 1) / kHistChunk);
    hipLaunchKernelGGL(rank_init_kernel, dim3(BH), dim3(256), 0, stream, args);
    for (int p = 0; p < kPasses; ++p) {
      hipLaunchKernelGGL(rank_hist_kernel, dim3(chunks, BH), dim3(256), 0, stream, args, p);
      hipLaunchKernelGGL(rank_scan_kernel, dim3(BH), dim3(256), 0, stream, args, p);
    }
  } else {
    int P = 1;
    while (P < args.R) P <<= 1;
    hipLaunchKernelGGL(rank_row_select_kernel, dim3(args.R, BH), dim3(256), P * sizeof(uint64_t), stream, args, P);
  }
  hipLaunchKernelGGL(rank_classify_kernel, dim3(args.R, BH), dim3(256), 0, stream, args);
  hipLaunchKernelGGL(rank_order_kernel, dim3(1), dim3(1024), 0, stream, args);
  return hipGetLastError();
}

}  // namespace da2
