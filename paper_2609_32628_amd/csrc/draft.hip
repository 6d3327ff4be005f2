// Draft map kernels (descriptor equation; Definition 3.1).
//
//   draft_pool     one workgroup per (block, head, Q or K): mean (float64 sum /
//                  n_a) and channel max over the valid tokens, plus the per-head
//                  max|Q|, max|K| used by the NVFP4 tensor scales.
//   draft_logits   64x64 tiles of Qbar Kbar^T / sqrt d and Qmax Kmax^T / sqrt d in
//                  float64, both operands staged through LDS in 16-channel slices.
//   draft_softmax  one workgroup per row: the two row softmaxes (max subtracted)
//                  mixed with weight lambda, rounded once to float32.
#include "common.hpp"
#include "launch.hpp"

namespace da2 {

__global__ void zero_u32_kernel(uint32_t* p, int64_t stride, int count, int64_t n_rows) {
  int64_t row = blockIdx.x;
  for (int i = threadIdx.x; i < count; i += blockDim.x) p[row * stride + i] = 0u;
  (void)n_rows;
}

// One workgroup per (block, head, Q or K). Thread (row group rg, chunk cc)
// reads 16-byte chunks of the block's valid slots rg, rg + RG, ...; the
// per-channel float64 sums and float32 maxima are reduced across row groups
// (lanes CPR apart, then the four waves through LDS).
template <int D, typename T>
__global__ __launch_bounds__(256) void draft_pool_kernel(DraftArgs args) {
  constexpr int EPC = 16 / sizeof(T);  // elements per 16-byte load
  constexpr int CPR = D / EPC;         // loads per slot row
  constexpr int RG = 256 / CPR;        // row groups
  constexpr int RPT = kCap / RG;       // rows per thread
  __shared__ double s_sum[4][D];
  __shared__ float s_max[4][D];
  __shared__ float s_amax[4];
  const int a = blockIdx.x, bh = blockIdx.y, which = blockIdx.z;
  const int b = bh / args.H, h = bh % args.H, tid = threadIdx.x;
  const Layout L = layout_view(args.layout, args.R, args.Npad);
  const int n = L.n_a[a];
  const int32_t* slots = L.slot2tok + (int64_t)a * kCap;
  const int cc = tid % CPR, rg = tid / CPR;
  const T* X = static_cast<const T*>(which == 0 ? args.Q : args.K) + (int64_t)b * args.sb + (int64_t)h * args.sh +
               cc * EPC;
  float x[RPT][EPC];
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    const int s = rg + RG * k;
    if (s < n) load_chunk(X + (int64_t)slots[s] * args.sn, x[k]);
  }
  double sum[EPC];
  float mx[EPC];
  float amax = 0.0f;
#pragma unroll
  for (int e = 0; e < EPC; ++e) {
    sum[e] = 0.0;
    mx[e] = -INFINITY;
  }
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    if (rg + RG * k < n) {
#pragma unroll
      for (int e = 0; e < EPC; ++e) {
        sum[e] += (double)x[k][e];
        mx[e] = fmaxf(mx[e], x[k][e]);
        amax = fmaxf(amax, fabsf(x[k][e]));
      }
    }
  }
#pragma unroll
  for (int o = CPR; o < 64; o <<= 1)
#pragma unroll
    for (int e = 0; e < EPC; ++e) {
      sum[e] += __shfl_xor(sum[e], o, 64);
      mx[e] = fmaxf(mx[e], __shfl_xor(mx[e], o, 64));
    }
  const int w = tid >> 6, lane = tid & 63;
  if (lane < CPR)
#pragma unroll
    for (int e = 0; e < EPC; ++e) {
      s_sum[w][cc * EPC + e] = sum[e];
      s_max[w][cc * EPC + e] = mx[e];
    }
  amax = wave_max(amax);
  if (lane == 0) s_amax[w] = amax;
  __syncthreads();
  if (tid < D) {
    const double t = (s_sum[0][tid] + s_sum[1][tid]) + (s_sum[2][tid] + s_sum[3][tid]);
    const float m = fmaxf(fmaxf(s_max[0][tid], s_max[1][tid]), fmaxf(s_max[2][tid], s_max[3][tid]));
    const int64_t o = ((int64_t)bh * args.R + a) * D + tid;
    (which == 0 ? args.Qbar : args.Kbar)[o] = t / (double)n;
    (which == 0 ? args.Qmax : args.Kmax)[o] = (double)m;
  }
  if (tid == 0) {
    const float m = fmaxf(fmaxf(s_amax[0], s_amax[1]), fmaxf(s_amax[2], s_amax[3]));
    atomic_max_pos(args.stats + (int64_t)bh * (4 + D) + which, m);
  }
}

// 64x64 logit tile of both branches; 256 threads, 4x4 outputs per thread per branch.
__global__ __launch_bounds__(256) void draft_logits_kernel(DraftArgs args) {
  constexpr int KC = 16;
  __shared__ double sA[2][64][KC + 1];
  __shared__ double sB[2][64][KC + 1];
  const int R = args.R, d = args.d, bh = blockIdx.z;
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  const double* Qs[2] = {args.Qbar + (int64_t)bh * R * d, args.Qmax + (int64_t)bh * R * d};
  const double* Ks[2] = {args.Kbar + (int64_t)bh * R * d, args.Kmax + (int64_t)bh * R * d};
  double acc[2][4][4] = {};
  for (int k0 = 0; k0 < d; k0 += KC) {
    for (int e = threadIdx.x; e < 64 * KC; e += 256) {
      int row = e / KC, kk = e % KC;
      for (int br = 0; br < 2; ++br) {
        sA[br][row][kk] = (r0 + row < R) ? Qs[br][(int64_t)(r0 + row) * d + k0 + kk] : 0.0;
        sB[br][row][kk] = (c0 + row < R) ? Ks[br][(int64_t)(c0 + row) * d + k0 + kk] : 0.0;
      }
    }
    __syncthreads();
#pragma unroll 4
    for (int kk = 0; kk < KC; ++kk) {
#pragma unroll
      for (int br = 0; br < 2; ++br) {
        double av[4], bv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) av[i] = sA[br][ty + 16 * i][kk];
#pragma unroll
        for (int j = 0; j < 4; ++j) bv[j] = sB[br][tx + 16 * j][kk];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[br][i][j] = __builtin_fma(av[i], bv[j], acc[br][i][j]);
      }
    }
    __syncthreads();
  }
  const double sqd = sqrt((double)d);
  double* outs[2] = {args.S1 + (int64_t)bh * R * R, args.S2 + (int64_t)bh * R * R};
  for (int br = 0; br < 2; ++br)
    for (int i = 0; i < 4; ++i)
      for (int j = 0; j < 4; ++j) {
        int r = r0 + ty + 16 * i, cc = c0 + tx + 16 * j;
        if (r < R && cc < R) outs[br][(int64_t)r * R + cc] = acc[br][i][j] / sqd;
      }
}

__device__ inline double block_reduce(double v, bool is_max, double* sh) {
  for (int o = 32; o > 0; o >>= 1) {
    double w = __shfl_xor(v, o, 64);
    v = is_max ? fmax(v, w) : v + w;
  }
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  __syncthreads();
  double r = sh[0];
  for (int q = 1; q < (int)(blockDim.x >> 6); ++q) r = is_max ? fmax(r, sh[q]) : r + sh[q];
  return r;
}

__global__ __launch_bounds__(256) void draft_softmax_kernel(DraftArgs args) {
  __shared__ double sh[4];
  const int R = args.R, a = blockIdx.x, bh = blockIdx.y;
  const double* s1 = args.S1 + ((int64_t)bh * R + a) * R;
  const double* s2 = args.S2 + ((int64_t)bh * R + a) * R;
  double m1 = -INFINITY, m2 = -INFINITY;
  for (int i = threadIdx.x; i < R; i += 256) {
    m1 = fmax(m1, s1[i]);
    m2 = fmax(m2, s2[i]);
  }
  m1 = block_reduce(m1, true, sh);
  m2 = block_reduce(m2, true, sh);
  double z1 = 0.0, z2 = 0.0;
  for (int i = threadIdx.x; i < R; i += 256) {
    z1 += exp(s1[i] - m1);
    z2 += exp(s2[i] - m2);
  }
  z1 = block_reduce(z1, false, sh);
  z2 = block_reduce(z2, false, sh);
  const double lam = args.lambda;
  float* out = args.A + ((int64_t)bh * R + a) * R;
  for (int i = threadIdx.x; i < R; i += 256) {
    double p1 = exp(s1[i] - m1) / z1, p2 = exp(s2[i] - m2) / z2;
    out[i] = (float)((1.0 - lam) * p1 + lam * p2);
  }
}

hipError_t launch_draft(const DraftArgs& args, hipStream_t stream) {
  const int BH = args.B * args.H;
  hipLaunchKernelGGL(zero_u32_kernel, dim3(BH), dim3(64), 0, stream, args.stats, (int64_t)(4 + args.d), 2,
                     (int64_t)BH);
  const dim3 pool_grid(args.R, BH, 2);
  if (args.d == 128) {
    if (args.dtype == DA2_BF16)
      hipLaunchKernelGGL((draft_pool_kernel<128, uint16_t>), pool_grid, dim3(256), 0, stream, args);
    else
      hipLaunchKernelGGL((draft_pool_kernel<128, float>), pool_grid, dim3(256), 0, stream, args);
  } else {
    if (args.dtype == DA2_BF16)
      hipLaunchKernelGGL((draft_pool_kernel<64, uint16_t>), pool_grid, dim3(256), 0, stream, args);
    else
      hipLaunchKernelGGL((draft_pool_kernel<64, float>), pool_grid, dim3(256), 0, stream, args);
  }
  const int nt = (args.R + 63) / 64;
  hipLaunchKernelGGL(draft_logits_kernel, dim3(nt, nt, BH), dim3(256), 0, stream, args);
  hipLaunchKernelGGL(draft_softmax_kernel, dim3(args.R, BH), dim3(256), 0, stream, args);
  return hipGetLastError();
}

}  // namespace da2
