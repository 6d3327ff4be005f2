// Draft map kernels (descriptor equation; Definition 3.1).
//
//   draft_pool     one workgroup per (block, head, Q or K): mean (float64 sum /
//                  n_a) and channel max over the valid tokens, plus the per-head
//                  max|Q|, max|K| used by the NVFP4 tensor scales.
//   draft_logits   128x128 tiles of Qbar Kbar^T / sqrt d or Qmax Kmax^T / sqrt d
//                  on the float64 matrix cores (16x16x4 MFMA).
//   draft_softmax  one wave per row: the two row softmaxes (max subtracted)
//                  mixed with weight lambda, rounded once to float32.
#include "common.hpp"
#include "launch.hpp"

namespace da2 {

// One workgroup per (block, head, Q or K). The block's slots are read with
// coalesced 16-byte loads into an LDS tile (padding rows repeat the last valid
// row); thread
// (channel pair p, row group q) then reduces rows [q RPQ, (q + 1) RPQ) of its
// two channels: float64 sums, float32 maxima over the valid rows and max |x|
// (written per block; the logits launch reduces it per head, which avoids
// hundreds of workgroups contending for one atomic address).
// The row groups are combined through LDS in order. Sums of bf16 values in
// float64 are exact, so for bf16 inputs the order of the additions does not
// change the mean.
template <int D, typename T>
__global__ __launch_bounds__(256) void draft_pool_kernel(DraftArgs args) {
  constexpr int EPC = 16 / sizeof(T);    // elements per 16-byte load
  constexpr int CPR = D / EPC;           // loads per slot row
  constexpr int LPT = kCap * CPR / 256;  // loads per thread
  constexpr int CP = D / 2;              // channel pairs
  constexpr int RQ = 256 / CP;           // row groups of the reduction
  constexpr int RPQ = kCap / RQ;         // rows per group
  __shared__ __align__(16) T tile[kCap * D];
  // the per-group partial sums and maxima reuse the tile once it is read
  static_assert(RQ * D * (sizeof(double) + sizeof(float)) <= sizeof(T) * kCap * D, "partials fit in the tile");
  double (*s_sum)[D] = reinterpret_cast<double (*)[D]>(tile);
  float (*s_max)[D] = reinterpret_cast<float (*)[D]>(reinterpret_cast<char*>(tile) + RQ * D * sizeof(double));
  __shared__ float s_amax[4];
  const int a = blockIdx.x, bh = blockIdx.y, which = blockIdx.z;
  const int b = bh / args.H, h = bh % args.H, tid = threadIdx.x;
  const Layout L = layout_view(args.layout, args.R, args.Npad);
  const int n = L.n_a[a];
  const int32_t* slots = L.slot2tok + (int64_t)a * kCap;
  const T* X = static_cast<const T*>(which == 0 ? args.Q : args.K) + (int64_t)b * args.sb + (int64_t)h * args.sh;
  // token indices first, then the data loads, all unconditional so that they
  // overlap: padding slots read the last valid row again (a copy changes no
  // maximum; the sums skip those rows)
  int tok[LPT];
#pragma unroll
  for (int k = 0; k < LPT; ++k) tok[k] = slots[min((tid + 256 * k) / CPR, n - 1)];
  uint4 v[LPT];
#pragma unroll
  for (int k = 0; k < LPT; ++k) {
    const int cc = (tid + 256 * k) % CPR;
    v[k] = *reinterpret_cast<const uint4*>(X + (int64_t)tok[k] * args.sn + cc * EPC);
  }
#pragma unroll
  for (int k = 0; k < LPT; ++k) reinterpret_cast<uint4*>(tile)[tid + 256 * k] = v[k];
  __syncthreads();
  const int p = tid % CP, q = tid / CP;
  double s0 = 0.0, s1 = 0.0;
  float m0 = -INFINITY, m1 = -INFINITY, am = 0.0f;
#pragma unroll
  for (int r = 0; r < RPQ; ++r) {
    const int s = q * RPQ + r;
    const float2 f = tile_pair(tile, D, s, p);
    if (s < n) {
      s0 += (double)f.x;
      s1 += (double)f.y;
    }
    m0 = fmaxf(m0, f.x);
    m1 = fmaxf(m1, f.y);
    am = fmaxf(am, fmaxf(fabsf(f.x), fabsf(f.y)));
  }
  __syncthreads();  // every thread is done with the tile
  s_sum[q][2 * p] = s0;
  s_sum[q][2 * p + 1] = s1;
  s_max[q][2 * p] = m0;
  s_max[q][2 * p + 1] = m1;
  am = wave_max(am);
  if ((tid & 63) == 0) s_amax[tid >> 6] = am;
  __syncthreads();
  if (tid < D) {
    double t = s_sum[0][tid];
    float m = s_max[0][tid];
#pragma unroll
    for (int g = 1; g < RQ; ++g) {
      t += s_sum[g][tid];
      m = fmaxf(m, s_max[g][tid]);
    }
    const int64_t o = ((int64_t)bh * args.R + a) * D + tid;
    (which == 0 ? args.Qbar : args.Kbar)[o] = t / (double)n;
    (which == 0 ? args.Qmax : args.Kmax)[o] = (double)m;
  }
  if (tid == 0) {
    const float m = fmaxf(fmaxf(s_amax[0], s_amax[1]), fmaxf(s_amax[2], s_amax[3]));
    args.blkmax[((int64_t)which * args.B * args.H + bh) * args.R + a] = m;
  }
}

typedef double f64x4 __attribute__((ext_vector_type(4)));

// One 128x160 logit tile of one branch (blockIdx.z = 2*head + branch) on the
// float64 matrix cores: each wave owns a 64x80 quarter as 4x5 MFMA tiles of
// 16x16x4, so every query value loaded feeds five MFMAs and every key value
// four. (On R = 588 this makes 1,920 waves, which two waves per SIMD take in
// one round; 64x64 quarters made 2,400 and a thin second round.) The
// reduction over channels may visit them in any order as long as both
// operands agree: lane group q = lane/16 of k-step 2t+h reads channel
// 8t + 2q + h, so one 16-byte load per operand tile feeds two k-steps. The
// loads run one group of 8 channels ahead of the MFMAs, and consecutive MFMAs
// update different accumulators. Operand rows are addressed as 32-bit byte
// offsets from the branch's base (one VGPR each), which keeps the kernel
// within 256 VGPRs. Rows and columns beyond R read row R-1 and are not stored.
constexpr int kLogitTile = 128;  // rows per workgroup
constexpr int kLogitCols = 160;  // columns per workgroup
template <int D>
__global__ __launch_bounds__(256) void draft_logits_kernel(DraftArgs args) {
  constexpr int d = D, NI = 4, NJ = 5;
  const int R = args.R, bh = blockIdx.z >> 1, br = blockIdx.z & 1;
  const double* Qs = (br == 0 ? args.Qbar : args.Qmax) + (int64_t)bh * R * d;
  const double* Ks = (br == 0 ? args.Kbar : args.Kmax) + (int64_t)bh * R * d;
  double* out = (br == 0 ? args.S1 : args.S2) + (int64_t)bh * R * R;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, li = lane & 15, q = lane >> 4;
  const int r0 = blockIdx.y * kLogitTile + (wave >> 1) * 64, c0 = blockIdx.x * kLogitCols + (wave & 1) * 80;
  // byte offsets of each lane's operand rows from the branch's base (one VGPR each)
  uint32_t oa[NI], ob[NJ];
#pragma unroll
  for (int i = 0; i < NI; ++i) oa[i] = (uint32_t)(min(r0 + 16 * i + li, R - 1) * d + 2 * q) * 8u;
#pragma unroll
  for (int j = 0; j < NJ; ++j) ob[j] = (uint32_t)(min(c0 + 16 * j + li, R - 1) * d + 2 * q) * 8u;
  auto lda = [&](int i, int t) {
    return *reinterpret_cast<const double2*>(reinterpret_cast<const char*>(Qs) + oa[i] + 64 * t);
  };
  auto ldb = [&](int j, int t) {
    return *reinterpret_cast<const double2*>(reinterpret_cast<const char*>(Ks) + ob[j] + 64 * t);
  };
  f64x4 acc[NI][NJ];
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = f64x4{0.0, 0.0, 0.0, 0.0};
  double2 a[2][NI], b[2][NJ];  // [buffer][tile]
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    a[0][i] = lda(i, 0);
  }
#pragma unroll
  for (int j = 0; j < NJ; ++j) b[0][j] = ldb(j, 0);
#pragma unroll
  for (int t = 0; t < d / 8; ++t) {
    const int cur = t & 1;
    if (t + 1 < d / 8) {
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        a[cur ^ 1][i] = lda(i, t + 1);
      }
#pragma unroll
      for (int j = 0; j < NJ; ++j) b[cur ^ 1][j] = ldb(j, t + 1);
    }
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[cur][i].x, b[cur][j].x, acc[i][j], 0, 0, 0);
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[cur][i].y, b[cur][j].y, acc[i][j], 0, 0, 0);
  }
  // workgroup (0, 0, 2 head + branch) also reduces the per-block max |Q|
  // (branch 0) or max |K| (branch 1) of its head into the statistics entry
  if (blockIdx.x == 0 && blockIdx.y == 0) {
    __shared__ float s_red[4];
    const float* bm = args.blkmax + ((int64_t)br * args.B * args.H + bh) * R;
    float m = 0.0f;
    for (int i = threadIdx.x; i < R; i += 256) m = fmaxf(m, bm[i]);
    m = wave_max(m);
    if (lane == 0) s_red[wave] = m;
    __syncthreads();
    if (threadIdx.x == 0)
      args.stats[(int64_t)bh * (4 + d) + br] =
          __float_as_uint(fmaxf(fmaxf(s_red[0], s_red[1]), fmaxf(s_red[2], s_red[3])));
  }
  // accumulator element e of lane l: row l/16 + 4e, column l%16
  const double sqd = sqrt((double)d);
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = r0 + 16 * i + q + 4 * e, col = c0 + 16 * j + li;
        if (row < R && col < R) out[(int64_t)row * R + col] = acc[i][j][e] / sqd;
      }
}

__device__ inline double wave_max_f64(double v) {
  for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, 64));
  return v;
}

// e^x for x <= 0 in float64: Cody-Waite range reduction x = k ln2 + r with
// |r| <= ln2/2 (two multiply-adds, ln2 split into its nearest double and the
// remainder), then the Taylor series of e^r to degree 13 in Horner form (the
// truncation error is below 5e-18 relative on that interval) and ldexp(., k).
// The coefficients are 1/n! rounded to the nearest double; they live in
// constant memory, so the multiply-adds read them from scalar registers
// instead of copying each into a vector register first. Inputs below -746
// give 0, like e^x itself in float64; a NaN gives NaN.
__constant__ double kExpTaylor[14] = {1.0,
                                      1.0,
                                      0.5,
                                      0.16666666666666666,
                                      0.041666666666666664,
                                      0.008333333333333333,
                                      0.001388888888888889,
                                      0.0001984126984126984,
                                      2.48015873015873e-05,
                                      2.7557319223985893e-06,
                                      2.755731922398589e-07,
                                      2.505210838544172e-08,
                                      2.08767569878681e-09,
                                      1.6059043836821613e-10};
__device__ inline double exp_neg(double x) {
  constexpr double kLog2e = 1.4426950408889634, kLn2Hi = 0.6931471805599453, kLn2Lo = 2.3190468138462996e-17;
  x = x < -746.0 ? -746.0 : x;  // (a NaN stays NaN)
  const double k = rint(x * kLog2e);
  double r = fma(-k, kLn2Hi, x);
  r = fma(-k, kLn2Lo, r);
  double p = kExpTaylor[13];
#pragma unroll
  for (int n = 12; n >= 0; --n) p = fma(p, r, kExpTaylor[n]);
  return ldexp(p, static_cast<int>(k));
}

// One wave per row of A (four rows per workgroup): the two row softmaxes (max
// subtracted) mixed with weight lambda, rounded once to float32. Rows of up to
// 64 KMAX entries keep their logits and exponentials in registers (one exp per
// entry and branch); longer rows take the three-pass form below.
template <int KMAX>
__global__ __launch_bounds__(256) void draft_softmax_reg_kernel(DraftArgs args) {
  const int R = args.R, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= (int64_t)args.B * args.H * R) return;
  const double* s1 = args.S1 + row * R;
  const double* s2 = args.S2 + row * R;
  double e1[KMAX], e2[KMAX];
  double m1 = -INFINITY, m2 = -INFINITY;
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    const int i = lane + 64 * k;
    e1[k] = i < R ? s1[i] : -INFINITY;
    e2[k] = i < R ? s2[i] : -INFINITY;
    m1 = fmax(m1, e1[k]);
    m2 = fmax(m2, e2[k]);
  }
  m1 = wave_max_f64(m1);
  m2 = wave_max_f64(m2);
  double z1 = 0.0, z2 = 0.0;
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    const bool in = lane + 64 * k < R;
    e1[k] = in ? exp_neg(e1[k] - m1) : 0.0;
    e2[k] = in ? exp_neg(e2[k] - m2) : 0.0;
    z1 += e1[k];
    z2 += e2[k];
  }
  z1 = wave_sum_f64(z1);
  z2 = wave_sum_f64(z2);
  const double lam = args.lambda;
  // both normalizations and the mixing weights folded into one factor per
  // branch (float64; A is rounded once, to float32, at the end)
  const double r1 = (1.0 - lam) / z1, r2 = lam / z2;
  float* out = args.A + row * R;
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    const int i = lane + 64 * k;
    if (i < R) out[i] = (float)(e1[k] * r1 + e2[k] * r2);
  }
}

__global__ __launch_bounds__(256) void draft_softmax_kernel(DraftArgs args) {
  const int R = args.R, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= (int64_t)args.B * args.H * R) return;
  const double* s1 = args.S1 + row * R;
  const double* s2 = args.S2 + row * R;
  double m1 = -INFINITY, m2 = -INFINITY;
  for (int i = lane; i < R; i += 64) {
    m1 = fmax(m1, s1[i]);
    m2 = fmax(m2, s2[i]);
  }
  m1 = wave_max_f64(m1);
  m2 = wave_max_f64(m2);
  double z1 = 0.0, z2 = 0.0;
  for (int i = lane; i < R; i += 64) {
    z1 += exp_neg(s1[i] - m1);
    z2 += exp_neg(s2[i] - m2);
  }
  z1 = wave_sum_f64(z1);
  z2 = wave_sum_f64(z2);
  const double lam = args.lambda;
  const double r1 = (1.0 - lam) / z1, r2 = lam / z2;
  float* out = args.A + row * R;
  for (int i = lane; i < R; i += 64) out[i] = (float)(exp_neg(s1[i] - m1) * r1 + exp_neg(s2[i] - m2) * r2);
}

hipError_t launch_draft(const DraftArgs& args, hipStream_t stream) {
  const int BH = args.B * args.H;
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
  const int nt = (args.R + kLogitTile - 1) / kLogitTile, ntc = (args.R + kLogitCols - 1) / kLogitCols;
  if (args.d == 128)
    hipLaunchKernelGGL(draft_logits_kernel<128>, dim3(ntc, nt, 2 * BH), dim3(256), 0, stream, args);
  else
    hipLaunchKernelGGL(draft_logits_kernel<64>, dim3(ntc, nt, 2 * BH), dim3(256), 0, stream, args);
  const int64_t rows = (int64_t)BH * args.R;
  const dim3 sgrid((unsigned)((rows + 3) / 4));
  if (args.R <= 64 * 10)
    hipLaunchKernelGGL(draft_softmax_reg_kernel<10>, sgrid, dim3(256), 0, stream, args);
  else if (args.R <= 64 * 32)
    hipLaunchKernelGGL(draft_softmax_reg_kernel<32>, sgrid, dim3(256), 0, stream, args);
  else
    hipLaunchKernelGGL(draft_softmax_kernel, sgrid, dim3(256), 0, stream, args);
  return hipGetLastError();
}

}  // namespace da2
