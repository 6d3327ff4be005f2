// Phased mixed-precision attention (phased-execution appendix; precision-state-
// conversion equation; NVFP4 probability equation; INT8 paragraph).
//
// One wavefront owns one query block a (64 query slots = two 32-query tiles qt)
// and walks its retained key blocks: the NVFP4 ones in ascending order, then the
// INT8 ones. All blocks share the fp32 running maxima m, the denominators l and
// the numerator U.
//
// Tiles use 32x32 MFMAs with the transposed products
//     S^T = K Q^T      (rows = key slots, cols = queries)
//     O^T = V^T P^T    (rows = channels,  cols = queries)
// so that accumulator lane l always holds query 32qt + l%32: row statistics are
// lane-local up to one exchange between the two lane halves. The key rows of
// S^T are permuted (kappa) so lane half g of key tile j holds the logical slots
// 32j+16g+[0,16), i.e. one whole 16-slot NVFP4 probability group; the same
// registers then feed the P^T operand of O^T with V rows in the matching order
// (the operand permutation equation (P Pi)(Pi^T V) = P V).
//
// Units: the 4-bit phase multiplies fp16 sigma*e operands, so U carries a factor
// 2688/g_V and l the unamplified weights; Enter converts to the 8-bit path's
// units U_c / (eta delta_c), l / eta; the 8-bit phase accumulates amplified
// weights 2^(z - m + 8.807) and E4M3 codes; Exit converts back.
#include "common.hpp"
#include "launch.hpp"

namespace da2 {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kExpOffset = 8.807f;

__device__ inline float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

template <int NT>
__device__ inline void rescale(f32x16 (&U)[NT], float alpha) {
#pragma unroll
  for (int t = 0; t < NT; ++t) U[t] *= alpha;
}

// Running-max update for one 32-query tile: bm_in is this lane's maximum raw
// logit of the block (-inf on padding), scale converts raw logits to log2 units.
// Rescales l and U by 2^(m_old - m_new) and returns m_new.
template <int NT>
__device__ inline float update_max(float bm_in, float scale, float& m, float& l, f32x16 (&U)[NT]) {
  float bm = fmaxf(bm_in, __shfl_xor(bm_in, 32, 64));
  const float mn = fmaxf(m, bm * scale);
  const float alpha = exp2_fast(m - mn);
  m = mn;
  l *= alpha;
  if (__ballot(alpha != 1.0f)) rescale<NT>(U, alpha);
  return mn;
}

template <int D>
__global__ __launch_bounds__(64) void mixed_attn_kernel(AttnArgs args) {
  constexpr int NS16 = D / 16, NS32 = D / 32, NT = D / 32;
  const int lane = threadIdx.x, r = lane & 31, g = lane >> 5;
  const int R = args.R;
  const int item = args.order[blockIdx.x];
  const int bh = item / R, a = item % R;
  const Layout L = layout_view(args.layout, R, args.Npad);
  const int n4 = args.counts[2 * item], n8 = args.counts[2 * item + 1];
  const uint16_t* keys = args.keys + (int64_t)item * R;
  const int64_t blk0 = (int64_t)bh * R;  // first block of this head
  const float rsqd = 1.0f / sqrtf((float)D);

  f32x16 U[2][NT];
#pragma unroll
  for (int qt = 0; qt < 2; ++qt)
#pragma unroll
    for (int t = 0; t < NT; ++t) U[qt][t] = f32x16{};
  float m[2] = {-INFINITY, -INFINITY}, l[2] = {0.0f, 0.0f};
  const float gV = args.g[bh * 4 + 2];

  // ------------------------------ NVFP4 phase ------------------------------
  if (n4 > 0) {
    const float c4 = args.g[bh * 4 + 0] * args.g[bh * 4 + 1] * kLog2e * rsqd;
    f16x8 Qf[2][NS16];
    const _Float16* Qa = args.Q4 + (blk0 + a) * (int64_t)kCap * D;
#pragma unroll
    for (int qt = 0; qt < 2; ++qt)
#pragma unroll
      for (int s = 0; s < NS16; ++s) Qf[qt][s] = *reinterpret_cast<const f16x8*>(Qa + ((qt * NS16 + s) * 64 + lane) * 8);

    for (int it = 0; it < n4; ++it) {
      const int kb = keys[it];
      const int nb = L.n_a[kb];
      const _Float16* Kb = args.K4 + (blk0 + kb) * (int64_t)kCap * D;
      const _Float16* Vb = args.V4 + (blk0 + kb) * (int64_t)kCap * D;
      f32x16 S[2][2];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        S[0][j] = f32x16{};
        S[1][j] = f32x16{};
#pragma unroll
        for (int s = 0; s < NS16; ++s) {
          const f16x8 kf = *reinterpret_cast<const f16x8*>(Kb + ((j * NS16 + s) * 64 + lane) * 8);
          S[0][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kf, Qf[0][s], S[0][j], 0, 0, 0);
          S[1][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kf, Qf[1][s], S[1][j], 0, 0, 0);
        }
      }
      f16x8 Pf[2][4];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        float gm[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          if (nb < kCap) {
#pragma unroll
            for (int i = 0; i < 16; ++i)
              if (32 * j + 16 * g + i >= nb) S[qt][j][i] = -INFINITY;
          }
          float x = S[qt][j][0];
#pragma unroll
          for (int i = 1; i < 16; ++i) x = fmaxf(x, S[qt][j][i]);
          gm[j] = x;
        }
        const float mn = update_max<NT>(fmaxf(gm[0], gm[1]), c4, m[qt], l[qt], U[qt]);
        float lsum = 0.0f;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          // group maximum of Pt = exp2 of the group's maximum logit
          const float pmax = exp2_fast(__builtin_fmaf(gm[j], c4, -mn));
          const float sigma = e4m3_round_mag(448.0f * pmax);
          const float rs = sigma == 0.0f ? 0.0f : __fdiv_rn(2688.0f, sigma);
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const float p = exp2_fast(__builtin_fmaf(S[qt][j][i], c4, -mn));
            lsum += p;
            Pf[qt][2 * j + (i >> 3)][i & 7] = (_Float16)(sigma * e2m1_round(p * rs));
          }
        }
        l[qt] += lsum;
      }
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const f16x8 vf = *reinterpret_cast<const f16x8*>(Vb + ((t * 4 + s) * 64 + lane) * 8);
          U[0][t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vf, Pf[0][s], U[0][t], 0, 0, 0);
          U[1][t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vf, Pf[1][s], U[1][t], 0, 0, 0);
        }
    }
  }

  // per-lane channel of accumulator register i of channel tile t
  auto chan = [&](int t, int i) { return 32 * t + 8 * (i >> 2) + 4 * g + (i & 3); };
  const float eta = exp2_fast(-kExpOffset);
  const float* dV = args.dV + (int64_t)bh * D;

  // ------------------------------- INT8 phase -------------------------------
  if (n8 > 0) {
    // Enter: U_c <- U_c / (eta delta_c), l <- l / eta (after restoring the 4-bit
    // phase's factor g_V/2688).
    const float restore = n4 > 0 ? gV / 2688.0f : 1.0f;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float dc = dV[chan(t, i)];
        const float f = dc == 0.0f ? 0.0f : restore / (eta * dc);
        U[0][t][i] *= f;
        U[1][t][i] *= f;
      }
    l[0] /= eta;
    l[1] /= eta;

    i32x4 Qf[2][NS32];
    const int8_t* Qa = args.Q8 + (blk0 + a) * (int64_t)kCap * D;
#pragma unroll
    for (int qt = 0; qt < 2; ++qt)
#pragma unroll
      for (int s = 0; s < NS32; ++s) Qf[qt][s] = *reinterpret_cast<const i32x4*>(Qa + ((qt * NS32 + s) * 64 + lane) * 16);
    const float c8a = args.dQ[blk0 + a] * kLog2e * rsqd;

    for (int it = 0; it < n8; ++it) {
      const int kb = keys[n4 + it];
      const int nb = L.n_a[kb];
      const float cb = c8a * args.dK[blk0 + kb];
      const int8_t* Kb = args.K8 + (blk0 + kb) * (int64_t)kCap * D;
      const uint8_t* Vb = args.V8 + (blk0 + kb) * (int64_t)kCap * D;
      i32x16 S[2][2];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        S[0][j] = i32x16{};
        S[1][j] = i32x16{};
#pragma unroll
        for (int s = 0; s < NS32; ++s) {
          const i32x4 kf = *reinterpret_cast<const i32x4*>(Kb + ((j * NS32 + s) * 64 + lane) * 16);
          S[0][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(kf, Qf[0][s], S[0][j], 0, 0, 0);
          S[1][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(kf, Qf[1][s], S[1][j], 0, 0, 0);
        }
      }
      long Pf[2][4];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        float sf[2][16];
        float bm = -INFINITY;
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            float v = (float)S[qt][j][i];
            if (nb < kCap && 32 * j + 16 * g + i >= nb) v = -INFINITY;
            sf[j][i] = v;
            bm = fmaxf(bm, v);
          }
        const float mn = update_max<NT>(bm, cb, m[qt], l[qt], U[qt]);
        const float off = kExpOffset - mn;
        float lsum = 0.0f;
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int h2 = 0; h2 < 2; ++h2) {
            float p[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              p[e] = exp2_fast(__builtin_fmaf(sf[j][8 * h2 + e], cb, off));
              lsum += p[e];
            }
            int lo = __builtin_amdgcn_cvt_pk_fp8_f32(p[0], p[1], 0, false);
            lo = __builtin_amdgcn_cvt_pk_fp8_f32(p[2], p[3], lo, true);
            int hi = __builtin_amdgcn_cvt_pk_fp8_f32(p[4], p[5], 0, false);
            hi = __builtin_amdgcn_cvt_pk_fp8_f32(p[6], p[7], hi, true);
            Pf[qt][2 * j + h2] = (long)(((unsigned long)(unsigned)hi << 32) | (unsigned)lo);
          }
        l[qt] += lsum;
      }
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const long vf = *reinterpret_cast<const long*>(Vb + ((t * 2 + (s >> 1)) * 64 + lane) * 16 + 8 * (s & 1));
          U[0][t] = __builtin_amdgcn_mfma_f32_32x32x16_fp8_fp8(vf, Pf[0][s], U[0][t], 0, 0, 0);
          U[1][t] = __builtin_amdgcn_mfma_f32_32x32x16_fp8_fp8(vf, Pf[1][s], U[1][t], 0, 0, 0);
        }
    }
    // Exit: U_c <- eta delta_c U_c, l <- eta l
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float f = eta * dV[chan(t, i)];
        U[0][t][i] *= f;
        U[1][t][i] *= f;
      }
    l[0] *= eta;
    l[1] *= eta;
  } else if (n4 > 0) {
    const float restore = gV / 2688.0f;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      U[0][t] *= restore;
      U[1][t] *= restore;
    }
  }

  // ------------------------- normalize and scatter -------------------------
  const int nq = L.n_a[a];
  const int32_t* s2t = L.slot2tok + (int64_t)a * kCap;
  const int b = bh / args.H, h = bh % args.H;
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    const float lt = l[qt] + __shfl_xor(l[qt], 32, 64);
    const float inv = lt > 0.0f ? 1.0f / lt : 0.0f;
    const int q = 32 * qt + r;
    if (q < nq) {
      const int64_t row = (int64_t)b * args.ob + (int64_t)h * args.oh + (int64_t)s2t[q] * args.on;
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float v = U[qt][t][i] * inv;
          if (args.odtype == DA2_FP32) {
            reinterpret_cast<float*>(args.O)[row + chan(t, i)] = v;
          } else {
            const uint32_t u = __float_as_uint(v);
            const uint32_t rb = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
            reinterpret_cast<uint16_t*>(args.O)[row + chan(t, i)] = static_cast<uint16_t>(rb);
          }
        }
    }
  }
}

hipError_t launch_attn(const AttnArgs& args, hipStream_t stream) {
  const int items = args.B * args.H * args.R;
  if (args.d == 128)
    hipLaunchKernelGGL(mixed_attn_kernel<128>, dim3(items), dim3(64), 0, stream, args);
  else
    hipLaunchKernelGGL(mixed_attn_kernel<64>, dim3(items), dim3(64), 0, stream, args);
  return hipGetLastError();
}

}  // namespace da2
