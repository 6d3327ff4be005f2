// Operand preparation kernels (format appendix; NVFP4 quantization equation).
//
//   prep_vstats   per (b,h,channel) max|V| over valid keys and per-head max|V|.
//   prep_encode   one workgroup per (block, head): stages the 64-slot tile of Q,
//                 K and V in LDS (gathered through slot2tok, padding = 0) and
//                 writes every encoding in the MFMA fragment order of the
//                 attention kernel (16-byte chunks, one per lane of a fragment):
//                   INT8 Q, K with per-block scales,
//                   E4M3 V with per-channel scales,
//                   NVFP4 Q, K (16-channel groups) and V (16-slot groups) as the
//                   exact fp16 value sigma*e.
// Scale arithmetic is float32 with one rounding per operation in the documented
// order (the build uses -ffp-contract=off); division by a scale is a
// multiplication by its correctly rounded float32 reciprocal.
#include "common.hpp"
#include "launch.hpp"

namespace da2 {

__global__ void zero_vstats_kernel(uint32_t* stats, int d) {
  uint32_t* s = stats + (int64_t)blockIdx.x * (4 + d);
  for (int i = 2 + threadIdx.x; i < 4 + d; i += blockDim.x) s[i] = 0u;
}

template <int D>
__global__ __launch_bounds__(256) void prep_vstats_kernel(PrepArgs args) {
  constexpr int G = 256 / D;
  __shared__ float s_max[G][D];
  const int a = blockIdx.x, bh = blockIdx.y;
  const int b = bh / args.H, h = bh % args.H;
  const Layout L = layout_view(args.layout, args.R, args.Npad);
  const int n = L.n_a[a];
  const int32_t* slots = L.slot2tok + (int64_t)a * kCap;
  const int c = threadIdx.x % D, grp = threadIdx.x / D;
  const int64_t base = (int64_t)b * args.sb + (int64_t)h * args.sh;
  float m = 0.0f;
  for (int i = grp; i < n; i += G) m = fmaxf(m, fabsf(load_elem(args.V, base + (int64_t)slots[i] * args.sn + c, args.dtype)));
  s_max[grp][c] = m;
  __syncthreads();
  if (threadIdx.x < D) {
    float t = s_max[0][c];
    for (int q = 1; q < G; ++q) t = fmaxf(t, s_max[q][c]);
    uint32_t* st = args.stats + (int64_t)bh * (4 + D);
    atomic_max_pos(st + 4 + c, t);
    atomic_max_pos(st + 2, t);
  }
}

// Row (slot) of MFMA A-operand row r of key tile j: puts the 16-slot group
// 32j+16g+[0,16) of a query row into lane group g of the 32x32 accumulator.
__device__ inline int kappa(int j, int r) { return 32 * j + 16 * ((r >> 2) & 1) + 4 * (r >> 3) + (r & 3); }

__device__ inline float nvfp4_scale_global(uint32_t amax_bits) {
  const float g = __fdiv_rn(__uint_as_float(amax_bits), 2688.0f);
  return g == 0.0f ? 1.0f : g;
}

template <int D>
__global__ __launch_bounds__(256) void prep_encode_kernel(PrepArgs args) {
  constexpr int LD = D + 1;
  constexpr int NS16 = D / 16, NS32 = D / 32;
  __shared__ float tile[kCap * LD];
  __shared__ float s_red[4];
  __shared__ float s_invc[D];  // E4M3 V: f32(1/delta_c) (0 for a zero channel)
  const int a = blockIdx.x, bh = blockIdx.y;
  const int b = bh / args.H, h = bh % args.H;
  const int R = args.R;
  const Layout L = layout_view(args.layout, R, args.Npad);
  const int n = L.n_a[a];
  const int32_t* slots = L.slot2tok + (int64_t)a * kCap;
  const int64_t base = (int64_t)b * args.sb + (int64_t)h * args.sh;
  const uint32_t* st = args.stats + (int64_t)bh * (4 + D);
  const int64_t blk = (int64_t)bh * R + a;  // block index in [B*H*R]
  const int tid = threadIdx.x;

  for (int which = 0; which < 3; ++which) {
    const void* X = which == 0 ? args.Q : (which == 1 ? args.K : args.V);
    // ---- stage the tile (slot order, padding 0) and its abs max ----
    float amax = 0.0f;
    for (int e = tid; e < kCap * D; e += 256) {
      const int s = e / D, c = e % D;
      float x = 0.0f;
      if (s < n) x = load_elem(X, base + (int64_t)slots[s] * args.sn + c, args.dtype);
      tile[s * LD + c] = x;
      amax = fmaxf(amax, fabsf(x));
    }
    amax = wave_max(amax);
    if ((tid & 63) == 0) s_red[tid >> 6] = amax;
    if (which == 2 && tid < D) {
      const float dlt = __fdiv_rn(__uint_as_float(st[4 + tid]), 2.25f);
      s_invc[tid] = dlt == 0.0f ? 0.0f : __fdiv_rn(1.0f, dlt);
    }
    __syncthreads();
    const float gX = nvfp4_scale_global(st[which]);
    const float sixg = __fmul_rn(6.0f, gX);

    if (which < 2) {
      // ---- INT8, per-block scale ----
      const float bmax = fmaxf(fmaxf(s_red[0], s_red[1]), fmaxf(s_red[2], s_red[3]));
      const float delta = __fadd_rn(__fdiv_rn(bmax, 127.0f), 1e-7f);
      const float inv = __fdiv_rn(1.0f, delta);
      if (tid == 0) (which == 0 ? args.dQ : args.dK)[blk] = delta;
      int8_t* out8 = (which == 0 ? args.Q8 : args.K8) + blk * (int64_t)kCap * D;
      for (int ch = tid; ch < 2 * NS32 * 64; ch += 256) {  // 16-byte chunks
        const int lane = ch & 63, s = (ch >> 6) % NS32, jq = (ch >> 6) / NS32;
        const int r = lane & 31, gg = lane >> 5;
        const int slot = which == 0 ? 32 * jq + r : kappa(jq, r);
        const float* row = tile + slot * LD + 32 * s + 16 * gg;
        uint32_t w[4];
        for (int q = 0; q < 4; ++q) {
          uint32_t packed = 0;
          for (int e = 0; e < 4; ++e) {
            float y = __fmul_rn(row[4 * q + e], inv);
            float v = fminf(fmaxf(roundf(y), -127.0f), 127.0f);
            packed |= (static_cast<uint32_t>(static_cast<int>(v)) & 0xFFu) << (8 * e);
          }
          w[q] = packed;
        }
        *reinterpret_cast<uint4*>(out8 + (int64_t)ch * 16) = make_uint4(w[0], w[1], w[2], w[3]);
      }
      // ---- NVFP4 along channels ----
      _Float16* out4 = (which == 0 ? args.Q4 : args.K4) + blk * (int64_t)kCap * D;
      for (int ch = tid; ch < 2 * NS16 * 64; ch += 256) {
        const int lane = ch & 63, s = (ch >> 6) % NS16, jq = (ch >> 6) / NS16;
        const int r = lane & 31, gg = lane >> 5;
        const int slot = which == 0 ? 32 * jq + r : kappa(jq, r);
        const float* grp = tile + slot * LD + 16 * s;
        float gm = 0.0f;
        for (int e = 0; e < 16; ++e) gm = fmaxf(gm, fabsf(grp[e]));
        const float sigma = e4m3_round_mag(__fdiv_rn(gm, sixg));
        f16x8 o;
        if (sigma == 0.0f) {
          for (int e = 0; e < 8; ++e) o[e] = (_Float16)0.0f;
        } else {
          const float inv = __fdiv_rn(1.0f, __fmul_rn(gX, sigma));
          for (int e = 0; e < 8; ++e) o[e] = (_Float16)__fmul_rn(sigma, e2m1_round(__fmul_rn(grp[8 * gg + e], inv)));
        }
        *reinterpret_cast<f16x8*>(out4 + (int64_t)ch * 8) = o;
      }
    } else {
      // ---- E4M3 V, per-channel scale; layout [t][h2][lane][16] ----
      uint8_t* out8 = args.V8 + blk * (int64_t)kCap * D;
      for (int ch = tid; ch < NS32 * 2 * 64; ch += 256) {
        const int lane = ch & 63, h2 = (ch >> 6) & 1, t = ch >> 7;
        const int c = 32 * t + (lane & 31), s0 = 32 * h2 + 16 * (lane >> 5);
        const float inv = s_invc[c];
        uint32_t w[4];
        for (int q = 0; q < 4; ++q) {
          uint32_t packed = 0;
          for (int e = 0; e < 4; ++e) {
            const uint32_t code = inv == 0.0f ? 0u : e4m3_code(__fmul_rn(tile[(s0 + 4 * q + e) * LD + c], inv));
            packed |= code << (8 * e);
          }
          w[q] = packed;
        }
        *reinterpret_cast<uint4*>(out8 + (int64_t)ch * 16) = make_uint4(w[0], w[1], w[2], w[3]);
      }
      // ---- NVFP4 V along key slots; layout [t][s:4][lane][8] ----
      _Float16* out4 = args.V4 + blk * (int64_t)kCap * D;
      for (int ch = tid; ch < NS32 * 4 * 64; ch += 256) {
        const int lane = ch & 63, s = (ch >> 6) & 3, t = ch >> 8;
        const int c = 32 * t + (lane & 31), gg = lane >> 5;
        const int g0 = 32 * (s >> 1) + 16 * gg;           // first slot of the 16-slot group
        const int e0 = g0 + 8 * (s & 1);                  // first slot of this chunk
        float gm = 0.0f;
        for (int e = 0; e < 16; ++e) gm = fmaxf(gm, fabsf(tile[(g0 + e) * LD + c]));
        const float sigma = e4m3_round_mag(__fdiv_rn(gm, sixg));
        f16x8 o;
        if (sigma == 0.0f) {
          for (int e = 0; e < 8; ++e) o[e] = (_Float16)0.0f;
        } else {
          const float inv = __fdiv_rn(1.0f, __fmul_rn(gX, sigma));
          for (int e = 0; e < 8; ++e) o[e] = (_Float16)__fmul_rn(sigma, e2m1_round(__fmul_rn(tile[(e0 + e) * LD + c], inv)));
        }
        *reinterpret_cast<f16x8*>(out4 + (int64_t)ch * 8) = o;
      }
      if (a == 0) {
        if (tid < D) {
          args.dV[(int64_t)bh * D + tid] = __fdiv_rn(__uint_as_float(st[4 + tid]), 2.25f);
        }
        if (tid < 4) {
          args.g[(int64_t)bh * 4 + tid] = tid < 3 ? nvfp4_scale_global(st[tid]) : 0.0f;
        }
      }
    }
    __syncthreads();
  }
}

hipError_t launch_prep(const PrepArgs& args, hipStream_t stream) {
  const int BH = args.B * args.H;
  hipLaunchKernelGGL(zero_vstats_kernel, dim3(BH), dim3(64), 0, stream, args.stats, args.d);
  if (args.d == 128) {
    hipLaunchKernelGGL(prep_vstats_kernel<128>, dim3(args.R, BH), dim3(256), 0, stream, args);
    hipLaunchKernelGGL(prep_encode_kernel<128>, dim3(args.R, BH), dim3(256), 0, stream, args);
  } else {
    hipLaunchKernelGGL(prep_vstats_kernel<64>, dim3(args.R, BH), dim3(256), 0, stream, args);
    hipLaunchKernelGGL(prep_encode_kernel<64>, dim3(args.R, BH), dim3(256), 0, stream, args);
  }
  return hipGetLastError();
}

}  // namespace da2
