// Operand preparation kernels (format appendix; NVFP4 quantization equation).
//
//   prep_vstats  token-major pass over V of each head: per-channel max|V| and
//                the head's max|V| (every token is a valid key).
//   prep_qk      one workgroup per (block, head, Q or K): gathers the block's
//                64 slots through slot2tok in 16-byte loads (unconditional, so
//                they overlap; padding slots are masked to 0);
//                each thread owns whole 16-channel groups, so the INT8 block
//                code and the NVFP4 group code of a group come from registers.
//   prep_v       one workgroup per (block, head): the V tile is staged in LDS
//                and read transposed, each thread owning channels c and c + d/2
//                and one 16-slot group (the NVFP4 group of V runs along
//                slots), so each store fills consecutive fragment lanes.
// Every encoding is written in the MFMA fragment order of the attention kernel
// (16-byte chunks, one per lane of a fragment):
//   INT8 Q, K with per-block scales, E4M3 V with per-channel scales,
//   NVFP4 Q, K (16-channel groups) and V (16-slot groups) as E2M1 codes with
//   one E4M3 scale byte per group, ordered by the attention thread that
//   decodes them (the per-head tensor scales and an encoding tag go to g),
//   and, when asked for, the half-precision Q, K, V of the 16-bit path in the
//   fp16 fragment order the NVFP4 codes decode to;
//   with the MXFP4 encoding instead of NVFP4: E2M1 codes of 32-element blocks
//   (channels for Q and K, key slots for V) with E8M0 scale words, in the
//   operand order of the scaled fp4 MFMA.
// Scale arithmetic is float32 with one rounding per operation in the documented
// order (the build uses -ffp-contract=off); division by a scale is a
// multiplication by its correctly rounded float32 reciprocal. The E2M1 and E4M3
// casts of scaled values use the gfx950 conversion instructions (round to
// nearest even, saturating, signed zeros kept; checked by the device format
// tests).
#include "common.hpp"
#include "launch.hpp"

namespace da2 {

__global__ void zero_vstats_kernel(uint32_t* stats, int d) {
  uint32_t* s = stats + (int64_t)blockIdx.x * (4 + d);
  for (int i = 2 + threadIdx.x; i < 4 + d; i += blockDim.x) s[i] = 0u;
}

// ---- V statistics -----------------------------------------------------------
constexpr int kVstatRows = 1024;  // tokens per workgroup (one atomic max per channel per workgroup)

template <int D, typename T>
__global__ __launch_bounds__(256) void prep_vstats_kernel(PrepArgs args) {
  constexpr int EPC = 16 / sizeof(T);   // elements per 16-byte load
  constexpr int CPR = D / EPC;          // loads per token row
  constexpr int RG = 256 / CPR;         // row groups
  constexpr int RPR = 16;               // rows per thread per round (loads in flight)
  constexpr int ROUNDS = kVstatRows / (RG * RPR);
  static_assert(ROUNDS * RG * RPR == kVstatRows, "whole rounds");
  __shared__ float s_max[4][D];
  __shared__ float s_all[4];
  const int bh = blockIdx.y, b = bh / args.H, h = bh % args.H, tid = threadIdx.x;
  const int cc = tid % CPR, rg = tid / CPR;
  const int t0 = blockIdx.x * kVstatRows;
  const T* X = static_cast<const T*>(args.V) + (int64_t)b * args.sb + (int64_t)h * args.sh + cc * EPC;
  float m[EPC];
#pragma unroll
  for (int e = 0; e < EPC; ++e) m[e] = 0.0f;
#pragma unroll 1
  for (int rd = 0; rd < ROUNDS; ++rd) {
    // unconditional loads so that they overlap: rows past the end read the
    // last token again, which changes no maximum
    uint4 raw[RPR];
#pragma unroll
    for (int k = 0; k < RPR; ++k) {
      const int t = min(t0 + rd * RG * RPR + rg + RG * k, args.N - 1);
      raw[k] = *reinterpret_cast<const uint4*>(X + (int64_t)t * args.sn);
    }
#pragma unroll
    for (int k = 0; k < RPR; ++k) {
      float x[EPC];
      chunk_floats<T>(raw[k], x);
#pragma unroll
      for (int e = 0; e < EPC; ++e) m[e] = fmaxf(m[e], fabsf(x[e]));
    }
  }
  // lanes with the same chunk column sit CPR apart in a wave
#pragma unroll
  for (int o = CPR; o < 64; o <<= 1)
#pragma unroll
    for (int e = 0; e < EPC; ++e) m[e] = fmaxf(m[e], __shfl_xor(m[e], o, 64));
  const int w = tid >> 6, lane = tid & 63;
  if (lane < CPR)
#pragma unroll
    for (int e = 0; e < EPC; ++e) s_max[w][cc * EPC + e] = m[e];
  __syncthreads();
  if (tid < D) {
    const float t = fmaxf(fmaxf(s_max[0][tid], s_max[1][tid]), fmaxf(s_max[2][tid], s_max[3][tid]));
    uint32_t* st = args.stats + (int64_t)bh * (4 + D);
    atomic_max_pos(st + 4 + tid, t);
    const float wm = wave_max(t);
    if ((tid & 63) == 0) s_all[tid >> 6] = wm;
  }
  __syncthreads();
  if (tid == 0) {
    float t = s_all[0];
    for (int q = 1; q < D / 64; ++q) t = fmaxf(t, s_all[q]);
    atomic_max_pos(args.stats + (int64_t)bh * (4 + D) + 2, t);
  }
}

// ---- shared encoders ------------------------------------------------------------
// Row (slot) of MFMA A-operand row r of key tile j: puts the 16-slot group
// 32j+16g+[0,16) of a query row into lane group g of the 32x32 accumulator.
__device__ inline int kappa(int j, int r) { return 32 * j + 16 * ((r >> 2) & 1) + 4 * (r >> 3) + (r & 3); }

// Eight values as fp16 (round to nearest even), one 16-byte chunk.
__device__ inline uint4 half8(const float* x) {
  f16x8 h;
#pragma unroll
  for (int e = 0; e < 8; ++e) h[e] = (_Float16)x[e];
  return __builtin_bit_cast(uint4, h);
}

__device__ inline float nvfp4_scale_global(uint32_t amax_bits) {
  const float g = __fdiv_rn(__uint_as_float(amax_bits), 2688.0f);
  return g == 0.0f ? 1.0f : g;
}

// INT8 codes of 16 values: round half away from zero of f32(x * inv), clamped.
__device__ inline uint4 int8_codes16(const float* x, float inv) {
  uint32_t w[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t packed = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      packed |= (static_cast<uint32_t>(int8_code(__fmul_rn(x[4 * q + e], inv))) & 0xFFu) << (8 * e);
    }
    w[q] = packed;
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// ---- MXFP4 / NVFP4 codes --------------------------------------------------------
// E2M1 codes of 8 values, value e in nibble e (low nibble first).
__device__ inline uint32_t fp4_codes8(const float* y) {
  uint32_t c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, y[0], y[1], 1.0f, 0);
  c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, y[2], y[3], 1.0f, 1);
  c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, y[4], y[5], 1.0f, 2);
  return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, y[6], y[7], 1.0f, 3);
}

// NVFP4 encoding of one 16-element group x with tensor scale gX (sixg =
// f32(6 gX)): the E2M1 codes of elements [0,8) and [8,16) (value e in nibble
// e) and the E4M3 code of the group scale sigma (a zero sigma gives zero codes;
// an E2M1 zero keeps the sign of its scaled value, as the hardware cast does).
__device__ inline void nvfp4_group16(const float* x, float gX, float sixg, uint32_t& lo, uint32_t& hi,
                                     uint32_t& scode) {
  float gm = 0.0f;
#pragma unroll
  for (int e = 0; e < 16; ++e) gm = fmaxf(gm, fabsf(x[e]));
  const float sigma = e4m3_round_mag(__fdiv_rn(gm, sixg));
  if (sigma == 0.0f) {
    lo = hi = scode = 0u;
    return;
  }
  const float inv = __fdiv_rn(1.0f, __fmul_rn(gX, sigma));
  float y[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) y[e] = __fmul_rn(x[e], inv);
  lo = fp4_codes8(y);
  hi = fp4_codes8(y + 8);
  scode = e4m3_code(sigma);  // sigma is an E4M3 value: its exact code
}

// ---- MXFP4 --------------------------------------------------------------------
// E8M0 exponent of a 32-element block with largest magnitude amax >= 0:
// floor(log2 amax) - 2, clamped below at -127 (zero and subnormal amax give
// -127); finite fp32 amax keeps it below 126.
__device__ inline int mx_exponent(float amax) { return max((int)(__float_as_uint(amax) >> 23) - 129, -127); }
// 2^-k as a float (normal for every k from mx_exponent).
__device__ inline float mx_inv_scale(int k) { return __uint_as_float(static_cast<uint32_t>(127 - k) << 23); }
// MXFP4 sections: bytes per block (d/32 data fragments and the scale fragment).
constexpr int mx_block_bytes(int D) { return 1024 * (D / 32 + 1); }

// ---- Q and K ----------------------------------------------------------------
template <int D, typename T>
__global__ __launch_bounds__(256) void prep_qk_kernel(PrepArgs args) {
  constexpr int EPC = 16 / sizeof(T);
  constexpr int NG = D / 16;                // 16-channel groups per slot
  constexpr int UPT = kCap * NG / 256;      // groups per thread
  constexpr int NS32 = D / 32, NS64 = D / 64;
  __shared__ float s_red[4];
  const int a = blockIdx.x, bh = blockIdx.y, which = blockIdx.z;  // which: 0 = Q, 1 = K
  const int b = bh / args.H, h = bh % args.H, R = args.R, tid = threadIdx.x;
  const Layout L = layout_view(args.layout, R, args.Npad);
  const int n = L.n_a[a];
  const int32_t* slots = L.slot2tok + (int64_t)a * kCap;
  const T* X = static_cast<const T*>(which == 0 ? args.Q : args.K) + (int64_t)b * args.sb + (int64_t)h * args.sh;
  const int64_t blk = (int64_t)bh * R + a;

  // group u: fragment row rr = 32 jq + r (slot rr for Q, kappa(jq, r) for K),
  // channels [16 c16, 16 c16 + 16)
  // token indices first, then the data loads, all unconditional (padding slots
  // read the last valid row and are zeroed), so the loads overlap
  constexpr int CPG = 16 / EPC;  // 16-byte chunks per group
  int tok[UPT];
#pragma unroll
  for (int k = 0; k < UPT; ++k) {
    const int u = tid + 256 * k, rr = u / NG;
    const int slot = which == 0 ? rr : kappa(rr >> 5, rr & 31);
    tok[k] = slots[min(slot, n - 1)];
  }
  uint4 raw[UPT][CPG];
#pragma unroll
  for (int k = 0; k < UPT; ++k) {
    const int c16 = (tid + 256 * k) % NG;
    const T* p = X + (int64_t)tok[k] * args.sn + 16 * c16;
#pragma unroll
    for (int q = 0; q < CPG; ++q) raw[k][q] = *reinterpret_cast<const uint4*>(p + q * EPC);
  }
  float x[UPT][16];
  float amax = 0.0f;
#pragma unroll
  for (int k = 0; k < UPT; ++k) {
    const int u = tid + 256 * k, rr = u / NG;
    const int slot = which == 0 ? rr : kappa(rr >> 5, rr & 31);
#pragma unroll
    for (int q = 0; q < CPG; ++q) chunk_floats<T>(masked(raw[k][q], lane_mask(slot < n)), x[k] + q * EPC);
#pragma unroll
    for (int e = 0; e < 16; ++e) amax = fmaxf(amax, fabsf(x[k][e]));
  }
  amax = wave_max(amax);
  if ((tid & 63) == 0) s_red[tid >> 6] = amax;
  __syncthreads();
  const float bmax = fmaxf(fmaxf(s_red[0], s_red[1]), fmaxf(s_red[2], s_red[3]));
  const float delta = __fadd_rn(__fdiv_rn(bmax, 127.0f), 1e-7f);
  const float inv8 = __fdiv_rn(1.0f, delta);
  if (tid == 0) (which == 0 ? args.dQ : args.dK)[blk] = delta;
  const float gX = nvfp4_scale_global(args.stats[(int64_t)bh * (4 + D) + which]);
  const float sixg = __fmul_rn(6.0f, gX);
  int8_t* out8 = (which == 0 ? args.Q8 : args.K8) + blk * (int64_t)kCap * D;
  uint8_t* out4 = (which == 0 ? args.Q4 : args.K4) + blk * (int64_t)nv_block_bytes(D);
#pragma unroll
  for (int k = 0; k < UPT; ++k) {
    const int u = tid + 256 * k, c16 = u % NG, rr = u / NG;
    const int jq = rr >> 5, r = rr & 31;
    // INT8 chunk: [jq][c16/2][lane = r + 32 (c16%2)][16]
    const int64_t c8 = ((int64_t)(jq * NS32 + (c16 >> 1)) * 64 + r + 32 * (c16 & 1)) * 16;
    *reinterpret_cast<uint4*>(out8 + c8) = int8_codes16(x[k], inv8);
    // fp16 chunks of the 16-bit path: [jq][c16][lane = r + 32 g][8] for halves g = 0, 1
    const int64_t c4 = ((int64_t)(jq * NG + c16) * 64 + r) * 8;
    if (args.fmt4 == DA2_FMT4_NVFP4) {
      // packed NVFP4: the codes of elements 8g + [0, 8) are dword c16 of lane
      // r + 32 g of tile jq; the scale is byte c16 of row r of tile jq
      uint32_t lo, hi, sc;
      nvfp4_group16(x[k], gX, sixg, lo, hi, sc);
      *reinterpret_cast<uint32_t*>(out4 + ((int64_t)(jq * 64 + r) * NG + c16) * 4) = lo;
      *reinterpret_cast<uint32_t*>(out4 + ((int64_t)(jq * 64 + r + 32) * NG + c16) * 4) = hi;
      out4[32 * D + (jq * 32 + r) * NG + c16] = static_cast<uint8_t>(sc);
    } else {
      // MXFP4: the 32-channel block is this group and its neighbour c16 ^ 1,
      // held by the adjacent lane. The group's 16 codes are half of a lane's
      // 16 bytes in data fragment (tile, s = c16/4), lane row + 32 ((c16/2)%2),
      // where (tile, row) places the slot by kappa_mx for K.
      float m16 = 0.0f;
#pragma unroll
      for (int e = 0; e < 16; ++e) m16 = fmaxf(m16, fabsf(x[k][e]));
      const int ke = mx_exponent(fmaxf(m16, __shfl_xor(m16, 1, 64)));
      const float inv = mx_inv_scale(ke);
      float y[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) y[e] = __fmul_rn(x[k][e], inv);  // exact (power of two)
      const int slot = which == 0 ? rr : kappa(jq, r);
      const int tile = which == 0 ? jq : (slot >> 4) & 1;
      const int row = which == 0 ? r : 8 * ((slot & 15) >> 2) + 4 * (slot >> 5) + (slot & 3);
      const int s = c16 >> 2, ml = row + 32 * ((c16 >> 1) & 1);
      uint8_t* base = (which == 0 ? args.Q4mx : args.K4mx) + blk * (int64_t)mx_block_bytes(D);
      *reinterpret_cast<uint2*>(base + ((tile * NS64 + s) * 64 + ml) * 16 + 8 * (c16 & 1)) =
          make_uint2(fp4_codes8(y), fp4_codes8(y + 8));
      if ((c16 & 1) == 0) {  // scale word tile*NS64+s of lane ml; unused words are zero
        uint32_t* sw = reinterpret_cast<uint32_t*>(base + (2 * NS64 * 64 + ml) * 16);
        sw[tile * NS64 + s] = static_cast<uint32_t>(ke + 127);
        if (2 * NS64 < 4 && tile == 0 && s == 0)
          for (int wd = 2 * NS64; wd < 4; ++wd) sw[wd] = 0u;
      }
    }
    if (args.with16) {  // 16-bit path: the same chunks as fp16(x)
      _Float16* out16 = (which == 0 ? args.Q16 : args.K16) + blk * (int64_t)kCap * D;
      *reinterpret_cast<uint4*>(out16 + c4) = half8(x[k]);
      *reinterpret_cast<uint4*>(out16 + c4 + 32 * 8) = half8(x[k] + 8);
    }
  }
}

// ---- V ------------------------------------------------------------------------

template <int D, typename T>
__global__ __launch_bounds__(256) void prep_v_kernel(PrepArgs args) {
  constexpr int EPC = 16 / sizeof(T);
  constexpr int CPR = D / EPC;
  constexpr int LPT = kCap * CPR / 256;  // 16-byte loads per thread
  __shared__ __align__(16) T tile[kCap * D];
  const int a = blockIdx.x, bh = blockIdx.y;
  const int b = bh / args.H, h = bh % args.H, R = args.R, tid = threadIdx.x;
  const Layout L = layout_view(args.layout, R, args.Npad);
  const int n = L.n_a[a];
  const int32_t* slots = L.slot2tok + (int64_t)a * kCap;
  const T* X = static_cast<const T*>(args.V) + (int64_t)b * args.sb + (int64_t)h * args.sh;
  const uint32_t* st = args.stats + (int64_t)bh * (4 + D);
  const int64_t blk = (int64_t)bh * R + a;

  // token indices first, then the data loads, all unconditional (padding slots
  // read the last valid row and are zeroed), so the loads overlap
  int tok[LPT];
#pragma unroll
  for (int k = 0; k < LPT; ++k) tok[k] = slots[min((tid + 256 * k) / CPR, n - 1)];
  uint4 v[LPT];
#pragma unroll
  for (int k = 0; k < LPT; ++k) {
    const int ci = tid + 256 * k, s = ci / CPR, cc = ci % CPR;
    const uint4 x = *reinterpret_cast<const uint4*>(X + (int64_t)tok[k] * args.sn + cc * EPC);
    v[k] = masked(x, lane_mask(s < n));
  }
  // this thread's statistics (the head's NVFP4 amax and the amax of channels
  // p and p + D/2), loaded beside the tile rather than after the barrier
  const int p = tid % (D / 2), sg = tid / (D / 2);
  const uint32_t st_g = st[2], st_c0 = st[4 + p], st_c1 = st[4 + p + D / 2];
#pragma unroll
  for (int k = 0; k < LPT; ++k) {
    const int ci = tid + 256 * k;
    reinterpret_cast<uint4*>(tile)[ci] = v[k];
  }
  __syncthreads();

  // unit: channels p and p + D/2, 16-slot group sg (consecutive threads own
  // consecutive channels, so each store instruction below fills consecutive
  // 16-byte lanes of a fragment)
  if (sg < 4) {
    float x0[16], x1[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      x0[i] = tile_value(tile, D, 16 * sg + i, p);
      x1[i] = tile_value(tile, D, 16 * sg + i, p + D / 2);
    }
    const float gV = nvfp4_scale_global(st_g);
    const float sixg = __fmul_rn(6.0f, gV);
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const float* xc = q == 0 ? x0 : x1;
      const int c = p + q * (D / 2);
      const int lane = (c & 31) + 32 * (sg & 1), t = c >> 5;
      // E4M3, per-channel scale: chunk [t][h = sg/2][lane][16]
      const float dlt = __fdiv_rn(__uint_as_float(q == 0 ? st_c0 : st_c1), 2.25f);
      uint4 code = make_uint4(0u, 0u, 0u, 0u);
      if (dlt != 0.0f) {
        const float inv = __fdiv_rn(1.0f, dlt);
        uint32_t w[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          int lo = __builtin_amdgcn_cvt_pk_fp8_f32(__fmul_rn(xc[4 * j], inv), __fmul_rn(xc[4 * j + 1], inv), 0, false);
          w[j] = static_cast<uint32_t>(__builtin_amdgcn_cvt_pk_fp8_f32(__fmul_rn(xc[4 * j + 2], inv),
                                                                       __fmul_rn(xc[4 * j + 3], inv), lo, true));
        }
        code = make_uint4(w[0], w[1], w[2], w[3]);
      }
      *reinterpret_cast<uint4*>(args.V8 + blk * (int64_t)kCap * D + ((int64_t)(2 * t + (sg >> 1)) * 64 + lane) * 16) = code;
      // fp16 chunks of the 16-bit path: [t][s = 2 (sg/2) + half][lane][8]
      const int64_t c4 = blk * (int64_t)kCap * D + ((int64_t)(4 * t + 2 * (sg >> 1)) * 64 + lane) * 8;
      if (args.fmt4 == DA2_FMT4_NVFP4) {
        // packed NVFP4 along slots: channel tile t = w NT/2 + t2 belongs to
        // attention wave w; the codes of fragments s = 2 (sg/2) and 2 (sg/2) + 1
        // are dwords s of the lane's tile t2, the scale is byte h = sg/2
        constexpr int NTH = D / 64;  // channel tiles per wave
        const int w = t / NTH, t2 = t % NTH;
        uint32_t lo, hi, sc;
        nvfp4_group16(xc, gV, sixg, lo, hi, sc);
        uint8_t* base = args.V4 + blk * (int64_t)nv_block_bytes(D);
        *reinterpret_cast<uint2*>(base + ((int64_t)((w * 64 + lane) * NTH + t2) * 4 + 2 * (sg >> 1)) * 4) =
            make_uint2(lo, hi);
        base[32 * D + ((w * 64 + lane) * NTH + t2) * 2 + (sg >> 1)] = static_cast<uint8_t>(sc);
      }
      if (args.with16) {  // 16-bit path: the same chunks as fp16(v)
        *reinterpret_cast<uint4*>(args.V16 + c4) = half8(xc);
        *reinterpret_cast<uint4*>(args.V16 + c4 + 64 * 8) = half8(xc + 8);
      }
    }
  }
  // MXFP4 along slots: unit = channels p and p + D/2, 32-slot block hb; the block's
  // 32 codes fill the 16 bytes of lane c%32 + 32 hb in data fragment t = c/32.
  constexpr int NT = D / 32;
  if (args.fmt4 == DA2_FMT4_MXFP4 && tid < D) {
    const int hb = tid / (D / 2);
    float x0[32], x1[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      x0[i] = tile_value(tile, D, 32 * hb + i, p);
      x1[i] = tile_value(tile, D, 32 * hb + i, p + D / 2);
    }
    uint8_t* base = args.V4mx + blk * (int64_t)mx_block_bytes(D);
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      float* xc = q == 0 ? x0 : x1;
      const int c = p + q * (D / 2), t = c >> 5, ml = (c & 31) + 32 * hb;
      float m = 0.0f;
#pragma unroll
      for (int i = 0; i < 32; ++i) m = fmaxf(m, fabsf(xc[i]));
      const int ke = mx_exponent(m);
      const float inv = mx_inv_scale(ke);
#pragma unroll
      for (int i = 0; i < 32; ++i) xc[i] = __fmul_rn(xc[i], inv);  // exact (power of two)
      *reinterpret_cast<uint4*>(base + (t * 64 + ml) * 16) =
          make_uint4(fp4_codes8(xc), fp4_codes8(xc + 8), fp4_codes8(xc + 16), fp4_codes8(xc + 24));
      uint32_t* sw = reinterpret_cast<uint32_t*>(base + (NT * 64 + ml) * 16);
      sw[t] = static_cast<uint32_t>(ke + 127);
      if (NT < 4 && t == 0)
        for (int wd = NT; wd < 4; ++wd) sw[wd] = 0u;
    }
  }
  if (a == 0) {
    if (tid < D) args.dV[(int64_t)bh * D + tid] = __fdiv_rn(__uint_as_float(st[4 + tid]), 2.25f);
    if (tid < 4) args.g[(int64_t)bh * 4 + tid] = tid < 3 ? nvfp4_scale_global(st[tid]) : __uint_as_float(args.tag);
  }
}

template <int D, typename T>
void launch_prep_t(const PrepArgs& args, hipStream_t stream) {
  const int BH = args.B * args.H;
  hipLaunchKernelGGL(zero_vstats_kernel, dim3(BH), dim3(64), 0, stream, args.stats, args.d);
  hipLaunchKernelGGL((prep_vstats_kernel<D, T>), dim3((args.N + kVstatRows - 1) / kVstatRows, BH), dim3(256), 0,
                     stream, args);
  hipLaunchKernelGGL((prep_qk_kernel<D, T>), dim3(args.R, BH, 2), dim3(256), 0, stream, args);
  hipLaunchKernelGGL((prep_v_kernel<D, T>), dim3(args.R, BH), dim3(256), 0, stream, args);
}

hipError_t launch_prep(const PrepArgs& args, hipStream_t stream) {
  if (args.d == 128) {
    if (args.dtype == DA2_BF16)
      launch_prep_t<128, uint16_t>(args, stream);
    else
      launch_prep_t<128, float>(args, stream);
  } else {
    if (args.dtype == DA2_BF16)
      launch_prep_t<64, uint16_t>(args, stream);
    else
      launch_prep_t<64, float>(args, stream);
  }
  return hipGetLastError();
}

}  // namespace da2
