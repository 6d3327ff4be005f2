// Shared device helpers of the da2 kernels (gfx950 only).
//
// Number formats of the paper's format appendix, encoded with integer bit
// manipulation on IEEE float32 (OCP E4M3FN: bias 7, 3 mantissa bits, max 448;
// OCP E2M1: 1 mantissa bit, max 6). Rounding is to nearest even with
// saturation at the largest finite value.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/da2.h"

namespace da2 {

constexpr int kTile = 8;
constexpr int kCap = 64;  // slots per block (8x8 tile)
constexpr int kWave = 64;

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

// ---- layout buffer views -------------------------------------------------
struct Layout {
  const int32_t* n_a;       // [R]
  const int32_t* slot2tok;  // [Npad]
  const int32_t* tok2slot;  // [N]
};
__host__ __device__ inline Layout layout_view(const int32_t* base, int R, int Npad) {
  return Layout{base, base + R, base + R + Npad};
}

// ---- input loads ------------------------------------------------------------
__device__ inline float load_elem(const void* base, int64_t idx, int dtype) {
  if (dtype == DA2_BF16) {
    uint16_t h = reinterpret_cast<const uint16_t*>(base)[idx];
    return __uint_as_float(static_cast<uint32_t>(h) << 16);
  }
  return reinterpret_cast<const float*>(base)[idx];
}

// 16-byte vector load of consecutive channels at p (16-byte aligned) as floats:
// 8 bf16 or 4 fp32 values.
__device__ inline void load_chunk(const uint16_t* p, float* x) {
  const uint4 v = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}
__device__ inline void load_chunk(const float* p, float* x) {
  const float4 v = *reinterpret_cast<const float4*>(p);
  x[0] = v.x;
  x[1] = v.y;
  x[2] = v.z;
  x[3] = v.w;
}
// All ones for a valid lane, else zero. The empty asm hides how the mask was
// made, so a load masked with it is not turned back into a branch around the
// load (which would serialize the loads that are meant to overlap).
__device__ inline uint32_t lane_mask(bool valid) {
  uint32_t m = valid ? 0xFFFFFFFFu : 0u;
  asm("" : "+v"(m));
  return m;
}
__device__ inline uint4 masked(const uint4& v, uint32_t m) { return make_uint4(v.x & m, v.y & m, v.z & m, v.w & m); }

// The same for a 16-byte chunk already in registers (T selects bf16 or fp32).
template <typename T>
__device__ inline void chunk_floats(const uint4& v, float* x) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __uint_as_float(w[i] << 16);
      x[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = __uint_as_float(w[i]);
  }
}

// Two channels (2p, 2p+1) of row s of a [rows][D] tile in LDS, as floats.
__device__ inline float2 tile_pair(const uint16_t* tile, int D, int s, int p) {
  const uint32_t w = reinterpret_cast<const uint32_t*>(tile + s * D)[p];
  return make_float2(__uint_as_float(w << 16), __uint_as_float(w & 0xFFFF0000u));
}
__device__ inline float2 tile_pair(const float* tile, int D, int s, int p) {
  return reinterpret_cast<const float2*>(tile + s * D)[p];
}
// Channel c of row s of a [rows][D] tile in LDS, as a float.
__device__ inline float tile_value(const uint16_t* tile, int D, int s, int c) {
  return __uint_as_float(static_cast<uint32_t>(tile[s * D + c]) << 16);
}
__device__ inline float tile_value(const float* tile, int D, int s, int c) { return tile[s * D + c]; }

// ---- INT8 ------------------------------------------------------------------
// INT8 code of y: round half away from zero, clamped to [-127, 127]. After the
// clamp, truncating y + copysign(0.5 - 2^-25, y) (one correctly rounded add)
// rounds half away from zero exactly for every float32 with |y| <= 130 (checked
// exhaustively against the definition); the clamp commutes with the rounding
// because its bounds are integers.
__device__ inline int int8_code(float y) {
  const float t = fminf(fmaxf(y, -127.0f), 127.0f);
  return static_cast<int>(t + __builtin_copysignf(0.49999997f, t));
}

// ---- E4M3 ------------------------------------------------------------------
// Value of a >= 0 after a round-to-nearest-even cast to E4M3 (saturating).
// Branch-free: both the subnormal (step 2^-9) and the normal rounding are
// evaluated and selected.
__device__ inline float e4m3_round_mag(float a) {
  const float sub = __builtin_rintf(a * 512.0f) * 0.001953125f;
  uint32_t b = __float_as_uint(a);
  b += 0x7FFFFu + ((b >> 20) & 1u);
  b &= 0xFFF00000u;
  const float nrm = __uint_as_float(b);
  return fminf(a < 0.015625f ? sub : nrm, 448.0f);
}

// Byte code of x after a round-to-nearest-even, saturating cast to E4M3.
__device__ inline uint32_t e4m3_code(float x) {
  uint32_t sign = (__float_as_uint(x) >> 24) & 0x80u;
  float a = fabsf(x);
  uint32_t mag;
  if (!(a < 448.0f)) {
    mag = 0x7Eu;
  } else if (a < 0.015625f) {
    mag = static_cast<uint32_t>(__builtin_rintf(a * 512.0f));  // 0..8 (8 = smallest normal)
  } else {
    uint32_t b = __float_as_uint(a);
    b += 0x7FFFFu + ((b >> 20) & 1u);
    mag = (((b >> 23) - 120u) << 3) | ((b >> 20) & 7u);
    mag = mag > 0x7Eu ? 0x7Eu : mag;
  }
  return sign | mag;
}

// ---- E2M1 ------------------------------------------------------------------
// Value of y after a round-to-nearest-even, saturating cast to E2M1 (sign kept).
__device__ inline float e2m1_round(float y) {
  float a = fabsf(y);
  float r;
  if (a < 1.0f) {
    r = __builtin_rintf(a * 2.0f) * 0.5f;  // 0, 0.5 or 1 (subnormal step 0.5)
  } else {
    uint32_t b = __float_as_uint(a);
    b += 0x1FFFFFu + ((b >> 22) & 1u);
    b &= 0xFFC00000u;
    r = fminf(__uint_as_float(b), 6.0f);
  }
  return __builtin_copysignf(r, y);
}

// ---- misc ------------------------------------------------------------------
__device__ inline float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ inline double wave_sum_f64(double v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Float bits of a non-negative float, usable with atomicMax on uint32.
__device__ inline void atomic_max_pos(uint32_t* p, float v) { atomicMax(p, __float_as_uint(v)); }

}  // namespace da2
