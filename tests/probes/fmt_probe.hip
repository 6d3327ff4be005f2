// Device-side format checks for the tests: the library's software encoders
// (common.hpp) and the gfx950 conversion instructions the attention kernel
// uses, evaluated element-wise on a caller-given array. One thread per
// element, bounds-checked; test infrastructure only.
#include "../../paper_2609_32628_amd/csrc/common.hpp"

typedef _Float16 h2 __attribute__((ext_vector_type(2)));

__global__ void fmt_probe_kernel(const float* x, int n, float* e2m1_sw, float* e2m1_hw, float* e2m1_hw_s2,
                                 float* e2m1_hw_back3, uint32_t* e4m3_sw, uint32_t* e4m3_hw, float* e4m3_mag_sw,
                                 float* e4m3_mag_hw, int32_t* int8_code) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const float v = x[i];
  e2m1_sw[i] = da2::e2m1_round(v);
  // hardware E2M1: value -> fp4 (scale 1) -> f16 (scale 1)
  uint32_t f4 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, v, 0.0f, 1.0f, 0);
  h2 back = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(f4, 1.0f, 0);
  e2m1_hw[i] = (float)back[0];
  // scale semantics: encode with scale 2, decode with scale 1
  uint32_t f4s = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, v, 0.0f, 2.0f, 0);
  h2 b2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(f4s, 1.0f, 0);
  e2m1_hw_s2[i] = (float)b2[0];
  // decode scale 3 (is the whole fp32 scale applied, or only its exponent?)
  h2 b3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(f4, 3.0f, 0);
  e2m1_hw_back3[i] = (float)b3[0];
  e4m3_sw[i] = da2::e4m3_code(v);
  e4m3_hw[i] = static_cast<uint32_t>(__builtin_amdgcn_cvt_pk_fp8_f32(v, 0.0f, 0, false)) & 0xFFu;
  e4m3_mag_sw[i] = da2::e4m3_round_mag(fabsf(v));
  // value round trip as the attention's weight scales use it (|v| clamped to 448)
  e4m3_mag_hw[i] = __builtin_amdgcn_cvt_f32_fp8(__builtin_amdgcn_cvt_pk_fp8_f32(fminf(fabsf(v), 448.0f), 0.0f, 0, false), 0);
  int8_code[i] = da2::int8_code(v);
}

extern "C" int da2_probe_formats(const float* x, int n, float* e2m1_sw, float* e2m1_hw, float* e2m1_hw_s2,
                                 float* e2m1_hw_back3, uint32_t* e4m3_sw, uint32_t* e4m3_hw, float* e4m3_mag_sw,
                                 float* e4m3_mag_hw, int32_t* int8_code, void* stream) {
  if (n <= 0 || !x) return -1;
  hipLaunchKernelGGL(fmt_probe_kernel, dim3((n + 255) / 256), dim3(256), 0, (hipStream_t)stream, x, n, e2m1_sw,
                     e2m1_hw, e2m1_hw_s2, e2m1_hw_back3, e4m3_sw, e4m3_hw, e4m3_mag_sw, e4m3_mag_hw, int8_code);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

// LDS DMA placement: global_load_lds_dwordx4 issued by a wave with LDS base B
// writes lane i's 16 bytes to B + 16 i. The 4 KB buffer keeps any other
// stride up to 64 bytes inside the allocation; out[] receives the whole buffer.
__global__ void lds_dma_probe_kernel(const uint32_t* src, uint32_t* out) {
  __shared__ uint32_t buf[1024];
  for (int i = threadIdx.x; i < 1024; i += 64) buf[i] = 0xFFFFFFFFu;
  __syncthreads();
  __builtin_amdgcn_global_load_lds((const void*)(src + 4 * threadIdx.x),
                                   (__attribute__((address_space(3))) void*)(buf + 64), 16, 0, 0);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  for (int i = threadIdx.x; i < 1024; i += 64) out[i] = buf[i];
}

extern "C" int da2_probe_lds_dma(const uint32_t* src, uint32_t* out, void* stream) {
  hipLaunchKernelGGL(lds_dma_probe_kernel, dim3(1), dim3(64), 0, (hipStream_t)stream, src, out);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

// Scaled fp4 matrix product: one wave computes D = A B with
// v_mfma_scale_f32_32x32x64_f8f6f4 on E2M1 operands (format 4) for each byte
// selector 0..3 of the per-lane E8M0 scale words. a, b: 64 lanes x 4 words of
// packed codes; sa, sb: one scale word per lane; out: [4][64][16] floats in
// accumulator order.
typedef int i32x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__global__ void mfma_fp4_probe_kernel(const uint32_t* a, const uint32_t* b, const uint32_t* sa, const uint32_t* sb,
                                      float* out) {
  const int l = threadIdx.x;
  const i32x8_t av = {(int)a[4 * l], (int)a[4 * l + 1], (int)a[4 * l + 2], (int)a[4 * l + 3], 0, 0, 0, 0};
  const i32x8_t bv = {(int)b[4 * l], (int)b[4 * l + 1], (int)b[4 * l + 2], (int)b[4 * l + 3], 0, 0, 0, 0};
  const int xa = (int)sa[l], xb = (int)sb[l];
  f32x16_t d[4];
  d[0] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv, f32x16_t{}, 4, 4, 0, xa, 0, xb);
  d[1] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv, f32x16_t{}, 4, 4, 1, xa, 1, xb);
  d[2] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv, f32x16_t{}, 4, 4, 2, xa, 2, xb);
  d[3] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv, f32x16_t{}, 4, 4, 3, xa, 3, xb);
  for (int s = 0; s < 4; ++s)
    for (int i = 0; i < 16; ++i) out[(s * 64 + l) * 16 + i] = d[s][i];
}

extern "C" int da2_probe_mfma_fp4(const uint32_t* a, const uint32_t* b, const uint32_t* sa, const uint32_t* sb,
                                  float* out, void* stream) {
  hipLaunchKernelGGL(mfma_fp4_probe_kernel, dim3(1), dim3(64), 0, (hipStream_t)stream, a, b, sa, sb, out);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}
