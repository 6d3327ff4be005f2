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
//
// Latency: each block's V fragments are requested before its QK^T product and
// the next block's K fragments right after it, so both loads are in flight
// while the softmax runs. The query fragments sit in LDS (read once per block)
// to leave registers for these prefetches.
//
// Weight conversions use the gfx950 instructions v_cvt_pk_fp8_f32 (E4M3) and
// v_cvt_scalef32_pk_fp4_f32 / v_cvt_scalef32_pk_f16_fp4 (E2M1 and back, unit
// scales); both round to nearest even, which the device format tests check
// against the format definitions.
#include "common.hpp"
#include "launch.hpp"

namespace da2 {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kExpOffset = 8.807f;

__device__ inline float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

typedef __attribute__((address_space(3))) void* lds_ptr;

// Asynchronous copy of one 1 KB operand fragment (16 bytes per lane, lane
// order) from global memory to LDS at the wave-uniform address dst. Issued as
// inline assembly so that the compiler does not add its conservative
// "wait for every LDS copy" before later LDS reads; the kernel waits for
// exactly the copies it needs (wait_vmem_keep) instead.
__device__ inline void dma_fragment(const void* src_lane, void* dst) {
  const uint32_t lds = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_ptr)dst)));
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src_lane), "s"(lds)
               : "memory", "m0");
}
__device__ inline void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
__device__ inline void wait_lds() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

template <int NT>
__device__ inline void rescale(f32x16 (&U)[NT], float alpha) {
#pragma unroll
  for (int t = 0; t < NT; ++t) U[t] *= alpha;
}

// Running-max update for one 32-query tile: bm_lane is this lane's maximum raw
// logit of the block (-inf on padding), scale converts raw logits to log2
// units. Updates m and l, returns the new maximum and (via alpha) the factor
// 2^(m_old - m_new) that the numerator still has to be multiplied by.
__device__ inline float new_max(float bm_lane, float scale, float& m, float& l, float& alpha) {
  const float bm = fmaxf(bm_lane, __shfl_xor(bm_lane, 32, 64));
  const float mn = fmaxf(m, bm * scale);
  alpha = exp2_fast(m - mn);
  m = mn;
  l *= alpha;
  return mn;
}

__device__ inline float max16(const f32x16& v) {
  float a = fmaxf(fmaxf(v[0], v[1]), v[2]), b = fmaxf(fmaxf(v[3], v[4]), v[5]);
  float c = fmaxf(fmaxf(v[6], v[7]), v[8]), d = fmaxf(fmaxf(v[9], v[10]), v[11]);
  float e = fmaxf(fmaxf(v[12], v[13]), v[14]);
  return fmaxf(fmaxf(fmaxf(a, b), fmaxf(c, d)), fmaxf(e, v[15]));
}

constexpr float kLog2_2688 = 11.392317422778760f;  // log2(6 * 448)

// NVFP4 weights of one 16-slot group held by this lane (slots of S[0..15]):
// sigma_P = E4M3(448 max Pt), w = sigma_P * E2M1(Pt * 2688 / sigma_P) as fp16
// pairs for the P^T operand; returns the fp32 sum of Pt. The scaled weights
// y = Pt * 2688 / sigma_P come from one exp2 each (the factor is folded into
// the exponent); a zero sigma_P uses factor 1, and those y (all below 2^-18)
// round to E2M1 zero as the format requires.
__device__ inline float nvfp4_weights(const f32x16& S, float c, float mn, float gmax, f16x8& lo, f16x8& hi) {
  const float pmax = exp2_fast(__builtin_fmaf(gmax, c, -mn));
  const float sigma = e4m3_round_mag(fminf(448.0f * pmax, 448.0f));
  const bool nz = sigma > 0.0f;
  const float off = (nz ? kLog2_2688 - __builtin_amdgcn_logf(sigma) : 0.0f) - mn;
  const _Float16 sh = (_Float16)sigma;
  const f16x2 s2 = {sh, sh};
  float y[16];
  float sum = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    y[i] = exp2_fast(__builtin_fmaf(S[i], c, off));
    sum += y[i];
  }
  // E2M1 codes, two per byte (byte selector must be a literal)
  uint32_t f0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, y[0], y[1], 1.0f, 0);
  f0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f0, y[2], y[3], 1.0f, 1);
  f0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f0, y[4], y[5], 1.0f, 2);
  f0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f0, y[6], y[7], 1.0f, 3);
  uint32_t f1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, y[8], y[9], 1.0f, 0);
  f1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f1, y[10], y[11], 1.0f, 1);
  f1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f1, y[12], y[13], 1.0f, 2);
  f1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(f1, y[14], y[15], 1.0f, 3);
  // back to fp16 and times sigma_P (exact: at most 6 significant bits)
  const f16x2 a0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(f0, 1.0f, 0) * s2;
  const f16x2 a1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(f0, 1.0f, 1) * s2;
  const f16x2 a2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(f0, 1.0f, 2) * s2;
  const f16x2 a3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(f0, 1.0f, 3) * s2;
  const f16x2 b0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(f1, 1.0f, 0) * s2;
  const f16x2 b1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(f1, 1.0f, 1) * s2;
  const f16x2 b2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(f1, 1.0f, 2) * s2;
  const f16x2 b3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(f1, 1.0f, 3) * s2;
  lo = f16x8{a0[0], a0[1], a1[0], a1[1], a2[0], a2[1], a3[0], a3[1]};
  hi = f16x8{b0[0], b0[1], b1[0], b1[1], b2[0], b2[1], b3[0], b3[1]};
  return sum * (nz ? sigma * (1.0f / 2688.0f) : 1.0f);
}

// Padded key slots (slot >= nb) of a partial block get -inf logits.
__device__ inline void mask_tail(f32x16 (&S)[2], int nb, int g) {
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (32 * j + 16 * g + i >= nb) S[j][i] = -INFINITY;
}

// Key-list window: lane i holds entry first+i of the row's list of key blocks
// (block id, valid slots, INT8 key scale), so each iteration reads its entry
// with one readlane instead of a chain of dependent global loads.
struct KeyWin {
  int kb, nb;
  float dk;
};
__device__ inline KeyWin key_window(const uint16_t* list, int first, int count, const int32_t* n_a,
                                    const float* dK, int lane) {
  KeyWin w{0, kCap, 0.0f};
  const int e = first + lane;
  if (e < count) {
    w.kb = list[e];
    w.nb = n_a[w.kb];
    w.dk = dK[w.kb];
  }
  // Consume the loaded registers here, so the wait for these loads happens in
  // the (rare) refill and not at every later use of the window.
  asm volatile("" : "+v"(w.kb), "+v"(w.nb), "+v"(w.dk));
  return w;
}
__device__ inline int lane_value(int v, int lane) { return __builtin_amdgcn_readlane(v, lane); }
__device__ inline float lane_value(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// Waits for this wave's older vector-memory operations, leaving the N most
// recent ones in flight (they complete in issue order).
template <int N>
__device__ inline void wait_vmem_keep() {
  if constexpr (N == 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  else if constexpr (N == 2) asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
  else if constexpr (N == 4) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
  else if constexpr (N == 8) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
  else static_assert(N == 0, "unsupported count");
}
// Workgroup barrier without the memory fences of __syncthreads (the waits
// above make LDS contents ready; the fences would also drain in-flight DMA).
__device__ inline void wg_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Softmax of this wave's 32-query tile on the NVFP4 path: running max, NVFP4
// weights, denominator; the numerator's rescale factor comes back in alpha.
__device__ inline void softmax_fp4(f32x16 (&S)[2], int nb, int g, float c4, float& m, float& l, float& alpha,
                                   f16x8 (&Pf)[4]) {
  if (nb < kCap) mask_tail(S, nb, g);
  const float gm0 = max16(S[0]), gm1 = max16(S[1]);
  const float mn = new_max(fmaxf(gm0, gm1), c4, m, l, alpha);
  const float s0 = nvfp4_weights(S[0], c4, mn, gm0, Pf[0], Pf[1]);
  const float s1 = nvfp4_weights(S[1], c4, mn, gm1, Pf[2], Pf[3]);
  l += s0 + s1;
}

// Softmax of this wave's 32-query tile on the INT8 path: amplified weights
// 2^((s - m) log2 e + 8.807) in E4M3 for the fp8 P^T operand.
__device__ inline void softmax_fp8(const i32x16 (&Si)[2], int nb, int g, float cb, float& m, float& l, float& alpha,
                                   i32x8& Pf) {
  f32x16 sf[2];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) sf[j][i] = (float)Si[j][i];
  if (nb < kCap) mask_tail(sf, nb, g);
  const float mn = new_max(fmaxf(max16(sf[0]), max16(sf[1])), cb, m, l, alpha);
  const float off = kExpOffset - mn;
  float lsum = 0.0f;
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      float p[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        p[e] = exp2_fast(__builtin_fmaf(sf[j][4 * w + e], cb, off));
        lsum += p[e];
      }
      const int v = __builtin_amdgcn_cvt_pk_fp8_f32(p[0], p[1], 0, false);
      Pf[4 * j + w] = __builtin_amdgcn_cvt_pk_fp8_f32(p[2], p[3], v, true);
    }
  l += lsum;
}

// One precision phase of the block loop. The workgroup's two waves own the
// query tiles qt = 0, 1 of the block; the key and value tiles of each key
// block are copied into LDS once (each wave issues half of the fragments) and
// read by both waves. Per block i:
//   wait K(i) -> barrier -> S = K Q^T -> barrier -> DMA K(i+1)
//   softmax (overlaps the K(i+1) and V(i) copies)
//   wait V(i) -> barrier -> U += V^T P^T -> barrier -> DMA V(i+1)
// Frag: fragment type; NFK/NFV: fragments per K/V tile.
// Orders a wait after the computation of v (an empty use of the register).
template <typename T>
__device__ inline void after(const T& v) {
  asm volatile("" ::"v"(v));
}

template <int NFK, int NFV, typename Frag, typename QK, typename SM, typename PV>
__device__ inline void phase_loop(const uint16_t* list, int n, const int32_t* n_a, const float* dKh,
                                  const Frag* Kh, const Frag* Vh, Frag* sK, Frag* sV, int wave, int lane,
                                  QK qk, SM softmax, PV pv) {
  constexpr int TILE = NFK * 64;  // fragments per block, in Frag units (K and V have the same size)
  static_assert(NFK == NFV, "K and V tiles hold the same number of fragments");
  constexpr int HALF = NFK / 2;
  auto dma_tile = [&](const Frag* src, Frag* dst) {
#pragma unroll
    for (int f = wave * HALF; f < (wave + 1) * HALF; ++f) dma_fragment(src + f * 64 + lane, dst + f * 64);
  };
  KeyWin win = key_window(list, 0, n, n_a, dKh, lane);
  dma_tile(Kh + (int64_t)lane_value(win.kb, 0) * TILE, sK);
  dma_tile(Vh + (int64_t)lane_value(win.kb, 0) * TILE, sV);
  for (int it = 0; it < n; ++it) {
    const int sl = it & 63;
    if (sl == 0 && it > 0) win = key_window(list, it, n, n_a, dKh, lane);
    const int kb = lane_value(win.kb, sl);
    const int nb = lane_value(win.nb, sl);
    const float dk = lane_value(win.dk, sl);
    const bool more = it + 1 < n;
    const int kb_next = !more ? 0 : (sl < 63 ? lane_value(win.kb, sl + 1) : (int)list[it + 1]);
    wait_vmem_keep<HALF>();  // K(i) copied (V(i), issued later, may still be in flight)
    wg_barrier();
    qk(nb, dk);
    wait_lds();
    wg_barrier();  // both waves are done with sK
    if (more) dma_tile(Kh + (int64_t)kb_next * TILE, sK);
    softmax(nb, dk);  // returns after its results exist, so the wait below cannot move above it
    if (more)
      wait_vmem_keep<HALF>();  // V(i) copied, K(i+1) may still be in flight
    else
      wait_vmem_keep<0>();
    wg_barrier();
    pv();
    wait_lds();
    wg_barrier();  // both waves are done with sV
    if (more) dma_tile(Vh + (int64_t)kb_next * TILE, sV);
    (void)kb;
  }
}

template <int D>
__global__ __launch_bounds__(128) void mixed_attn_kernel(AttnArgs args) {
  constexpr int NS16 = D / 16, NS32 = D / 32, NT = D / 32;
  __shared__ f16x8 sK[2 * NS16 * 64];  // key tile of the current block (16 KB at d=128)
  __shared__ f16x8 sV[NT * 4 * 64];    // value tile of the current block
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, r = lane & 31, g = lane >> 5;
  const int qt = wave;  // this wave's 32-query tile
  const int R = args.R;
  // XCD-aware mapping: workgroup b runs on XCD b mod 8 and takes the next row
  // of that XCD's contiguous segment of the work order.
  const int n_items = args.B * args.H * R;
  const int seg = (n_items + 7) >> 3;
  const int idx = (int)(blockIdx.x & 7) * seg + (int)(blockIdx.x >> 3);
  if (idx >= n_items) return;
  const int item = args.order[idx];
  const int bh = item / R, a = item % R;
  const Layout L = layout_view(args.layout, R, args.Npad);
  const int n4 = args.counts[2 * item], n8 = args.counts[2 * item + 1];
  const uint16_t* keys = args.keys + (int64_t)item * R;
  const int64_t blk0 = (int64_t)bh * R;  // first block of this head
  const float* dKh = args.dK + blk0;
  const float rsqd = 1.0f / sqrtf((float)D);

  f32x16 U[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) U[t] = f32x16{};
  float m = -INFINITY, l = 0.0f;
  const float gV = args.g[bh * 4 + 2];

  // ------------------------------ NVFP4 phase ------------------------------
  if (n4 > 0) {
    const float c4 = args.g[bh * 4 + 0] * args.g[bh * 4 + 1] * kLog2e * rsqd;
    f16x8 Qf[NS16];
    const f16x8* Qa = reinterpret_cast<const f16x8*>(args.Q4) + (blk0 + a) * (kCap * D / 8);
#pragma unroll
    for (int s = 0; s < NS16; ++s) Qf[s] = Qa[(qt * NS16 + s) * 64 + lane];
    f32x16 S[2];
    f16x8 P[4];
    float alpha = 1.0f;
    auto qk = [&](int, float) {
      S[0] = S[1] = f32x16{};
#pragma unroll
      for (int s = 0; s < NS16; ++s)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          S[j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(sK[(j * NS16 + s) * 64 + lane], Qf[s], S[j], 0, 0, 0);
    };
    auto sm = [&](int nb, float) {
      softmax_fp4(S, nb, g, c4, m, l, alpha, P);
      after(P[0]), after(P[1]), after(P[2]), after(P[3]), after(l);
    };
    auto pv = [&]() {
      if (__ballot(alpha != 1.0f)) rescale<NT>(U, alpha);
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int t = 0; t < NT; ++t)
          U[t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(sV[(t * 4 + s) * 64 + lane], P[s], U[t], 0, 0, 0);
    };
    phase_loop<2 * NS16, NT * 4>(keys, n4, L.n_a, dKh, reinterpret_cast<const f16x8*>(args.K4) + blk0 * (kCap * D / 8),
                                 reinterpret_cast<const f16x8*>(args.V4) + blk0 * (kCap * D / 8), sK, sV, wave, lane,
                                 qk, sm, pv);
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
        U[t][i] *= dc == 0.0f ? 0.0f : restore / (eta * dc);
      }
    l /= eta;
    i32x4 Qf[NS32];
    const i32x4* Qa = reinterpret_cast<const i32x4*>(args.Q8) + (blk0 + a) * (kCap * D / 16);
#pragma unroll
    for (int s = 0; s < NS32; ++s) Qf[s] = Qa[(qt * NS32 + s) * 64 + lane];
    const float c8a = args.dQ[blk0 + a] * kLog2e * rsqd;
    i32x4* sK8 = reinterpret_cast<i32x4*>(sK);
    i32x4* sV8 = reinterpret_cast<i32x4*>(sV);
    i32x16 S[2];
    i32x8 P;
    float alpha = 1.0f;
    auto qk = [&](int, float) {
      S[0] = S[1] = i32x16{};
#pragma unroll
      for (int s = 0; s < NS32; ++s)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          S[j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(sK8[(j * NS32 + s) * 64 + lane], Qf[s], S[j], 0, 0, 0);
    };
    auto sm = [&](int nb, float dk) {
      softmax_fp8(S, nb, g, c8a * dk, m, l, alpha, P);
      after(P), after(l);
    };
    auto pv = [&]() {
      if (__ballot(alpha != 1.0f)) rescale<NT>(U, alpha);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const i32x4 v0 = sV8[(t * 2 + 0) * 64 + lane], v1 = sV8[(t * 2 + 1) * 64 + lane];
        const i32x8 vf = i32x8{v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
        U[t] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(vf, P, U[t], 0, 0, 0, 127, 0, 127);
      }
    };
    wait_lds();
    wg_barrier();  // the NVFP4 phase is done with sK / sV
    phase_loop<2 * NS32, NT * 2>(keys + n4, n8, L.n_a, dKh,
                                 reinterpret_cast<const i32x4*>(args.K8) + blk0 * (kCap * D / 16),
                                 reinterpret_cast<const i32x4*>(args.V8) + blk0 * (kCap * D / 16), sK8, sV8, wave,
                                 lane, qk, sm, pv);
    // Exit: U_c <- eta delta_c U_c, l <- eta l
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 16; ++i) U[t][i] *= eta * dV[chan(t, i)];
    l *= eta;
  } else if (n4 > 0) {
    const float restore = gV / 2688.0f;
#pragma unroll
    for (int t = 0; t < NT; ++t) U[t] *= restore;
  }

  // ------------------------- normalize and scatter -------------------------
  const int nq = L.n_a[a];
  const int32_t* s2t = L.slot2tok + (int64_t)a * kCap;
  const int b = bh / args.H, h = bh % args.H;
  const float lt = l + __shfl_xor(l, 32, 64);
  const float inv = lt > 0.0f ? 1.0f / lt : 0.0f;
  const int q = 32 * qt + r;
  if (q < nq) {
    const int64_t row = (int64_t)b * args.ob + (int64_t)h * args.oh + (int64_t)s2t[q] * args.on;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float v = U[t][i] * inv;
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

template __global__ void mixed_attn_kernel<64>(AttnArgs);
template __global__ void mixed_attn_kernel<128>(AttnArgs);

hipError_t launch_attn(const AttnArgs& args, hipStream_t stream) {
  const int items = args.B * args.H * args.R;
  const int grid = 8 * ((items + 7) / 8);
  if (args.d == 128)
    hipLaunchKernelGGL(mixed_attn_kernel<128>, dim3(grid), dim3(128), 0, stream, args);
  else
    hipLaunchKernelGGL(mixed_attn_kernel<64>, dim3(grid), dim3(128), 0, stream, args);
  return hipGetLastError();
}

}  // namespace da2
