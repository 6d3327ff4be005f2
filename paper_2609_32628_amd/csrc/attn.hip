// Phased mixed-precision attention (phased-execution appendix; precision-state-
// conversion equation; NVFP4 probability equation; INT8 and FP16 paragraph).
//
// One workgroup of two waves owns one query block a (64 query slots); wave w
// owns the 32-query tile qt = w. The workgroup walks the block's retained key
// blocks: the 4-bit ones in ascending order (NVFP4, or MXFP4 when the
// operands were prepared in that encoding), then the INT8 ones, then the
// 16-bit ones. All blocks share the fp32 running maxima m, the denominators l
// and the numerator U.
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
// Units: the NVFP4 phase multiplies fp16 sigma*e operands, so U carries a
// factor 2688/g_V and l the unamplified weights (the MXFP4 alternative of the
// 4-bit phase runs scaled fp4 MFMAs and stays in the common units); Enter
// converts to the 8-bit path's units U_c / (eta delta_c), l / eta; the 8-bit
// phase accumulates amplified
// weights 2^(z - m + 8.807) and E4M3 codes; Exit converts back; the 16-bit
// phase then accumulates fp16 weights times fp16 values in the common units.
//
// Data movement: the K and V tiles of a key block are copied into LDS once per
// workgroup (each wave copies half) and read by both waves; the loop is
// software-pipelined by one block (see phase_loop), and the query fragments
// of the wave's tile stay in registers for the whole phase.
//
// Weight conversions use the gfx950 instructions v_cvt_pk_fp8_f32 (E4M3) and
// v_cvt_scalef32_pk_fp4_f32 / v_cvt_scalef32_pk_f16_fp4 (E2M1 and back, unit
// scales); both round to nearest even, which the device format tests check
// against the format definitions.
#include <utility>

#include "common.hpp"
#include "launch.hpp"

namespace da2 {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kExpOffset = 8.807f;

__device__ inline float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

typedef __attribute__((address_space(3))) void* lds_ptr;

// Asynchronous copy of one 1 KB operand fragment (16 bytes per lane, lane
// order) from global memory to LDS. The source is tile + voff + OFS with the
// wave-uniform tile address in scalar registers and voff = 16 * lane, so the
// address needs no vector arithmetic; the destination is lds + OFS (the
// instruction adds its immediate offset to the LDS address in M0 as well).
// Issued as inline assembly so that the compiler does not add its conservative
// "wait for every LDS copy" before later LDS reads; the kernel waits for
// exactly the copies it needs (wait_vmem_keep) instead.
template <int OFS>
__device__ inline void dma_fragment(const void* tile, uint32_t voff, uint32_t lds) {
  static_assert(OFS >= 0 && OFS < 4096, "immediate offset out of range");
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 offset:%3" ::"v"(voff), "s"(tile),
               "s"(lds), "n"(OFS)
               : "memory", "m0");
}
__device__ inline uint32_t lds_address(void* p) {
  return __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_ptr)p)));
}
__device__ inline void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
__device__ inline void wait_lds() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

template <int NT>
__device__ inline void rescale(f32x16 (&U)[NT], float alpha) {
#pragma unroll
  for (int t = 0; t < NT; ++t) U[t] *= alpha;
}

// Maximum of v over lanes l and l ^ 32: one v_permlane32_swap hands each lane
// both halves' values (no LDS permute, so no wait on the tile reads in flight).
__device__ inline float max_halves(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Running-max update for one 32-query tile: bm_lane is this lane's maximum raw
// logit of the block (-inf on padding), scale converts raw logits to log2
// units. Updates m and l, returns the new maximum and (via alpha) the factor
// 2^(m_old - m_new) that the numerator still has to be multiplied by.
__device__ inline float new_max(float bm_lane, float scale, float& m, float& l, float& alpha) {
  const float bm = max_halves(bm_lane);
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

// NVFP4 weights of one 16-slot group held by this lane (slots of S[0..15]),
// computed in stages so that they can be interleaved with matrix work:
//   setup: sigma_P = E4M3(448 max Pt) from the group's maximum logit;
//   exps:  y = Pt * 2688 / sigma_P from one exp2 each (the factor is folded
//          into the exponent), their fp32 sum, and E2M1(y) as 4-bit codes,
//          converted in pairs as they are computed;
//   pack:  w = sigma_P * E2M1(y) as fp16 pairs for the P^T operand (exact:
//          at most 6 significant bits).
// A zero sigma_P uses factor 1, and those y (all below 2^-18) round to E2M1
// zero as the format requires. weight_sum() is the fp32 sum of Pt.
struct Fp4Group {
  float off, scale, sum;
  f16x2 s2;
  uint32_t code[2];  // E2M1 codes of slots [0,8) and [8,16), two per byte (written by fp4_exp_pair)
};
// E4M3 value of a in [0, 448]: v_cvt_pk_fp8_f32 rounds to nearest even (the
// device format tests check it against the format definition on that range)
// and v_cvt_f32_fp8 returns the exact value.
__device__ inline float e4m3_round_hw(float a) {
  // only byte 0 is read back, so the kept bytes may be anything: a's bits
  return __builtin_amdgcn_cvt_f32_fp8(__builtin_amdgcn_cvt_pk_fp8_f32(a, 0.0f, __float_as_int(a), false), 0);
}
__device__ inline void fp4_setup(Fp4Group& G, float gmax, float c, float mn) {
  const float pmax = exp2_fast(__builtin_fmaf(gmax, c, -mn));
  const float sigma = e4m3_round_hw(fminf(448.0f * pmax, 448.0f));
  const bool nz = sigma > 0.0f;
  G.off = (nz ? kLog2_2688 - __builtin_amdgcn_logf(sigma) : 0.0f) - mn;
  G.scale = nz ? sigma * (1.0f / 2688.0f) : 1.0f;
  const _Float16 sh = (_Float16)sigma;
  G.s2 = f16x2{sh, sh};
  G.sum = 0.0f;
}
// Weights of slots [I0, I1) (I0, I1 even): y = 2^(S c + off) from one exp2
// each, added to the fp32 sum and converted to E2M1 in pairs right away.
template <int I>
__device__ inline void fp4_exp_pair(Fp4Group& G, const f32x16& S, float c) {
  const float y0 = exp2_fast(__builtin_fmaf(S[I], c, G.off));
  const float y1 = exp2_fast(__builtin_fmaf(S[I + 1], c, G.off));
  G.sum += y0;
  G.sum += y1;
  // pairs are converted in ascending order, so byte 0 is the first byte
  // written in each code word: its conversion may keep anything in the other
  // bytes (the bits of an input that dies here; no register is cleared)
  const uint32_t kept = ((I >> 1) & 3) == 0 ? __float_as_uint(y1) : G.code[I >> 3];
  G.code[I >> 3] = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(kept, y0, y1, 1.0f, (I >> 1) & 3);
}
template <int I0, int I1>
__device__ inline void fp4_exps(Fp4Group& G, const f32x16& S, float c) {
  static_assert(I0 % 2 == 0 && I1 % 2 == 0, "whole pairs");
  [&]<int... P>(std::integer_sequence<int, P...>) {
    (fp4_exp_pair<I0 + 2 * P>(G, S, c), ...);
  }(std::make_integer_sequence<int, (I1 - I0) / 2>{});
}
// sigma_P * E2M1 codes as fp16 pairs for the P^T operand (exact: at most 6
// significant bits).
__device__ inline void fp4_pack(const Fp4Group& G, f16x8& lo, f16x8& hi) {
  const uint32_t f0 = G.code[0], f1 = G.code[1];
  const f16x2 s2 = G.s2;
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
}
__device__ inline float weight_sum(const Fp4Group& G) { return G.sum * G.scale; }

// INT8-path weights of 8 logits S[I0..I0+8) of this lane: amplified weights
// 2^((s - m) log2 e + 8.807) in E4M3 (two dwords of the fp8 P^T operand);
// returns their fp32 sum.
template <int I0>
__device__ inline float fp8_weights8(const f32x16& S, float cb, float off, int& w0, int& w1) {
  float p[8];
  float sum = 0.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    p[e] = exp2_fast(__builtin_fmaf(S[I0 + e], cb, off));
    sum += p[e];
  }
  // the high half of each word's first conversion is overwritten by the
  // second, so its kept half may be anything: the bits of an input that dies
  // here, which needs no register cleared for it
  w0 = __builtin_amdgcn_cvt_pk_fp8_f32(p[2], p[3], __builtin_amdgcn_cvt_pk_fp8_f32(p[0], p[1], __float_as_int(p[1]), false), true);
  w1 = __builtin_amdgcn_cvt_pk_fp8_f32(p[6], p[7], __builtin_amdgcn_cvt_pk_fp8_f32(p[4], p[5], __float_as_int(p[5]), false), true);
  return sum;
}

// 16-bit path weights of 8 logits S[I0..I0+8) of this lane: Pt = 2^(S c - mn)
// in fp32 (added to sum) and rounded to nearest-even fp16 for the P^T operand.
template <int I0>
__device__ inline f16x8 half_weights8(const f32x16& S, float c, float mn, float& sum) {
  f16x8 h;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float y = exp2_fast(__builtin_fmaf(S[I0 + e], c, -mn));
    sum += y;
    h[e] = (_Float16)y;
  }
  return h;
}

// MXFP4 path: D += A B on one 32x32x64 scaled fp4 MFMA. a, b: 32 E2M1 codes
// per lane (k = 32 (lane/32) + i in nibble i); sa, sb: the lanes' E8M0 scale
// words (byte 0 applies to the lane's 32 codes).
__device__ inline f32x16 mfma_fp4(const i32x4& a, const i32x4& b, const f32x16& c, int sa, int sb) {
  const i32x8 a8 = {a[0], a[1], a[2], a[3], 0, 0, 0, 0};
  const i32x8 b8 = {b[0], b[1], b[2], b[3], 0, 0, 0, 0};
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, c, 4, 4, 0, sa, 0, sb);
}

// E8M0 exponent of this lane's 32-slot weight block: floor(log2 max Pt) - 2,
// clamped below at -127, where max Pt = 2^(gm c - mn) comes from the block's
// largest logit gm with the same product as the running maximum, so the block
// that holds the row maximum gets max Pt = 1 exactly.
__device__ inline int mx_weight_exponent(float gm, float c, float mn) {
  const float pmax = exp2_fast(gm * c - mn);
  return max((int)(__float_as_uint(pmax) >> 23) - 129, -127);
}

// MXFP4 weights of 8 logits S[I0..I0+8): y = Pt 2^-k = 2^(S c + off) with
// off = -mn - k (added to sum), as E2M1 codes in one dword (value e in nibble e).
template <int I0>
__device__ inline int mx_codes8(const f32x16& S, float c, float off, float& sum) {
  float y[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    y[e] = exp2_fast(__builtin_fmaf(S[I0 + e], c, off));
    sum += y[e];
  }
  // bytes 1-3 are written below, so byte 0's conversion may keep anything
  // there: the bits of an input that dies here
  uint32_t w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(__float_as_uint(y[1]), y[0], y[1], 1.0f, 0);
  w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, y[2], y[3], 1.0f, 1);
  w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, y[4], y[5], 1.0f, 2);
  w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, y[6], y[7], 1.0f, 3);
  return static_cast<int>(w);
}

// Scheduling fence: no instruction moves across it, so the stages between two
// fences keep the interleaving of matrix and vector work written in the source.
__device__ inline void fence() { __builtin_amdgcn_sched_barrier(0); }

// Padded key slots (slot >= nb) of a partial block get -inf logits.
// Register i of logit tile j holds slot 32j + 16g + i.
__device__ inline void mask_tail(f32x16 (&S)[2], int nb, int g) {
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int valid = nb - 32 * j - 16 * g;  // valid registers of this lane
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (i >= valid) S[j][i] = -INFINITY;
  }
}

// The same for the MXFP4 key order: register i of tile j holds slot 32g + 16j + i.
__device__ inline void mask_tail_mx(f32x16 (&S)[2], int nb, int g) {
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int valid = nb - 32 * g - 16 * j;
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (i >= valid) S[j][i] = -INFINITY;
  }
}

// Key-list window: lane i holds entry first+i of the row's list of key blocks
// (block id, valid slots, INT8 key scale) and the block id of entry
// first+64+i, so each iteration reads the entries it needs (its own and the
// next two, for the copies) with readlane instead of global loads. A global
// load inside the loop would make the compiler wait for every outstanding
// vector-memory operation, including the tile copies still in flight.
struct KeyWin {
  int kb, nb;
  float dk;
  int kb_next;
};
__device__ inline KeyWin key_window(const uint16_t* list, int first, int count, const int32_t* n_a,
                                    const float* dK, int lane) {
  KeyWin w{0, kCap, 0.0f, 0};
  const int e = first + lane;
  if (e < count) {
    w.kb = list[e];
    w.nb = n_a[w.kb];
    w.dk = dK[w.kb];
  }
  if (e + 64 < count) w.kb_next = list[e + 64];
  // Consume the loaded registers here, so the wait for these loads happens in
  // the (rare) refill and not at every later use of the window.
  asm volatile("" : "+v"(w.kb), "+v"(w.nb), "+v"(w.dk), "+v"(w.kb_next));
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
  else if constexpr (N == 1) asm volatile("s_waitcnt vmcnt(1)" ::: "memory");
  else if constexpr (N == 2) asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
  else if constexpr (N == 3) asm volatile("s_waitcnt vmcnt(3)" ::: "memory");
  else if constexpr (N == 4) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
  else if constexpr (N == 8) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
  else static_assert(N == 0, "unsupported count");
}
// Waits until only the fragments of the most recent tile copy that this wave
// issued are in flight: NFK/2 each for even NFK; for odd NFK wave 0 copies
// (NFK+1)/2 fragments and wave 1 the rest.
template <int NFK>
__device__ inline void wait_keep_tile(int wave) {
  if constexpr (NFK % 2 == 0) {
    wait_vmem_keep<NFK / 2>();
  } else {
    if (wave == 0)
      wait_vmem_keep<(NFK + 1) / 2>();
    else
      wait_vmem_keep<NFK / 2>();
  }
}

// Workgroup barrier without the memory fences of __syncthreads (the waits
// above make LDS contents ready; the fences would also drain in-flight DMA).
__device__ inline void wg_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Orders a wait after the computation of v (an empty use of the register).
template <typename T>
__device__ inline void after(const T& v) {
  asm volatile("" ::"v"(v));
}

// ---- packed NVFP4 operands ---------------------------------------------------
// Each block of a packed NVFP4 section holds 32 D bytes of E2M1 codes and 4 D
// bytes of E4M3 group scales, ordered so that thread (wave w, lane l) of the
// workgroup finds its share contiguous: D/16 code dwords at dword (w 64 + l) D/16
// (dword i holds the 8 codes of one fp16 fragment, code e in nibble e), and
// its scale bytes at 32 D + (w 32 + l%32) D/16 (Q, K: byte s scales fragment
// s) or 32 D + (w 64 + l) D/32 (V: byte 2 t2 + h scales fragments (t2, 2h) and
// (t2, 2h + 1)).
template <int D>
struct NvShare {
  uint4 c[D / 64];  // D/16 code dwords
  uint32_t s[(D / 16 + 3) / 4];  // scale bytes
};

template <int D>
__device__ inline void nv_load_qk(NvShare<D>& x, const uint8_t* blk, int w, int lane) {
  const uint4* c = reinterpret_cast<const uint4*>(blk + (w * 64 + lane) * (D / 4));
#pragma unroll
  for (int i = 0; i < D / 64; ++i) x.c[i] = c[i];
  const uint8_t* sc = blk + 32 * D + (w * 32 + (lane & 31)) * (D / 16);
  if constexpr (D == 128) {
    const uint2 v = *reinterpret_cast<const uint2*>(sc);
    x.s[0] = v.x;
    x.s[1] = v.y;
  } else {
    x.s[0] = *reinterpret_cast<const uint32_t*>(sc);
  }
}
template <int D>
__device__ inline void nv_load_v(NvShare<D>& x, const uint8_t* blk, int w, int lane) {
  const uint4* c = reinterpret_cast<const uint4*>(blk + (w * 64 + lane) * (D / 4));
#pragma unroll
  for (int i = 0; i < D / 64; ++i) x.c[i] = c[i];
  const uint8_t* sc = blk + 32 * D + (w * 64 + lane) * (D / 32);
  if constexpr (D == 128)
    x.s[0] = *reinterpret_cast<const uint32_t*>(sc);
  else
    x.s[0] = *reinterpret_cast<const uint16_t*>(sc);
}
// fp16 fragment sigma * e of 8 codes (exact: at most 6 significant bits).
__device__ inline f16x8 nv_frag(uint32_t codes, f16x2 s2) {
  const f16x2 a0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(codes, 1.0f, 0) * s2;
  const f16x2 a1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(codes, 1.0f, 1) * s2;
  const f16x2 a2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(codes, 1.0f, 2) * s2;
  const f16x2 a3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(codes, 1.0f, 3) * s2;
  return f16x8{a0[0], a0[1], a1[0], a1[1], a2[0], a2[1], a3[0], a3[1]};
}
// Exact fp16 values of scale bytes 2p and 2p + 1 of a share (E4M3 -> fp16 is exact).
template <int D>
__device__ inline f16x2 nv_scale_pair(const NvShare<D>& x, int p) {
  return __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(x.s[p >> 1] >> (16 * (p & 1)), 1.0f, false);
}
// Fragment f of a Q or K share (f = s): codes dword f, scale byte f.
template <int D>
__device__ inline f16x8 nv_frag_qk(const NvShare<D>& x, int f) {
  const f16x2 pr = nv_scale_pair(x, f >> 1);
  const _Float16 sg = (f & 1) ? pr[1] : pr[0];
  return nv_frag(x.c[f >> 2][f & 3], f16x2{sg, sg});
}
// Fragment f = 4 t2 + s of a V share: codes dword f, scale byte 2 t2 + s/2.
template <int D>
__device__ inline f16x8 nv_frag_v(const NvShare<D>& x, int f) {
  const f16x2 pr = nv_scale_pair(x, f >> 2);
  const _Float16 sg = ((f >> 1) & 1) ? pr[1] : pr[0];
  return nv_frag(x.c[f >> 2][f & 3], f16x2{sg, sg});
}

// The NVFP4 phase's block loop. The key and value tiles of a block are decoded
// from their packed sections into fp16 tiles in LDS by the two waves together
// (each thread its own share), and read by both. Iteration i:
//   region 1: S' = K(i+1) Q^T with the softmax of block i, and V(i) decoded
//             into sV; then the packed V(i+1) is loaded
//   -> barrier -> value product of block i with K(i+2) decoded into sK; then
//   the packed K(i+3) is loaded -> barrier
// Two barriers per block; each packed load has one iteration to arrive.
// region1<MASK>(Sc, Sn, nb, vdec) calls vdec(f) once for each V fragment f;
// pv(Sc, kdec) calls kdec(f) once for each K fragment f.
template <int D, typename SA, typename FIRST, typename STEP1, typename PV>
__device__ inline void nv_phase_loop(const uint16_t* list, int n, const int32_t* n_a, const float* dKh,
                                     const uint8_t* Kh, const uint8_t* Vh, f16x8* sK, f16x8* sV, int wave, int lane,
                                     FIRST first_qk, STEP1 region1, PV pv) {
  constexpr int NB = nv_block_bytes(D);
  constexpr int NS16 = D / 16;
  NvShare<D> kx, vx;
  KeyWin win = key_window(list, 0, n, n_a, dKh, lane);
  auto block_at = [&](int e, int first) -> int {  // e - first < 128
    return e - first < 64 ? lane_value(win.kb, e - first) : lane_value(win.kb_next, e - first - 64);
  };
  auto kdec = [&](int f) { sK[(wave * NS16 + f) * 64 + lane] = nv_frag_qk<D>(kx, f); };
  auto vdec = [&](int f) { sV[(wave * NS16 + f) * 64 + lane] = nv_frag_v<D>(vx, f); };
  // prologue: K(0) decoded and its logits computed, K(1) decoded, V(0) and K(2) loaded
  const int kb0 = lane_value(win.kb, 0);
  nv_load_qk<D>(kx, Kh + (int64_t)kb0 * NB, wave, lane);
  nv_load_v<D>(vx, Vh + (int64_t)kb0 * NB, wave, lane);
#pragma unroll
  for (int f = 0; f < NS16; ++f) kdec(f);
  wait_lds();
  wg_barrier();
  SA Sa, Sb;
  first_qk(Sa);
  // The packed loads here and in the loop are issued on every path (past the
  // end of the list they fetch block 0, which is never decoded into a tile
  // that is read): where paths with different numbers of loads in flight
  // join, the compiler waits for all of them, including the share that the
  // next region does not need yet.
  nv_load_qk<D>(kx, Kh + (int64_t)(n > 1 ? block_at(1, 0) : 0) * NB, wave, lane);
  wait_lds();
  wg_barrier();  // both waves have read K(0)
  if (n > 1) {
#pragma unroll
    for (int f = 0; f < NS16; ++f) kdec(f);
  }
  nv_load_qk<D>(kx, Kh + (int64_t)(n > 2 ? block_at(2, 0) : 0) * NB, wave, lane);
  wait_lds();
  wg_barrier();  // K(1) is in sK

  auto step = [&](int it, SA& Sc, SA& Sn) {
    const int first = it & ~63;
    const int sl = it - first;
    if (sl == 0 && it > 0) win = key_window(list, it, n, n_a, dKh, lane);
    const int nb = lane_value(win.nb, sl);
    const bool more1 = it + 1 < n, more3 = it + 3 < n;
    const int kb1 = more1 ? block_at(it + 1, first) : 0;
    const int kb3 = more3 ? block_at(it + 3, first) : 0;
    // On the last block the logits of region 1 come from the unchanged tile and are not used.
    if (nb < kCap)
      region1.template operator()<true>(Sc, Sn, nb, vdec);
    else
      region1.template operator()<false>(Sc, Sn, nb, vdec);
    nv_load_v<D>(vx, Vh + (int64_t)kb1 * NB, wave, lane);
    wait_lds();
    wg_barrier();  // sV holds V(it); both waves are done with sK
    // K(it+2) is decoded unconditionally: past the end of the list the share
    // holds the previous block and the tile it writes is never read (one
    // instantiation of pv keeps the register allocation of the loop small)
    pv(Sc, kdec);
    nv_load_qk<D>(kx, Kh + (int64_t)kb3 * NB, wave, lane);
    wait_lds();
    wg_barrier();  // sK holds K(it+2); both waves are done with sV
  };
  for (int it = 0; it < n; it += 2) {
    step(it, Sa, Sb);
    if (it + 1 < n) step(it + 1, Sb, Sa);
  }
}

// One precision phase of the block loop, software-pipelined by one block: the
// logits of block i+1 are computed while the softmax of block i runs, so the
// matrix cores and the vector ALUs work side by side inside each wave. The
// workgroup's two waves own the query tiles qt = 0, 1 of the query block; the
// key and value tiles of each key block are copied into LDS once (each wave
// issues half of the fragments) and read by both waves. Iteration i:
//   wait K(i+1) -> barrier -> S' = K(i+1) Q^T interleaved with the first part
//   of the softmax of S -> barrier -> DMA K(i+2) -> rest of the softmax
//   -> wait V(i) -> barrier -> U += V(i)^T P^T -> barrier -> DMA V(i+1)
// Frag: fragment type; NFK: fragments per K (and V) tile; SA: logit tile type.
// first(S): logits of the first block. region1<MASK>(S, S', nb, dk): the
// logit MFMAs of block i+1 interleaved with the first part of the softmax of
// block i (MASK: block i is partial); region2(S): the rest of the softmax, after
// sK has been handed to the next copy. pv(S): the value product of block i.
template <int NFK, typename Frag, typename SA, typename FIRST, typename STEP1, typename STEP2, typename PV>
__device__ inline void phase_loop(const uint16_t* list, int n, const int32_t* n_a, const float* dKh,
                                  const Frag* Kh, const Frag* Vh, Frag* sK, Frag* sV, int wave, int lane,
                                  FIRST first_qk, STEP1 region1, STEP2 region2, PV pv) {
  constexpr int TILE = NFK * 64;       // fragments per tile
  constexpr int W0 = (NFK + 1) / 2;    // fragments wave 0 copies; wave 1 copies the rest
  // Wave 0 copies fragments [0, W0) of a tile, wave 1 the rest; fragment i of
  // a wave's share sits 1 KB * i after its first one, in both memories (4 KB
  // steps of the scalar bases, the remainder as the immediate offset).
  const uint32_t voff = 16u * static_cast<uint32_t>(lane);
  const int f0 = wave ? W0 : 0, nf = wave ? NFK - W0 : W0;
  auto dma_tile = [&](const Frag* src, Frag* dst) {
    const char* base = reinterpret_cast<const char*>(src + f0 * 64);
    const uint32_t lds = lds_address(dst + f0 * 64);
    [&]<int... I>(std::integer_sequence<int, I...>) {
      ((I < nf ? dma_fragment<(I % 4) * 1024>(base + (I / 4) * 4096, voff, lds + (I / 4) * 4096) : void()), ...);
    }(std::make_integer_sequence<int, W0>{});
  };
  KeyWin win = key_window(list, 0, n, n_a, dKh, lane);
  // key block of list entry e, first being the current window's first entry
  auto block_at = [&](int e, int first) -> int {  // e - first < 128
    return e - first < 64 ? lane_value(win.kb, e - first) : lane_value(win.kb_next, e - first - 64);
  };
  // prologue: logits of block 0, then K(1) and V(0) in flight
  const int kb0 = lane_value(win.kb, 0);
  dma_tile(Kh + (int64_t)kb0 * TILE, sK);
  wait_vmem_keep<0>();
  wg_barrier();
  SA Sa, Sb;
  first_qk(Sa);
  wait_lds();
  wg_barrier();
  if (n > 1) dma_tile(Kh + (int64_t)block_at(1, 0) * TILE, sK);
  dma_tile(Vh + (int64_t)kb0 * TILE, sV);

  auto step = [&](int it, SA& Sc, SA& Sn) {
    const int first = it & ~63;
    const int sl = it - first;
    if (sl == 0 && it > 0) win = key_window(list, it, n, n_a, dKh, lane);
    const int nb = lane_value(win.nb, sl);
    const float dk = lane_value(win.dk, sl);
    const bool more1 = it + 1 < n, more2 = it + 2 < n;
    const int kb1 = more1 ? block_at(it + 1, first) : 0;
    const int kb2 = more2 ? block_at(it + 2, first) : 0;
    // K(i+1) copied (V(i), issued later, may still be in flight). On the last
    // block the logits of the region are computed from the unchanged tile and
    // not used.
    wait_keep_tile<NFK>(wave);
    wg_barrier();
    if (nb < kCap)
      region1.template operator()<true>(Sc, Sn, nb, dk);
    else
      region1.template operator()<false>(Sc, Sn, nb, dk);
    wait_lds();
    wg_barrier();  // both waves are done with sK
    if (more2) dma_tile(Kh + (int64_t)kb2 * TILE, sK);
    region2(Sc);  // returns after its results exist, so the wait below stays after it
    if (more2)
      wait_keep_tile<NFK>(wave);  // V(i) copied, K(i+2) may still be in flight
    else
      wait_vmem_keep<0>();
    wg_barrier();
    pv(Sc);
    wait_lds();
    wg_barrier();  // both waves are done with sV
    if (more1) dma_tile(Vh + (int64_t)kb1 * TILE, sV);
  };
  for (int it = 0; it < n; it += 2) {
    step(it, Sa, Sb);
    if (it + 1 < n) step(it + 1, Sb, Sa);
  }
}

// Double-buffered form of phase_loop for the phases whose key and value tiles
// fit twice into sK and sV (8-bit and MXFP4 tiles at d = 64 and 128). The
// value product of block i-1 moves into iteration i, beside the second part of
// block i's softmax, so both halves of an iteration pair matrix work with
// vector work, and one barrier per block suffices. Iteration i:
//   copy K(i+2) into K buffer i%2 and V(i) into V buffer i%2
//   region1: S' = K(i+1) Q^T interleaved with the first part of block i's softmax
//   region2: U += V(i-1)^T P(i-1)^T interleaved with the rest of block i's softmax
//   rescale_cur(): U *= alpha of block i
//   wait for this wave's copies -> barrier
// and after the last block pv_last(): U += V(n-1)^T P(n-1)^T. The accumulator
// receives the same operations in the same order as in phase_loop (scaling by
// alpha of block i, then the product of block i). first(S, sK0): logits of the
// first block; region1<MASK>(Sc, Sn, Pc, nb, dk, sKn); region2<PV>(Sc, Pc, Pp,
// sVp) with PV = false on block 0; the weights of consecutive blocks alternate
// between two PT values, so no register copies are needed.
template <int NFK, typename Frag, typename SA, typename PT, typename FIRST, typename STEP1, typename STEP2,
          typename RESC, typename PVL>
__device__ inline void phase_loop_db(const uint16_t* list, int n, const int32_t* n_a, const float* dKh,
                                     const Frag* Kh, const Frag* Vh, Frag* sK, Frag* sV, int wave, int lane,
                                     FIRST first_qk, STEP1 region1, STEP2 region2, RESC rescale_cur,
                                     PVL pv_last) {
  constexpr int TILE = NFK * 64;     // fragments per tile
  constexpr int W0 = (NFK + 1) / 2;  // fragments wave 0 copies; wave 1 copies the rest
  const uint32_t voff = 16u * static_cast<uint32_t>(lane);
  const int f0 = wave ? W0 : 0, nf = wave ? NFK - W0 : W0;
  auto dma_tile = [&](const Frag* src, Frag* dst) {
    const char* base = reinterpret_cast<const char*>(src + f0 * 64);
    const uint32_t lds = lds_address(dst + f0 * 64);
    [&]<int... I>(std::integer_sequence<int, I...>) {
      ((I < nf ? dma_fragment<(I % 4) * 1024>(base + (I / 4) * 4096, voff, lds + (I / 4) * 4096) : void()), ...);
    }(std::make_integer_sequence<int, W0>{});
  };
  KeyWin win = key_window(list, 0, n, n_a, dKh, lane);
  auto block_at = [&](int e, int first) -> int {  // e - first < 128
    return e - first < 64 ? lane_value(win.kb, e - first) : lane_value(win.kb_next, e - first - 64);
  };
  // prologue: logits of block 0, then K(1) copied into the second K buffer
  dma_tile(Kh + (int64_t)lane_value(win.kb, 0) * TILE, sK);
  wait_vmem();
  wg_barrier();
  SA Sa, Sb;
  PT Pa, Pb;
  first_qk(Sa, sK);
  if (n > 1) dma_tile(Kh + (int64_t)block_at(1, 0) * TILE, sK + TILE);
  wait_vmem();
  wait_lds();
  wg_barrier();  // K(1) copied; both waves are done with K(0)

  auto step = [&]<bool PV>(int it, SA& Sc, SA& Sn, PT& Pc, PT& Pp) {
    const int first = it & ~63;
    const int sl = it - first;
    if (sl == 0 && it > 0) win = key_window(list, it, n, n_a, dKh, lane);
    const int nb = lane_value(win.nb, sl);
    const float dk = lane_value(win.dk, sl);
    const int kbc = lane_value(win.kb, sl);
    const bool more2 = it + 2 < n;
    const int kb2 = more2 ? block_at(it + 2, first) : 0;
    const int cur = it & 1;
    if (more2) dma_tile(Kh + (int64_t)kb2 * TILE, sK + cur * TILE);  // K(it) was read last iteration
    dma_tile(Vh + (int64_t)kbc * TILE, sV + cur * TILE);              // V(it-2) was read last iteration
    // On the last block the logits of region 1 come from a stale tile and are not used.
    if (nb < kCap)
      region1.template operator()<true>(Sc, Sn, Pc, nb, dk, sK + (cur ^ 1) * TILE);
    else
      region1.template operator()<false>(Sc, Sn, Pc, nb, dk, sK + (cur ^ 1) * TILE);
    region2.template operator()<PV>(Sc, Pc, Pp, sV + (cur ^ 1) * TILE);
    rescale_cur();
    wait_vmem();
    wait_lds();
    wg_barrier();  // K(it+2) and V(it) copied; both waves are done with K(it+1)'s other buffer and V(it-1)
  };
  step.template operator()<false>(0, Sa, Sb, Pa, Pb);
  int it = 1;
  for (; it + 1 < n; it += 2) {
    step.template operator()<true>(it, Sb, Sa, Pb, Pa);
    step.template operator()<true>(it + 1, Sa, Sb, Pa, Pb);
  }
  if (it < n) step.template operator()<true>(it, Sb, Sa, Pb, Pa);
  if ((n - 1) & 1)
    pv_last(Pb, sV + TILE);
  else
    pv_last(Pa, sV);
}

template <int D>
__global__ __launch_bounds__(128) __attribute__((amdgpu_waves_per_eu(2))) void mixed_attn_kernel(AttnArgs args) {
  constexpr int NS16 = D / 16, NS32 = D / 32, NT = D / 32;
  __shared__ f16x8 sK[2 * NS16 * 64];  // key tile of the current block (16 KB at d=128)
  __shared__ f16x8 sV[NT * 4 * 64];    // value tile of the current block
  // wave index as a uniform (scalar) value: LDS fragment addresses stay scalar
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, r = lane & 31, g = lane >> 5;
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
  const int n4 = args.counts[4 * item], n8 = args.counts[4 * item + 1], n16 = args.counts[4 * item + 2];
  // The operands must carry the tag of this layout version and fmt4, with the
  // 16-bit sections when the row has 16-bit blocks; otherwise the row's
  // output is zero and the mismatch is flagged in the lists meta area.
  {
    const uint32_t tag = __float_as_uint(args.g[(item / R) * 4 + 3]);
    const uint32_t err = ((tag & ~0x1Fu) != (args.tag & ~0x1Fu) ? DA2_ATTN_ERR_LAYOUT : 0u) |
                         ((tag & 0xFu) != (args.tag & 0xFu) ? DA2_ATTN_ERR_FMT4 : 0u) |
                         (n16 > 0 && (!(tag & 0x10u) || !args.has16) ? DA2_ATTN_ERR_NO16 : 0u);
    if (err) {
      if (threadIdx.x == 0) atomicOr(reinterpret_cast<uint32_t*>(args.meta) + 1, err);
      const Layout L0 = layout_view(args.layout, R, args.Npad);
      const int nq0 = L0.n_a[item % R], b0 = (item / R) / args.H, h0 = (item / R) % args.H;
      for (int i = threadIdx.x; i < nq0 * D; i += blockDim.x) {
        const int q = i / D, c = i % D;
        const int64_t o = (int64_t)b0 * args.ob + (int64_t)h0 * args.oh +
                          (int64_t)L0.slot2tok[(int64_t)(item % R) * kCap + q] * args.on + c;
        if (args.odtype == DA2_FP32)
          reinterpret_cast<float*>(args.O)[o] = 0.0f;
        else
          reinterpret_cast<uint16_t*>(args.O)[o] = 0;
      }
      return;
    }
  }
  const uint16_t* keys = args.keys + (int64_t)item * R;
  const int64_t blk0 = (int64_t)bh * R;  // first block of this head
  const float* dKh = args.dK + blk0;
  const float rsqd = 1.0f / sqrtf((float)D);

  f32x16 U[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) U[t] = f32x16{};
  float m = -INFINITY, l = 0.0f;
  const float gV = args.g[bh * 4 + 2];
  const bool mx = args.fmt4 == DA2_FMT4_MXFP4;

  // ------------------------------ NVFP4 phase ------------------------------
  if (n4 > 0 && !mx) {
    const float c4 = args.g[bh * 4 + 0] * args.g[bh * 4 + 1] * kLog2e * rsqd;
    // query fragments of this wave's tile, decoded once from the packed Q section
    f16x8 Qf[NS16];
    {
      NvShare<D> qx;
      nv_load_qk<D>(qx, args.Q4 + (blk0 + a) * nv_block_bytes(D), qt, lane);
#pragma unroll
      for (int s = 0; s < NS16; ++s) Qf[s] = nv_frag_qk<D>(qx, s);
    }
    f16x8 P[4];
    float alpha = 1.0f;
    typedef f32x16 SA[2];
    auto qk = [&](SA& S) {
      S[0] = S[1] = f32x16{};
#pragma unroll
      for (int s = 0; s < NS16; ++s)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          S[j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(sK[(j * NS16 + s) * 64 + lane], Qf[s], S[j], 0, 0, 0);
    };
    // Softmax state of the current block, shared by the two regions.
    float gm0 = 0.0f, gm1 = 0.0f, mn = 0.0f;
    Fp4Group G0, G1;
    // Region 1: logits of the next block (NS16 stages of two MFMAs, operands
    // read one stage ahead) with the row maxima, the first group's weights and
    // operands, the second group's scale (six pieces over the stages) and one
    // value fragment decoded into sV per stage.
    auto region1 = [&]<bool MASK, typename VDEC>(SA& Sc, SA& Sn, int nb, VDEC vdec) {
      if constexpr (MASK) mask_tail(Sc, nb, g);
      f16x8 k0 = sK[lane], k1 = sK[NS16 * 64 + lane];
      constexpr int NP = 6;
#pragma unroll
      for (int s = 0; s < NS16; ++s) {
        f16x8 n0 = k0, n1 = k1;
        if (s + 1 < NS16) {
          n0 = sK[(s + 1) * 64 + lane];
          n1 = sK[(NS16 + s + 1) * 64 + lane];
        }
        Sn[0] = __builtin_amdgcn_mfma_f32_32x32x16_f16(k0, Qf[s], s == 0 ? f32x16{} : Sn[0], 0, 0, 0);
        Sn[1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(k1, Qf[s], s == 0 ? f32x16{} : Sn[1], 0, 0, 0);
        vdec(s);
#pragma unroll
        for (int piece = 0; piece < NP; ++piece) {
          if (piece * NS16 / NP != s) continue;
          if (piece == 0) {
            gm0 = max16(Sc[0]);
          } else if (piece == 1) {
            gm1 = max16(Sc[1]);
            mn = new_max(fmaxf(gm0, gm1), c4, m, l, alpha);
          } else if (piece == 2) {
            fp4_setup(G0, gm0, c4, mn);
            fp4_exps<0, 6>(G0, Sc[0], c4);
          } else if (piece == 3) {
            fp4_exps<6, 10>(G0, Sc[0], c4);
          } else if (piece == 4) {
            fp4_exps<10, 16>(G0, Sc[0], c4);
          } else {
            fp4_pack(G0, P[0], P[1]);
            fp4_setup(G1, gm1, c4, mn);
          }
        }
        fence();
        k0 = n0;
        k1 = n1;
      }
    };
    // U += V^T P^T; value fragments are read two MFMAs ahead. The MFMAs of the
    // first group (k < 2 NT) carry the second group's exponentials and its
    // fp16 operands, which the remaining MFMAs use; one key fragment of the
    // block after next is decoded into sK every second MFMA.
    auto pv = [&]<typename KDEC>(SA& Sc, KDEC kdec) {
      if (__ballot(alpha != 1.0f)) rescale<NT>(U, alpha);
      constexpr int NM = 4 * NT;
      auto vfrag = [&](int k) { return sV[((k % NT) * 4 + k / NT) * 64 + lane]; };
      f16x8 v0 = vfrag(0), v1 = vfrag(1);
#pragma unroll
      for (int k = 0; k < NM; ++k) {
        const f16x8 cur = (k & 1) ? v1 : v0;
        if (k + 2 < NM) {
          if (k & 1)
            v1 = vfrag(k + 2);
          else
            v0 = vfrag(k + 2);
        }
        U[k % NT] = __builtin_amdgcn_mfma_f32_32x32x16_f16(cur, P[k / NT], U[k % NT], 0, 0, 0);
        // pieces of the second group, spread over the first group's MFMAs
        constexpr int NG = 2 * NT;  // MFMAs that read P[0], P[1]
        if (k == 0) fp4_exps<0, 4>(G1, Sc[1], c4);
        if (k == NG / 4) fp4_exps<4, 8>(G1, Sc[1], c4);
        if (k == NG / 2) fp4_exps<8, 12>(G1, Sc[1], c4);
        if (k == 3 * NG / 4) fp4_exps<12, 16>(G1, Sc[1], c4);
        if (k == NG - 1) {
          fp4_pack(G1, P[2], P[3]);
          l += weight_sum(G0) + weight_sum(G1);
        }
        if (k & 1) kdec(k >> 1);
        fence();
      }
    };
    nv_phase_loop<D, SA>(keys, n4, L.n_a, dKh, args.K4 + blk0 * nv_block_bytes(D), args.V4 + blk0 * nv_block_bytes(D),
                         sK, sV, wave, lane, qk, region1, pv);
  }

  // ------------------------------ MXFP4 phase ------------------------------
  // The scaled MFMAs apply the E8M0 block scales of both operands, so logits
  // and numerator are in the common units. Key rows follow kappa_mx: lane half
  // g of both logit tiles holds the 32-slot block 32g + [0, 32) (register i of
  // tile j: slot 32g + 16j + i), which is also the k order of the value
  // product, so each lane quantizes one whole weight block of its query.
  if (n4 > 0 && mx) {
    constexpr int NS64 = D / 64, NFM = D / 32 + 1;  // fragments per tile: data, then scales
    const float c4 = kLog2e * rsqd;
    const i32x4* Qa = reinterpret_cast<const i32x4*>(args.Q4mx) + (blk0 + a) * (NFM * 64);
    i32x4 Qf[NS64];
    int qsc[NS64];
    const i32x4 qsw = Qa[2 * NS64 * 64 + lane];
#pragma unroll
    for (int s = 0; s < NS64; ++s) {
      Qf[s] = Qa[(qt * NS64 + s) * 64 + lane];
      qsc[s] = qt ? qsw[NS64 + s] : qsw[s];
    }
    float alpha = 1.0f;
    typedef f32x16 SA[2];
    struct PT {
      i32x4 P;  // E2M1 weight codes of the block's two 16-slot groups per lane
      int psc;  // their E8M0 scale word
    };
    auto qk = [&](SA& S, const f16x8* sK0) {
      const i32x4* sKm = reinterpret_cast<const i32x4*>(sK0);
      const i32x4 ksw = sKm[2 * NS64 * 64 + lane];
      S[0] = S[1] = f32x16{};
#pragma unroll
      for (int s = 0; s < NS64; ++s)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          S[j] = mfma_fp4(sKm[(j * NS64 + s) * 64 + lane], Qf[s], S[j], ksw[j * NS64 + s], qsc[s]);
    };
    // Softmax state of the current block, shared by the two regions.
    float off = 0.0f, sum = 0.0f;
    int ke = 0;
    // Region 1: logits of the next block (NS64 stages of two MFMAs) with the
    // maxima, the block exponent and the first quarter of the weights.
    auto region1 = [&]<bool MASK>(SA& Sc, SA& Sn, PT& Pc, int nb, float, const f16x8* sKn) {
      const i32x4* sKm = reinterpret_cast<const i32x4*>(sKn);
      if constexpr (MASK) mask_tail_mx(Sc, nb, g);
      const i32x4 ksw = sKm[2 * NS64 * 64 + lane];
      i32x4 k0 = sKm[lane], k1 = sKm[NS64 * 64 + lane];
      constexpr int NP = 2;
#pragma unroll
      for (int s = 0; s < NS64; ++s) {
        i32x4 n0 = k0, n1 = k1;
        if (s + 1 < NS64) {
          n0 = sKm[(s + 1) * 64 + lane];
          n1 = sKm[(NS64 + s + 1) * 64 + lane];
        }
        Sn[0] = mfma_fp4(k0, Qf[s], s == 0 ? f32x16{} : Sn[0], ksw[s], qsc[s]);
        Sn[1] = mfma_fp4(k1, Qf[s], s == 0 ? f32x16{} : Sn[1], ksw[NS64 + s], qsc[s]);
#pragma unroll
        for (int piece = 0; piece < NP; ++piece) {
          if (piece * NS64 / NP != s) continue;
          if (piece == 0) {
            const float gm = fmaxf(max16(Sc[0]), max16(Sc[1]));  // this lane's block
            const float mn = new_max(gm, c4, m, l, alpha);
            ke = mx_weight_exponent(gm, c4, mn);
            off = -mn - (float)ke;
          } else {
            sum = 0.0f;
            Pc.P[0] = mx_codes8<0>(Sc[0], c4, off, sum);
          }
        }
        fence();
        k0 = n0;
        k1 = n1;
      }
    };
    // Region 2: U += V^T P^T of the previous block (one scaled MFMA per
    // channel tile) beside the rest of the weights, the scale word and l.
    auto region2 = [&]<bool PV>(SA& Sc, PT& Pc, PT& Pp, const f16x8* sVp) {
      const i32x4* sVm = reinterpret_cast<const i32x4*>(sVp);
      const i32x4 vsw = sVm[NT * 64 + lane];
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        if constexpr (PV) U[t] = mfma_fp4(sVm[t * 64 + lane], Pp.P, U[t], vsw[t], Pp.psc);
        // the three remaining groups of eight weights over the NT products
#pragma unroll
        for (int q = 1; q < 4; ++q) {
          if ((q - 1) * NT / 3 != t) continue;
          // each piece's results are used in its stage, which keeps the piece there
          if (q == 1) Pc.P[1] = mx_codes8<8>(Sc[0], c4, off, sum), after(Pc.P[1]), after(sum);
          if (q == 2) Pc.P[2] = mx_codes8<0>(Sc[1], c4, off, sum), after(Pc.P[2]), after(sum);
          if (q == 3) Pc.P[3] = mx_codes8<8>(Sc[1], c4, off, sum), after(Pc.P[3]), after(sum);
        }
        fence();
      }
      Pc.psc = ke + 127;
      l += __builtin_amdgcn_ldexpf(sum, ke);  // Pt = 2^k y, exact scaling
      // computed here, beside the products (not sunk into the next iteration)
      after(Pc.P), after(Pc.psc), after(l);
    };
    auto rescale_cur = [&]() {
      if (__ballot(alpha != 1.0f)) rescale<NT>(U, alpha);
    };
    auto pv_last = [&](PT& Pp, const f16x8* sVp) {
      const i32x4* sVm = reinterpret_cast<const i32x4*>(sVp);
      const i32x4 vsw = sVm[NT * 64 + lane];
#pragma unroll
      for (int t = 0; t < NT; ++t) U[t] = mfma_fp4(sVm[t * 64 + lane], Pp.P, U[t], vsw[t], Pp.psc);
    };
    static_assert(2 * NFM * 1024 <= sizeof(sK) && 2 * NFM * 1024 <= sizeof(sV), "two MXFP4 tiles fit");
    phase_loop_db<NFM, f16x8, SA, PT>(keys, n4, L.n_a, dKh, reinterpret_cast<const f16x8*>(args.K4mx) + blk0 * (NFM * 64),
                                      reinterpret_cast<const f16x8*>(args.V4mx) + blk0 * (NFM * 64), sK, sV, wave,
                                      lane, qk, region1, region2, rescale_cur, pv_last);
  }

  // per-lane channel of accumulator register i of channel tile t
  auto chan = [&](int t, int i) { return 32 * t + 8 * (i >> 2) + 4 * g + (i & 3); };
  const float eta = exp2_fast(-kExpOffset);
  const float* dV = args.dV + (int64_t)bh * D;

  // ------------------------------- INT8 phase -------------------------------
  if (n8 > 0) {
    // Enter: U_c <- U_c / (eta delta_c), l <- l / eta (after restoring the 4-bit
    // phase's factor g_V/2688).
    const float restore = n4 > 0 && !mx ? gV / 2688.0f : 1.0f;
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
    float alpha = 1.0f;
    typedef i32x16 SA[2];
    auto qk = [&](SA& S, const f16x8* sK0) {
      const i32x4* sK8 = reinterpret_cast<const i32x4*>(sK0);
      S[0] = S[1] = i32x16{};
#pragma unroll
      for (int s = 0; s < NS32; ++s)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          S[j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(sK8[(j * NS32 + s) * 64 + lane], Qf[s], S[j], 0, 0, 0);
    };
    // Softmax state of the current block, shared by the two regions.
    f32x16 sf[2];
    float cb = 0.0f, off = 0.0f, s0 = 0.0f;
    int w[2];
    // Region 1: logits of the next block (NS32 stages of two int8 MFMAs) with
    // the conversion, the row maxima and the first quarter of the weights.
    auto region1 = [&]<bool MASK>(SA& Sc, SA& Sn, i32x8&, int nb, float dk, const f16x8* sKn) {
      const i32x4* sK8 = reinterpret_cast<const i32x4*>(sKn);
      i32x4 k0 = sK8[lane], k1 = sK8[NS32 * 64 + lane];
      cb = c8a * dk;
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int i = 0; i < 16; ++i) sf[j][i] = (float)Sc[j][i];
      if constexpr (MASK) mask_tail(sf, nb, g);
      constexpr int NP = 2;
#pragma unroll
      for (int s = 0; s < NS32; ++s) {
        i32x4 n0 = k0, n1 = k1;
        if (s + 1 < NS32) {
          n0 = sK8[(s + 1) * 64 + lane];
          n1 = sK8[(NS32 + s + 1) * 64 + lane];
        }
        Sn[0] = __builtin_amdgcn_mfma_i32_32x32x32_i8(k0, Qf[s], s == 0 ? i32x16{} : Sn[0], 0, 0, 0);
        Sn[1] = __builtin_amdgcn_mfma_i32_32x32x32_i8(k1, Qf[s], s == 0 ? i32x16{} : Sn[1], 0, 0, 0);
#pragma unroll
        for (int piece = 0; piece < NP; ++piece) {
          if (piece * NS32 / NP != s) continue;
          if (piece == 0)
            off = kExpOffset - new_max(fmaxf(max16(sf[0]), max16(sf[1])), cb, m, l, alpha);
          else
            s0 = fp8_weights8<0>(sf[0], cb, off, w[0], w[1]);
        }
        fence();
        k0 = n0;
        k1 = n1;
      }
    };
    // Region 2: U += V^T P^T of the previous block (fp8 x fp8, unit scales;
    // value fragments read one MFMA ahead) beside the remaining three quarters
    // of the weights, the fp8 P^T operand and l.
    auto vfrag = [&](const i32x4* sV8, int t) {
      const i32x4 v0 = sV8[(t * 2 + 0) * 64 + lane], v1 = sV8[(t * 2 + 1) * 64 + lane];
      return i32x8{v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
    };
    auto region2 = [&]<bool PV>(SA&, i32x8& Pc, i32x8& Pp, const f16x8* sVp) {
      const i32x4* sV8 = reinterpret_cast<const i32x4*>(sVp);
      float s1 = 0.0f, s2 = 0.0f, s3 = 0.0f;
      int w2[6];
      i32x8 vf;
      if constexpr (PV) vf = vfrag(sV8, 0);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        if constexpr (PV) {
          const i32x8 cur = vf;
          if (t + 1 < NT) vf = vfrag(sV8, t + 1);
          U[t] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(cur, Pp, U[t], 0, 0, 0, 127, 0, 127);
        }
#pragma unroll
        for (int q = 1; q < 4; ++q) {
          if ((q - 1) * NT / 3 != t) continue;
          // each piece's results are used in its stage, which keeps the piece there
          if (q == 1) s1 = fp8_weights8<8>(sf[0], cb, off, w2[0], w2[1]), after(s1), after(w2[0]), after(w2[1]);
          if (q == 2) s2 = fp8_weights8<0>(sf[1], cb, off, w2[2], w2[3]), after(s2), after(w2[2]), after(w2[3]);
          if (q == 3) s3 = fp8_weights8<8>(sf[1], cb, off, w2[4], w2[5]), after(s3), after(w2[4]), after(w2[5]);
        }
        fence();
      }
      Pc = i32x8{w[0], w[1], w2[0], w2[1], w2[2], w2[3], w2[4], w2[5]};
      l += (s0 + s1) + (s2 + s3);
      // computed here, beside the products (not sunk into the next iteration)
      after(Pc), after(l);
    };
    auto rescale_cur = [&]() {
      if (__ballot(alpha != 1.0f)) rescale<NT>(U, alpha);
    };
    auto pv_last = [&](i32x8& Pp, const f16x8* sVp) {
      const i32x4* sV8 = reinterpret_cast<const i32x4*>(sVp);
#pragma unroll
      for (int t = 0; t < NT; ++t)
        U[t] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(vfrag(sV8, t), Pp, U[t], 0, 0, 0, 127, 0, 127);
    };
    wait_lds();
    wg_barrier();  // the NVFP4 phase is done with sK / sV
    static_assert(2 * 2 * NS32 * 1024 <= sizeof(sK) && 2 * 2 * NS32 * 1024 <= sizeof(sV), "two 8-bit tiles fit");
    phase_loop_db<2 * NS32, f16x8, SA, i32x8>(keys + n4, n8, L.n_a, dKh,
                                             reinterpret_cast<const f16x8*>(args.K8) + blk0 * (kCap * D / 16),
                                             reinterpret_cast<const f16x8*>(args.V8) + blk0 * (kCap * D / 16), sK, sV,
                                             wave, lane, qk, region1, region2, rescale_cur, pv_last);
    // Exit: U_c <- eta delta_c U_c, l <- eta l
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 16; ++i) U[t][i] *= eta * dV[chan(t, i)];
    l *= eta;
  } else if (n4 > 0 && !mx) {
    const float restore = gV / 2688.0f;
#pragma unroll
    for (int t = 0; t < NT; ++t) U[t] *= restore;
  }

  // ------------------------------ 16-bit phase ------------------------------
  // Continues in the common units: fp16 Q, K, V; Pt = 2^(s log2 e / sqrt d - m)
  // in fp32 (denominator), rounded to fp16 for the value product.
  if (n16 > 0) {
    const float c16 = kLog2e * rsqd;
    f16x8 Qf[NS16];
    const f16x8* Qa = reinterpret_cast<const f16x8*>(args.Q16) + (blk0 + a) * (kCap * D / 8);
#pragma unroll
    for (int s = 0; s < NS16; ++s) Qf[s] = Qa[(qt * NS16 + s) * 64 + lane];
    f16x8 P[4];
    float alpha = 1.0f;
    typedef f32x16 SA[2];
    auto qk = [&](SA& S) {
      S[0] = S[1] = f32x16{};
#pragma unroll
      for (int s = 0; s < NS16; ++s)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          S[j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(sK[(j * NS16 + s) * 64 + lane], Qf[s], S[j], 0, 0, 0);
    };
    float gm0 = 0.0f, gm1 = 0.0f, mn = 0.0f, sum0 = 0.0f, sum1 = 0.0f;
    // Region 1: logits of the next block with the maxima and the first
    // group's weights of the current block (four pieces over the stages).
    auto region1 = [&]<bool MASK>(SA& Sc, SA& Sn, int nb, float) {
      if constexpr (MASK) mask_tail(Sc, nb, g);
      f16x8 k0 = sK[lane], k1 = sK[NS16 * 64 + lane];
      constexpr int NP = 4;
      sum0 = 0.0f;
#pragma unroll
      for (int s = 0; s < NS16; ++s) {
        f16x8 n0 = k0, n1 = k1;
        if (s + 1 < NS16) {
          n0 = sK[(s + 1) * 64 + lane];
          n1 = sK[(NS16 + s + 1) * 64 + lane];
        }
        Sn[0] = __builtin_amdgcn_mfma_f32_32x32x16_f16(k0, Qf[s], s == 0 ? f32x16{} : Sn[0], 0, 0, 0);
        Sn[1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(k1, Qf[s], s == 0 ? f32x16{} : Sn[1], 0, 0, 0);
#pragma unroll
        for (int piece = 0; piece < NP; ++piece) {
          if (piece * NS16 / NP != s) continue;
          if (piece == 0) {
            gm0 = max16(Sc[0]);
          } else if (piece == 1) {
            gm1 = max16(Sc[1]);
            mn = new_max(fmaxf(gm0, gm1), c16, m, l, alpha);
          } else if (piece == 2) {
            P[0] = half_weights8<0>(Sc[0], c16, mn, sum0);
          } else {
            P[1] = half_weights8<8>(Sc[0], c16, mn, sum0);
          }
        }
        fence();
        k0 = n0;
        k1 = n1;
      }
    };
    // Region 2: the second group's weights.
    auto region2 = [&](SA& Sc) {
      sum1 = 0.0f;
      P[2] = half_weights8<0>(Sc[1], c16, mn, sum1);
      P[3] = half_weights8<8>(Sc[1], c16, mn, sum1);
      l += sum0 + sum1;
      after(P[0]), after(P[1]), after(P[2]), after(P[3]), after(l);
    };
    // U += V^T P^T; value fragments are read two MFMAs ahead.
    auto pv = [&](SA& Sc) {
      if (__ballot(alpha != 1.0f)) rescale<NT>(U, alpha);
      constexpr int NM = 4 * NT;
      auto vfrag = [&](int k) { return sV[((k % NT) * 4 + k / NT) * 64 + lane]; };
      f16x8 v0 = vfrag(0), v1 = vfrag(1);
#pragma unroll
      for (int k = 0; k < NM; ++k) {
        const f16x8 cur = (k & 1) ? v1 : v0;
        if (k + 2 < NM) {
          if (k & 1)
            v1 = vfrag(k + 2);
          else
            v0 = vfrag(k + 2);
        }
        U[k % NT] = __builtin_amdgcn_mfma_f32_32x32x16_f16(cur, P[k / NT], U[k % NT], 0, 0, 0);
        fence();
      }
    };
    wait_lds();
    wg_barrier();  // the previous phase is done with sK / sV
    phase_loop<2 * NS16, f16x8, SA>(keys + n4 + n8, n16, L.n_a, dKh,
                                    reinterpret_cast<const f16x8*>(args.K16) + blk0 * (kCap * D / 8),
                                    reinterpret_cast<const f16x8*>(args.V16) + blk0 * (kCap * D / 8), sK, sV, wave,
                                    lane, qk, region1, region2, pv);
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
