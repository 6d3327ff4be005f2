/*
 * da2.h - C ABI of the DraftAttention2 hot path on AMD Instinct MI355X (gfx950).
 *
 * Paper: "DraftAttention2: Fast Video Diffusion with Low-Resolution-Guided
 * Mixed-Precision Attention". One attention layer is computed in four calls,
 * all asynchronous on a caller-given HIP stream:
 *
 *   da2_draft_map      pooled draft attention map            (descriptor eq., Def. 3.1)
 *   da2_rank_assign    shared ranking into 16/8/4-bit or skip (Algorithm 1, routing appendix)
 *   da2_prep_operands  per-block INT8 / E4M3 / NVFP4 (or MXFP4) operands (format appendix,
 *                      NVFP4 eqs.)
 *   da2_mixed_attn     one phased mixed-precision attention   (phased execution,
 *                      kernel with shared softmax state       precision-state-conversion eq.)
 *
 * Conventions for every call
 * --------------------------
 * - Tokens are numbered frame-major raster: n = t*Hg*Wg + y*Wg + x. Each
 *   frame is split into R_f regions of at most C = 64 tokens (p->partition):
 *   DA2_PART_TILES8: 8x8 spatial tiles, block a = (t*nI + i)*nJ + j with
 *     nI = ceil(Hg/8), nJ = ceil(Wg/8), R_f = nI*nJ;
 *   DA2_PART_RAGGED (fused-reordering paragraph, ragged-padding and
 *     region-perimeter equations): R_f = ceil(Hg*Wg/64) connected regions
 *     with less than one block of padding per frame. Candidates split the
 *     frame into nb bands of balanced height (larger first), along rows or
 *     along columns; each band is walked in a snake order (down one column
 *     and up the next; along one row and back for column bands) and cut into
 *     ceil(band/64) consecutive runs of balanced size (larger first). Valid
 *     candidates have R_f runs; the smallest total perimeter (fewest
 *     neighbour pairs split between regions) wins, then row bands, then
 *     fewer bands. Regions are numbered band by band, run by run, and block
 *     a = t*R_f + region.
 *   R = T*R_f blocks, Npad = 64*R slots. The slots of a block hold its valid
 *   tokens in row-major order, then padding.
 * - Every device buffer is allocated and owned by the caller; sizes come from
 *   da2_sizes(). The library never allocates or frees device memory, never
 *   synchronizes the host and keeps no mutable global state (the one
 *   exception is the fixed per-device scratch array that
 *   da2_rank_assign_noalloc uses instead of a workspace). Buffers that a
 *   call writes must not be read or written by other work on other streams
 *   until the call has completed on its stream.
 * - "device" pointers must be device-accessible (hipMalloc / torch cuda
 *   tensors); "host" pointers are ordinary process memory.
 * - Every entry point validates its arguments on the host before touching the
 *   GPU and returns a da2_status; no C++ exception crosses this interface.
 *   Launch failures return DA2_ERR_HIP. Nothing is written when validation
 *   fails.
 * - Only gfx950 devices are supported (DA2_ERR_UNSUPPORTED otherwise). Head
 *   dimension d must be 64 or 128 (DA2_ERR_UNSUPPORTED otherwise).
 */
#ifndef DA2_H
#define DA2_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DA2_OK = 0,
  DA2_ERR_INVALID_ARG = -1, /* a null pointer, a bad size or an out-of-range value   */
  DA2_ERR_UNSUPPORTED = -2, /* valid request the library does not implement / no gfx950 */
  DA2_ERR_WORKSPACE = -3,   /* workspace smaller than da2_sizes() asks for           */
  DA2_ERR_HIP = -4          /* the HIP runtime reported an error (launch or query)   */
} da2_status;

typedef enum { DA2_BF16 = 0, DA2_FP32 = 1 } da2_dtype;
typedef enum { DA2_SCOPE_HEAD = 0, DA2_SCOPE_ROW = 1 } da2_scope;

/* Encodings of the 4-bit path. NVFP4 is the paper's format (E2M1 with an
 * E4M3 scale per 16 elements and a per-tensor scale). MXFP4 is the OCP
 * microscaling format that gfx950's matrix cores apply natively (E2M1 with a
 * power-of-two E8M0 scale per 32 elements); it is a hardware counterpart of
 * the paper's 4-bit path, not a format of the paper. */
typedef enum { DA2_FMT4_NVFP4 = 0, DA2_FMT4_MXFP4 = 1 } da2_fmt4;

/* Region partitions of each frame (capacity C = 64 slots per block). */
typedef enum {
  DA2_PART_TILES8 = 0, /* 8x8 spatial tiles: R_f = ceil(Hg/8)*ceil(Wg/8) blocks per frame */
  DA2_PART_RAGGED = 1  /* ragged minimum-perimeter regions: R_f = ceil(Hg*Wg/64) */
} da2_partition;

/* Problem shape: batch B, heads H, head dim d, latent grid T x Hg x Wg
 * (N = T*Hg*Wg tokens), region partition (da2_partition). */
typedef struct {
  int32_t B, H, d, T, Hg, Wg;
  int32_t partition;
} da2_problem;

/* A [B, H, N, d] tensor with d contiguous; strides are in elements. Input
 * tensors (Q, K, V) are read in 16-byte vectors: their base pointers must be
 * 16-byte aligned and every stride a multiple of 16 bytes (8 bf16 or 4 fp32
 * elements), else the call returns DA2_ERR_INVALID_ARG. */
typedef struct {
  int64_t stride_b, stride_h, stride_n;
  int32_t dtype; /* da2_dtype */
  int32_t reserved;
} da2_tensor;

/* Byte sizes of the caller-allocated device buffers of one problem. */
typedef struct {
  int32_t R, Npad;
  int64_t layout_bytes; /* int32 index maps, see da2_layout_build        */
  int64_t A_bytes;      /* float32 draft map [B,H,R,R]                    */
  int64_t cls_bytes;    /* uint8 precision map [B,H,R,R]                  */
  int64_t stats_bytes;  /* per-head amax statistics                       */
  int64_t lists_bytes;  /* per-row key-block lists, counts, work order    */
  int64_t ops_bytes;    /* encoded operands                               */
  int64_t ws_draft_bytes, ws_rank_bytes, ws_prep_bytes;
} da2_sizes_t;

/* Version of the documented layouts of the ops and lists buffers
 * (da2_ops_offsets, da2_lists_offsets). Version 2: packed NVFP4 sections,
 * sections sized and ordered by (fmt4, with16), encoding tag in g word 3. */
#define DA2_OPS_LAYOUT_VERSION 2

/* Error flags that da2_mixed_attn ORs into word 1 of the lists meta area
 * (da2_lists_offsets [3]) when the operands do not match the call; the rows
 * concerned are written as zeros. */
#define DA2_ATTN_ERR_LAYOUT 1u /* ops not written by this layout version (or never written) */
#define DA2_ATTN_ERR_FMT4 2u   /* ops prepared with another fmt4 */
#define DA2_ATTN_ERR_NO16 4u   /* a row has 16-bit blocks but ops were prepared with with16 = 0 */

/* Human-readable name of a status code (static string, never NULL). */
const char* da2_status_string(int32_t status);

/* Host only. Fills *out for problem p. The ranking scope sets ws_rank_bytes;
 * fmt4 (da2_fmt4) and with16 (0 or 1) set ops_bytes: the ops buffer holds only
 * the sections a run with that 4-bit encoding and 16-bit option writes.
 * Errors: INVALID_ARG for non-positive dims, an unknown partition, scope,
 * fmt4 or with16, or sizes that overflow the index types or launch grids
 * (R > 65535 blocks, B*H > 32767, B*H*R > 2^31-1); UNSUPPORTED for a head
 * dimension d other than 64 or 128 (every entry point that takes p). */
int32_t da2_sizes(const da2_problem* p, int32_t scope, int32_t fmt4, int32_t with16, da2_sizes_t* out);

/* DA2_OPS_LAYOUT_VERSION of the library (host only). */
int32_t da2_ops_layout_version(void);

/* Host only: region layout (fused-preparation section: each region packed
 * into one contiguous block, valid counts n_a, inverse index map).
 * host_layout receives layout_bytes/4 int32 values:
 *   [0, R)            n_a        valid tokens of block a (1..64)
 *   [R, R+Npad)       slot2tok   token of each slot, -1 for padding
 *   [R+Npad, +N)      tok2slot   slot of each token
 * Copy it to a device buffer of layout_bytes for the compute calls. */
int32_t da2_layout_build(const da2_problem* p, int32_t* host_layout, int64_t n_ints);

/* Draft map (descriptor equation; Definition 3.1):
 *   Qbar_a = mean, Qmax_a = channel max of Q over the valid tokens of block a
 *   (K alike), A = (1-lambda) softmax_row(Qbar Kbar^T/sqrt d)
 *                 + lambda softmax_row(Qmax Kmax^T/sqrt d),
 * pooling, logits and softmax in float64, A rounded once to float32.
 *   Q, K     device, [B,H,N,d] per *qk (bf16 or fp32)
 *   layout   device, as built by da2_layout_build
 *   lambda   in [0, 1]
 *   A        device out, float32 [B,H,R,R] row-major (row = query block)
 *   stats    device out, stats_bytes: uint32 [B*H][4 + d]; entry 0/1 hold the
 *            float32 bit patterns of max|Q|, max|K| of each head (entries 2..
 *            are written by da2_prep_operands)
 *   ws       device scratch of ws_draft_bytes (see da2_ws_draft_offsets). */
int32_t da2_draft_map(const void* Q, const void* K, const da2_tensor* qk, const int32_t* layout,
                      const da2_problem* p, double lambda, float* A, void* stats, void* ws,
                      int64_t ws_bytes, void* stream);

/* Offsets (bytes) inside ws_draft of: [0] Qbar, [1] Qmax, [2] Kbar, [3] Kmax
 * (float64 [B,H,R,d] each), [4] S_avg, [5] S_max (float64 [B,H,R,R] logits),
 * [6] the per-block max|Q| and max|K| (float32 [2][B*H][R]) that are reduced
 * into stats entries 0 and 1. */
int32_t da2_ws_draft_offsets(const da2_problem* p, int64_t* offsets7);

/* Shared ranking (Algorithm 1; routing appendix). Quotas from budgets
 * num16/den, num8/den and num4/den over M = R*R pairs per head
 * (DA2_SCOPE_HEAD) or M = R pairs per query block (DA2_SCOPE_ROW), cumulative
 * and rounded half up: with h(n) = floor(n*M/den + 1/2),
 *   T16 = h(num16), T8 = h(num16+num8) - T16, T4 = h(num16+num8+num4) - T16 - T8.
 * Pairs are ranked by (A descending, pair index ascending) with pair index
 * a*R+b (head) or b (row); ranks [0,T16) -> 16, the next T8 -> 8, the next
 * T4 -> 4, others -> 0. The hot path runs with num16 = 0.
 *   A      device float32 [B,H,R,R] (e.g. from da2_draft_map)
 *   cls    device out, uint8 [B,H,R,R] in {0,4,8,16}
 *   lists  device out, lists_bytes (see da2_lists_offsets)
 * Errors: INVALID_ARG if den <= 0, a budget < 0, num16+num8+num4 > den, or
 * head scope with R*R >= 2^22; UNSUPPORTED for row scope with R > 8192. */
int32_t da2_rank_assign(const float* A, const da2_problem* p, int32_t num16, int32_t num8,
                        int32_t num4, int32_t den, int32_t scope, uint8_t* cls, void* lists,
                        void* ws, int64_t ws_bytes, void* stream);

/* Allocation-free variant of da2_rank_assign, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc). Same arguments, results and errors as
 * da2_rank_assign, except that no workspace is passed: the ranking's
 * workspace is a fixed device array of DA2_RANK_NOALLOC_MAX_BYTES inside the
 * library (one copy per device, held until the process ends; its address is
 * looked up once per device on the first call there). The call allocates
 * nothing and clears what must start at zero with kernels.
 *   Errors: DA2_ERR_WORKSPACE when the problem's ws_rank_bytes (da2_sizes)
 *   exceeds DA2_RANK_NOALLOC_MAX_BYTES; DA2_ERR_HIP when the array's device
 *   address cannot be looked up.
 * Calls on one device share the array: two such calls that overlap in time on
 * the same device (different streams or threads without ordering) race and
 * give undefined results. Calls on different devices do not interact. */
#define DA2_RANK_NOALLOC_MAX_BYTES (8ll << 20)
int32_t da2_rank_assign_noalloc(const float* A, const da2_problem* p, int32_t num16, int32_t num8,
                                int32_t num4, int32_t den, int32_t scope, uint8_t* cls, void* lists,
                                void* stream);

/* Offsets (bytes) inside lists:
 *   [0] keys   uint16 [B*H*R][R]: row (b,h,a) holds its 4-bit key blocks
 *              ascending in [0,n4), then its 8-bit key blocks ascending in
 *              [n4, n4+n8), then its 16-bit key blocks ascending in
 *              [n4+n8, n4+n8+n16)
 *   [1] counts int32 [B*H*R][4] = (n4, n8, n16, 0)
 *   [2] order  int32 [B*H*R]: the work order of the rows (b*H+h)*R+a: grouped
 *              by head and by row parity, most expensive first in each group
 *              (cost 3 per 4-bit or 16-bit block and 2 per 8-bit block, the
 *              measured ratio of the attention's per-tile times);
 *              attention workgroup w takes order[(w mod 8)*ceil(n/8) + w div 8]
 *              (any permutation of the rows is a valid order)
 *   [3] meta   int32 [8]: [0] = number of rows in order; [1] = error flags
 *              (DA2_ATTN_ERR_*) of da2_mixed_attn calls on these lists,
 *              cleared by da2_rank_assign                                  */
int32_t da2_lists_offsets(const da2_problem* p, int64_t* offsets4);

/* Operand preparation (format appendix; NVFP4 quantization equation):
 *   INT8 Q, K: per block delta = f32(f32(amax/127) + 1e-7), code =
 *     round-half-away(f32(x * f32(1/delta))).
 *   E4M3 V: per (b,h,channel) delta_c = f32(amax_c / 2.25) over all valid
 *     keys, code = E4M3_rne(f32(v * f32(1/delta_c))); zero channels -> 0.
 *   NVFP4 Q, K (16-channel groups) and V (16 key slots per channel):
 *     g = f32(amax_head / 2688) (1 if zero), sigma = E4M3_rne(f32(amax_G /
 *     f32(6 g))), e = E2M1_rne(f32(x * f32(1 / f32(g sigma)))); sigma == 0 ->
 *     zeros. Stored as 4-bit E2M1 codes with one E4M3 scale byte per group
 *     (4.5 bits per value); the attention decodes sigma*e to fp16 (exact: at
 *     most 6 significant bits), since gfx950 has no MFMA that applies E4M3
 *     scales per 16 elements.
 *   FP16 Q, K, V (16-bit path, INT8 and FP16 paragraph): the values rounded
 *     to nearest-even half precision; written only when with16 = 1.
 *   MXFP4 Q, K (32-channel blocks) and V (32 key slots per channel), written
 *     instead of NVFP4 when fmt4 = DA2_FMT4_MXFP4: k = floor(log2 amax_G) - 2
 *     clamped to [-127, 127] (-127 for an all-zero block), e =
 *     E2M1_rne(x * 2^-k) (exact scaling), stored as 4-bit codes with the
 *     E8M0 byte k + 127.
 * Casts round to nearest even and saturate; padding slots encode to zero.
 *   Q, K, V  device [B,H,N,d] per *qkv; stats from da2_draft_map (this call
 *            fills entries 2.. : max|V| and the per-channel max|V_c|)
 *   with16   0 or 1: also write the 16-bit sections [10..12] of ops. A
 *            da2_mixed_attn call whose lists hold 16-bit blocks needs them.
 *   fmt4     da2_fmt4: NVFP4 writes sections [0..2], MXFP4 sections
 *            [13..15]; da2_mixed_attn must be called with the same fmt4.
 *            The call writes the tag (0xDA200000 | DA2_OPS_LAYOUT_VERSION << 8
 *            | with16 << 4 | fmt4) into word 3 of each head's g entry, which
 *            da2_mixed_attn checks.
 *   ops      device out of ops_bytes bytes, at least ops_bytes of
 *            da2_sizes(p, scope, fmt4, with16) (section offsets:
 *            da2_ops_offsets(p, fmt4, with16))
 * Errors: INVALID_ARG for with16 or fmt4 out of range, misaligned inputs, or
 * ops_bytes below the size the (fmt4, with16) sections need.                */
int32_t da2_prep_operands(const void* Q, const void* K, const void* V, const da2_tensor* qkv,
                          const int32_t* layout, const da2_problem* p, int32_t with16, int32_t fmt4,
                          void* stats, void* ops, int64_t ops_bytes, void* ws, int64_t ws_bytes,
                          void* stream);

/* Offsets (bytes) inside ops of the 16 sections, for a run with (fmt4,
 * with16); -1 for a section such a run neither writes nor reads. The buffer
 * holds, in this order: the 8-bit sections and the scales [3..9], the 4-bit
 * encoding in use ([0..2] for NVFP4, [13..15] for MXFP4), then the 16-bit
 * sections [10..12] when with16 = 1 (so no other offset depends on with16).
 * Each section is [B*H][R][...] with one 64-slot block per R; lane = 0..63,
 * g = lane/32, r = lane%32, NS = d/16, NT = d/32; "fragment" means the
 * 16-byte-per-lane operand of a gfx950 32x32 MFMA:
 *   [0] Q4, [1] K4, [2] V4  packed NVFP4, 36 d bytes per block: 32 d bytes of
 *        E2M1 codes (code e of a dword in nibble e, sign bit 3), then 4 d bytes
 *        of E4M3 scale codes. Ordered by the attention thread (wave w = 0,1,
 *        lane) that decodes them into the fp16 fragments
 *          Q: [qt:2][s:NS][lane][8] = sigma*e of Q[slot 32qt + r][16s + 8g + e]
 *          K: [j:2][s:NS][lane][8]  = sigma*e of K[kappa(j, r)][16s + 8g + e]
 *          V: [t:NT][s:4][lane][8]  = sigma*e of V[32(s/2)+16g+8(s%2)+e][32t + r]:
 *        codes: dword (w*64 + lane)*NS + f holds the 8 codes of fragment f of
 *          that thread: Q, K fragment (w, s = f); V fragment (t = w*NT/2 + f/4,
 *          s = f%4);
 *        scales: Q, K byte 32d + (w*32 + r)*NS + s = sigma of row (w, r),
 *          channel group s; V byte 32d + (w*64 + lane)*NT/2*2 + 2*t2 + h =
 *          sigma of channel 32t + r (t = w*NT/2 + t2), key group 2h + g.
 *   [3] Q8  int8 [qt:2][s:d/32][lane][16] = code of Q[slot 32qt+lane%32][32s+16g+e]
 *   [4] K8  int8 [j:2][s:d/32][lane][16]  = code of K[kappa(j,lane%32)][32s+16g+e]
 *   [5] V8  e4m3 [t:d/32][h:2][lane][16]  = code of V[32h+16g+e][32t+lane%32]
 *   [6] dQ  float32 [B*H][R]   INT8 scale of each query block
 *   [7] dK  float32 [B*H][R]   INT8 scale of each key block
 *   [8] dV  float32 [B*H][d]   E4M3 per-channel scale of V
 *   [9] g   float32 [B*H][4]   (g_Q, g_K, g_V, tag) NVFP4 tensor scales and the
 *            encoding tag (uint32 bits, see da2_prep_operands)
 *   [10] Q16, [11] K16, [12] V16  fp16, the half-precision values of the
 *            16-bit path in the fp16 fragment orders of Q, K, V above
 *   [13] Q4mx, [14] K4mx, [15] V4mx  MXFP4 operands, (d/32 + 1) fragments of
 *            1 KB per block: d/32 data fragments, then one scale fragment.
 *            Code i (0..31) of a lane sits in byte i/2 of the lane's 16 bytes,
 *            low nibble first (sign bit 3).
 *     Q4mx data [qt:2][s:d/64][lane][32 codes] = Q[slot 32qt+lane%32][64s+32g+i]
 *     K4mx data [j:2][s:d/64][lane][32 codes]  = K[kappa_mx(j,lane%32)][64s+32g+i]
 *     V4mx data [t:d/32][lane][32 codes]       = V[32g+i][32t+lane%32]
 *     scale fragment: uint32 [lane][4], word w = 127 + k of the block that
 *     the lane's codes in data fragment w belong to (w = qt*(d/64)+s, j*(d/64)+s
 *     or t); unused words are 0.
 * with kappa(j, r) = 32j + 16((r/4)%2) + 4(r/8) + r%4 (the key permutation
 * that puts each 16-slot group of a query row into one lane, see the operand
 * permutation equation) and kappa_mx(j, r) = 32((r/4)%2) + 16j + 4(r/8) + r%4
 * (the one that puts each 32-slot MXFP4 block of a query row into one lane
 * half). Errors: INVALID_ARG for fmt4 or with16 out of range. */
int32_t da2_ops_offsets(const da2_problem* p, int32_t fmt4, int32_t with16, int64_t* offsets16);

/* Phased mixed-precision attention (phased-execution appendix;
 * precision-state-conversion equation). For each query block a (one
 * workgroup, 64 query slots) the NVFP4 key blocks are processed in ascending
 * order, then the INT8 ones, then the 16-bit ones, sharing fp32 row maxima m,
 * denominator l and numerator U:
 *   s = Qhat Khat^T / sqrt d; m_j = max(m_{j-1}, rowmax_j s); Pt = exp(s - m_j)
 *   4-bit: l += sum Pt; sigma_P = E4M3(448 max_16 Pt); U += (sigma_P/2688)
 *          E2M1(2688 Pt/sigma_P) Vhat4 (fp16 MFMA on sigma*e operands decoded
 *          from the packed NVFP4 sections)
 *   Enter: U_c /= eta delta_c, l /= eta   (eta = 2^-8.807)
 *   8-bit: int8 MFMA logits; P = 2^((s - m) log2 e + 8.807); l += sum P;
 *          U += E4M3(P) V8 (fp8 MFMA)
 *   Exit:  U_c *= eta delta_c, l *= eta
 *   16-bit: fp16 MFMA logits; Pt = exp(s - m); l += sum Pt; U += fp16(Pt) V16
 *   O = U / l (0 if no retained block)
 * and the rows are written to token order through slot2tok. With fmt4 =
 * DA2_FMT4_MXFP4 the 4-bit phase runs on the MXFP4 sections instead:
 *   4-bit: scaled fp4 MFMA logits; l += sum Pt; per query and 32-slot block
 *          k = floor(log2 max Pt) - 2 (clamped at -127); U += 2^k
 *          E2M1(Pt 2^-k) Vhat4 (scaled fp4 MFMA), already in the common units
 *          (no factor g_V/2688 to restore).
 *   ops, lists, layout  device, from the calls above; ops_bytes is the size
 *            of the ops buffer (at least da2_sizes(p, ., fmt4, 0).ops_bytes)
 *   fmt4     da2_fmt4 used by da2_prep_operands for these ops
 *   out      descriptor of O (dtype fp32 or bf16)
 *   O        device out [B,H,N,d]; every token row is written.
 * The kernel checks each head's tag in g word 3 against this version and
 * fmt4, and a row with 16-bit blocks against the tag's with16 bit; a row
 * that fails is written as zeros and the failure ORed into lists meta word 1
 * (DA2_ATTN_ERR_*), so a mismatch is detectable after the stream completes.
 * Errors: INVALID_ARG for fmt4 out of range, a bad descriptor or an ops
 * buffer smaller than the sections of a run without the 16-bit path.       */
int32_t da2_mixed_attn(const void* ops, int64_t ops_bytes, const void* lists, const int32_t* layout,
                       const da2_problem* p, int32_t fmt4, const da2_tensor* out, void* O,
                       void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DA2_H */
