// Kernel argument blocks and launchers shared by the host library and the
// kernel translation units. Internal to libda2.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/da2.h"

namespace da2 {

// Bytes of one block (64 slots x D channels) of a packed NVFP4 section: the
// E2M1 codes (4 bits per value) and one E4M3 scale byte per 16 values.
constexpr int nv_block_bytes(int D) { return 32 * D + 4 * D; }

struct DraftArgs {
  const void* Q;
  const void* K;
  int64_t sb, sh, sn;
  int dtype;
  int B, H, d, R, Npad;
  const int32_t* layout;
  double lambda;
  float* A;
  uint32_t* stats;
  double *Qbar, *Qmax, *Kbar, *Kmax, *S1, *S2;
  float* blkmax;  // [2][B*H][R]: max |Q| (then |K|) of each block
};

constexpr int kCuts = 3;  // rank cut points: T16, T16+T8, T16+T8+T4

constexpr int kRankCand = 2048;  // candidate keys per (head, cut) the ranking resolves directly

struct RankArgs {
  const float* A;
  int B, H, R;
  int scope;
  int64_t cut[kCuts];      // cumulative quotas per head (head scope) or per row (row scope)
  uint8_t* cls;
  uint16_t* keys;          // lists: [BH*R][R]
  int32_t* counts;         // [BH*R][4] = (n4, n8, n16, 0)
  int32_t* order;          // [BH*R]
  int32_t* meta;           // [8]
  // workspace
  uint32_t* hist;          // [BH][kCuts][2048]
  uint64_t* thr;           // head: [BH][kCuts]; row: [BH*R][kCuts]
  uint64_t* prefix;        // [BH][kCuts]
  int64_t* kleft;          // [BH][kCuts]
  uint64_t* cand;          // [BH][kCuts][kRankCand] keys collected in the third histogram pass
  uint32_t* ccount;        // [BH][kCuts] number collected (> kRankCand: too many, not used)
  int32_t* cost;           // [BH*R]
};

struct PrepArgs {
  const void* Q;
  const void* K;
  const void* V;
  int64_t sb, sh, sn;
  int dtype;
  int B, H, d, R, Npad, N;
  const int32_t* layout;
  uint32_t* stats;
  // ops sections
  uint8_t *Q4, *K4, *V4;  // packed NVFP4 (codes and E4M3 scales)
  int8_t *Q8, *K8;
  uint8_t* V8;
  float *dQ, *dK, *dV, *g;
  _Float16 *Q16, *K16, *V16;  // 16-bit path operands (written when with16)
  uint8_t *Q4mx, *K4mx, *V4mx;  // MXFP4 operands (written instead of Q4/K4/V4 when fmt4 = MXFP4)
  int with16;
  int fmt4;
  uint32_t tag;  // ops_tag(fmt4, with16), written into word 3 of each head's g entry
};

struct AttnArgs {
  const uint8_t *Q4, *K4, *V4;  // packed NVFP4 (codes and E4M3 scales)
  const int8_t *Q8, *K8;
  const uint8_t* V8;
  const float *dQ, *dK, *dV, *g;
  const _Float16 *Q16, *K16, *V16;
  const uint8_t *Q4mx, *K4mx, *V4mx;
  int fmt4;
  uint32_t tag;   // ops_tag(fmt4, 0): expected tag of the operands (the with16 bit is checked per row)
  int has16;      // the ops buffer is large enough to hold the 16-bit sections
  int32_t* meta;  // lists meta area: word 1 collects the error flags of a mismatch
  const uint16_t* keys;
  const int32_t* counts;
  const int32_t* order;
  const int32_t* layout;
  int B, H, d, R, Npad;
  void* O;
  int64_t ob, oh, on;
  int odtype;
};

// Size of the fixed device scratch that da2_rank_assign_noalloc uses instead
// of a caller workspace (8 MiB per device).
constexpr int64_t kRankScratchBytes = 8ll << 20;
// Device address of the current device's scratch array (looked up once per device).
hipError_t rank_scratch_address(void** out);

// Tag that da2_prep_operands writes into word 3 of each head's g entry and
// da2_mixed_attn checks: a fixed marker, the ops layout version, with16 (bit
// 4) and fmt4 (bits 0..3).
constexpr uint32_t kTagMarker = 0xDA200000u;
constexpr uint32_t ops_tag(int fmt4, int with16) {
  return kTagMarker | (static_cast<uint32_t>(DA2_OPS_LAYOUT_VERSION) << 8) | (with16 ? 0x10u : 0u) |
         static_cast<uint32_t>(fmt4);
}

hipError_t launch_draft(const DraftArgs& args, hipStream_t stream);
hipError_t launch_rank(const RankArgs& args, hipStream_t stream);
hipError_t launch_prep(const PrepArgs& args, hipStream_t stream);
hipError_t launch_attn(const AttnArgs& args, hipStream_t stream);

}  // namespace da2
