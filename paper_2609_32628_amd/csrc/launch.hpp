// Kernel argument blocks and launchers shared by the host library and the
// kernel translation units. Internal to libda2.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace da2 {

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
  _Float16 *Q4, *K4, *V4;
  int8_t *Q8, *K8;
  uint8_t* V8;
  float *dQ, *dK, *dV, *g;
  _Float16 *Q16, *K16, *V16;  // 16-bit path operands (written when with16)
  uint8_t *Q4mx, *K4mx, *V4mx;  // MXFP4 operands (written instead of Q4/K4/V4 when fmt4 = MXFP4)
  int with16;
  int fmt4;
};

struct AttnArgs {
  const _Float16 *Q4, *K4, *V4;
  const int8_t *Q8, *K8;
  const uint8_t* V8;
  const float *dQ, *dK, *dV, *g;
  const _Float16 *Q16, *K16, *V16;
  const uint8_t *Q4mx, *K4mx, *V4mx;
  int fmt4;
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

hipError_t launch_draft(const DraftArgs& args, hipStream_t stream);
hipError_t launch_rank(const RankArgs& args, hipStream_t stream);
hipError_t launch_prep(const PrepArgs& args, hipStream_t stream);
hipError_t launch_attn(const AttnArgs& args, hipStream_t stream);

}  // namespace da2
