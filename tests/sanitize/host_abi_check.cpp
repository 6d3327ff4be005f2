// Host-side exercise of libda2 under AddressSanitizer and UndefinedBehavior-
// Sanitizer (test infrastructure, CPU only): every size, offset and layout
// query on valid and invalid problems, the ragged and tiled layouts of many
// grids, and every argument error of the compute entry points. Compute calls
// are made only with arguments that validation rejects, so no kernel is ever
// launched. Exits 0 when every returned status is the expected one.
#include <cstdint>
#include <cstdio>
#include <vector>

#include "../../include/da2.h"

static int failures = 0;
#define EXPECT(cond)                                                  \
  do {                                                                \
    if (!(cond)) {                                                    \
      std::fprintf(stderr, "%s:%d: failed: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                     \
    }                                                                 \
  } while (0)

static da2_problem P(int B, int H, int d, int T, int Hg, int Wg, int part) { return da2_problem{B, H, d, T, Hg, Wg, part}; }

int main() {
  for (int s = -6; s <= 2; ++s) EXPECT(da2_status_string(s) != nullptr);
  EXPECT(da2_ops_layout_version() == DA2_OPS_LAYOUT_VERSION);
  const da2_problem good[] = {P(1, 2, 64, 2, 16, 16, 0), P(1, 12, 128, 21, 30, 52, 0), P(1, 12, 128, 21, 30, 52, 1),
                              P(2, 3, 128, 3, 13, 21, 1), P(1, 1, 64, 4, 1, 1, 0), P(1, 2, 64, 3, 1, 5, 1),
                              P(1, 56, 128, 31, 42, 84, 1), P(1, 1, 64, 1, 2, 100, 1), P(1, 1, 64, 1, 100, 2, 1),
                              P(1, 1, 64, 1, 33, 7, 1)};
  for (const auto& p : good) {
    for (int scope = 0; scope < 2; ++scope)
      for (int fmt4 = 0; fmt4 < 2; ++fmt4)
        for (int w16 = 0; w16 < 2; ++w16) {
          da2_sizes_t sz;
          EXPECT(da2_sizes(&p, scope, fmt4, w16, &sz) == DA2_OK);
          int64_t off[16];
          EXPECT(da2_ops_offsets(&p, fmt4, w16, off) == DA2_OK);
          for (int i = 0; i < 16; ++i) EXPECT(off[i] < sz.ops_bytes);
        }
    da2_sizes_t sz;
    EXPECT(da2_sizes(&p, 0, 0, 0, &sz) == DA2_OK);
    int64_t lo[4], wo[7];
    EXPECT(da2_lists_offsets(&p, lo) == DA2_OK);
    EXPECT(da2_ws_draft_offsets(&p, wo) == DA2_OK);
    std::vector<int32_t> L(sz.layout_bytes / 4);
    EXPECT(da2_layout_build(&p, L.data(), (int64_t)L.size()) == DA2_OK);
    EXPECT(da2_layout_build(&p, L.data(), (int64_t)L.size() - 1) == DA2_ERR_INVALID_ARG);
    // every token has a slot and every valid slot a token
    const int64_t R = sz.R, Npad = sz.Npad, N = (int64_t)p.T * p.Hg * p.Wg;
    for (int64_t t = 0; t < N; ++t) EXPECT(L[R + L[R + Npad + t]] == t);
  }
  const da2_problem bad[] = {P(0, 1, 64, 1, 8, 8, 0), P(1, 1, 128, 1, 0, 8, 0), P(1, 1, 128, -1, 8, 8, 0),
                             P(1, 1, 64, 1, 8, 8, 2), P(1, 1, 64, 2000, 80, 80, 0), P(2, 16384, 64, 1, 8, 8, 0)};
  da2_sizes_t sz;
  for (const auto& p : bad) EXPECT(da2_sizes(&p, 0, 0, 0, &sz) == DA2_ERR_INVALID_ARG);
  const da2_problem d96 = P(1, 1, 96, 1, 8, 8, 0);
  EXPECT(da2_sizes(&d96, 0, 0, 0, &sz) == DA2_ERR_UNSUPPORTED);
  EXPECT(da2_sizes(nullptr, 0, 0, 0, &sz) == DA2_ERR_INVALID_ARG);
  EXPECT(da2_sizes(&good[0], 0, 2, 0, &sz) == DA2_ERR_INVALID_ARG);
  EXPECT(da2_sizes(&good[0], 0, 0, 2, &sz) == DA2_ERR_INVALID_ARG);
  EXPECT(da2_sizes(&good[0], 5, 0, 0, &sz) == DA2_ERR_INVALID_ARG);

  // compute entry points: arguments that validation rejects before any GPU call
  const da2_problem& mid = good[1];
  EXPECT(da2_sizes(&mid, 0, 0, 0, &sz) == DA2_OK);
  void* fake = reinterpret_cast<void*>(0x1000);
  da2_tensor t{12ll * 32760 * 128, 32760ll * 128, 128, DA2_BF16, 0};
  da2_tensor bad_t{12ll * 32760 * 128, 32760ll * 128, 64, DA2_BF16, 0};
  const int32_t* lay = reinterpret_cast<const int32_t*>(fake);
  EXPECT(da2_draft_map(nullptr, fake, &t, lay, &mid, 0.2, (float*)fake, fake, fake, sz.ws_draft_bytes, nullptr) ==
         DA2_ERR_INVALID_ARG);
  EXPECT(da2_draft_map(fake, fake, &t, lay, &mid, 1.5, (float*)fake, fake, fake, sz.ws_draft_bytes, nullptr) ==
         DA2_ERR_INVALID_ARG);
  EXPECT(da2_draft_map(fake, fake, &bad_t, lay, &mid, 0.2, (float*)fake, fake, fake, sz.ws_draft_bytes, nullptr) ==
         DA2_ERR_INVALID_ARG);
  EXPECT(da2_draft_map(fake, fake, &t, lay, &mid, 0.2, (float*)fake, fake, fake, sz.ws_draft_bytes - 1, nullptr) ==
         DA2_ERR_WORKSPACE);
  uint8_t* cls = reinterpret_cast<uint8_t*>(fake);
  EXPECT(da2_rank_assign((float*)fake, &mid, 0, 60, 50, 100, 0, cls, fake, fake, sz.ws_rank_bytes, nullptr) ==
         DA2_ERR_INVALID_ARG);
  EXPECT(da2_rank_assign((float*)fake, &mid, 0, 10, 30, 100, 0, cls, fake, fake, sz.ws_rank_bytes - 1, nullptr) ==
         DA2_ERR_WORKSPACE);
  EXPECT(da2_rank_assign_noalloc((float*)fake, &mid, 0, 10, 30, 0, 0, cls, fake, nullptr) == DA2_ERR_INVALID_ARG);
  const da2_problem many = P(1, 128, 128, 21, 30, 52, 0);
  EXPECT(da2_rank_assign_noalloc((float*)fake, &many, 0, 10, 30, 100, 0, cls, fake, nullptr) == DA2_ERR_WORKSPACE);
  EXPECT(da2_prep_operands(fake, fake, fake, &t, lay, &mid, 2, 0, fake, fake, 1ll << 40, nullptr, 0, nullptr) ==
         DA2_ERR_INVALID_ARG);
  EXPECT(da2_prep_operands(fake, fake, fake, &t, lay, &mid, 0, 0, fake, fake, sz.ops_bytes - 1, nullptr, 0, nullptr) ==
         DA2_ERR_INVALID_ARG);
  EXPECT(da2_mixed_attn(fake, sz.ops_bytes - 1, fake, lay, &mid, 0, &t, fake, nullptr) == DA2_ERR_INVALID_ARG);
  EXPECT(da2_mixed_attn(fake, sz.ops_bytes, fake, lay, &mid, 3, &t, fake, nullptr) == DA2_ERR_INVALID_ARG);
  if (failures) std::fprintf(stderr, "%d failures\n", failures);
  else std::printf("host ABI checks passed\n");
  return failures ? 1 : 0;
}
