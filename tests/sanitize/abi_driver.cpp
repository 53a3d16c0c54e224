// Host-side exercise of the C ABI for AddressSanitizer / UndefinedBehavior-
// Sanitizer builds (tests/test_host_sanitizers.py): every argument check of
// every entry point, the workspace-size planning over many shapes, the
// canonical converters on random contents, and the status, debug and timing
// calls.  The library is built host-only (no device code), so no call may
// reach a kernel launch: every launching call here has an invalid argument.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <random>
#include <vector>

#include "elas.h"

static int g_fail = 0;
#define EXPECT(cond)                                                   \
  do {                                                                 \
    if (!(cond)) {                                                     \
      fprintf(stderr, "FAIL line %d: %s (%s)\n", __LINE__, #cond, elas_last_error()); \
      ++g_fail;                                                        \
    }                                                                  \
  } while (0)

int main() {
  void* A = (void*)0x10000;   // aligned, never dereferenced
  void* U = (void*)0x10008;   // misaligned
  uint16_t* a = (uint16_t*)A;
  uint8_t* am = (uint8_t*)A;
  float* af = (float*)A;

  for (int c = -1; c <= 7; ++c) EXPECT(elas_status_string(c) != nullptr);
  EXPECT(elas_vals_ld(5464) == 2752 && elas_meta_ld(5464) == 688 && elas_vals_ld(0) == 0 && elas_meta_ld(-5) == 0);

  // sparsify
  EXPECT(elas_sparsify_24(a, 4, 64, 7u, a, am, nullptr) == ELAS_ERR_FLAGS);
  EXPECT(elas_sparsify_24(a, -1, 64, 0, a, am, nullptr) == ELAS_ERR_SHAPE);
  EXPECT(elas_sparsify_24(a, 4, 12, 0, a, am, nullptr) == ELAS_ERR_SHAPE);
  EXPECT(elas_sparsify_24(a, 4, 0, 0, a, am, nullptr) == ELAS_ERR_SHAPE);
  EXPECT(elas_sparsify_24(a, (int64_t)1 << 40, 64, 0, a, am, nullptr) == ELAS_ERR_SHAPE);
  EXPECT(elas_sparsify_24(nullptr, 4, 64, 0, a, am, nullptr) == ELAS_ERR_NULL);
  EXPECT(elas_sparsify_24(a, 4, 64, 0, (uint16_t*)U, am, nullptr) == ELAS_ERR_ALIGN);
  EXPECT(elas_sparsify_24(nullptr, 0, 64, 0, nullptr, nullptr, nullptr) == ELAS_OK);

  // spmm
  EXPECT(elas_spmm_24(a, am, 4, 64, a, 32, 2, a, A, 1 << 20, nullptr) == ELAS_ERR_FLAGS);
  EXPECT(elas_spmm_24(a, am, 4, 70000, a, 32, ELAS_B_NK, a, A, 1 << 20, nullptr) == ELAS_ERR_SHAPE);
  EXPECT(elas_spmm_24(a, am, 4, 64, a, 12, ELAS_B_NK, a, A, 1 << 20, nullptr) == ELAS_ERR_SHAPE);
  EXPECT(elas_spmm_24(a, nullptr, 4, 64, a, 32, ELAS_B_NK, a, A, 1 << 20, nullptr) == ELAS_ERR_NULL);
  EXPECT(elas_spmm_24(a, am, 4, 64, a, 32, ELAS_B_KN, a, A, 16, nullptr) == ELAS_ERR_WORKSPACE);
  EXPECT(elas_spmm_24(a, am, 4, 64, a, 32, ELAS_B_KN, a, U, 1 << 20, nullptr) == ELAS_ERR_ALIGN);
  EXPECT(elas_spmm_24(nullptr, nullptr, 0, 64, nullptr, 32, ELAS_B_KN, nullptr, nullptr, 0, nullptr) == ELAS_OK);

  // forward
  EXPECT(elas_lowrank_ffn_fwd(a, a, a, a, a, 8, 64, 64, 16, 64u, a, a, a, am, a, A, 1 << 30, nullptr) == ELAS_ERR_FLAGS);
  EXPECT(elas_lowrank_ffn_fwd(a, a, a, a, a, 8, 64, 64, 16, ELAS_FWD_FUSED | ELAS_FWD_UNFUSED, a, a, a, am, a, A, 1 << 30,
                              nullptr) == ELAS_ERR_FLAGS);
  EXPECT(elas_lowrank_ffn_fwd(a, a, a, a, a, 8, 64, 64, 16, ELAS_FWD_FUSED | ELAS_MODE_DENSE, a, a, a, am, a, A, 1 << 30,
                              nullptr) == ELAS_ERR_FLAGS);
  EXPECT(elas_lowrank_ffn_fwd(a, a, a, a, a, 8, 2048, 5464, 512, ELAS_FWD_FUSED, a, a, a, am, a, A, 1 << 30, nullptr) ==
         ELAS_ERR_SHAPE);
  EXPECT(elas_lowrank_ffn_fwd(a, a, a, a, a, 8, 60, 64, 16, 0, a, a, a, am, a, A, 1 << 30, nullptr) == ELAS_ERR_SHAPE);
  EXPECT(elas_lowrank_ffn_fwd(a, a, a, a, a, 8, 64, 65544, 16, 0, a, a, a, am, a, A, 1 << 30, nullptr) == ELAS_ERR_SHAPE);
  EXPECT(elas_lowrank_ffn_fwd(a, a, a, a, a, -2, 64, 64, 16, 0, a, a, a, am, a, A, 1 << 30, nullptr) == ELAS_ERR_SHAPE);
  EXPECT(elas_lowrank_ffn_fwd(a, a, nullptr, a, a, 8, 64, 64, 16, 0, a, a, a, am, a, A, 1 << 30, nullptr) == ELAS_ERR_NULL);
  EXPECT(elas_lowrank_ffn_fwd(a, a, a, a, a, 8, 64, 64, 16, 0, a, a, a, nullptr, a, A, 1 << 30, nullptr) == ELAS_ERR_NULL);
  EXPECT(elas_lowrank_ffn_fwd(a, a, a, a, a, 8, 64, 64, 16, 0, a, (uint16_t*)U, a, am, a, A, 1 << 30, nullptr) ==
         ELAS_ERR_ALIGN);
  EXPECT(elas_lowrank_ffn_fwd(a, a, a, a, a, 300, 2048, 5464, 512, 0, a, a, a, am, a, A, 64, nullptr) ==
         ELAS_ERR_WORKSPACE);
  EXPECT(elas_lowrank_ffn_fwd(nullptr, nullptr, nullptr, nullptr, nullptr, 0, 64, 64, 16, 0, nullptr, nullptr, nullptr,
                              nullptr, nullptr, nullptr, 0, nullptr) == ELAS_OK);
  // the no-allocation forward: arguments, and shapes beyond its static scratch
  EXPECT(elas_noalloc_scratch_bytes() == ELAS_NOALLOC_SCRATCH_BYTES);
  EXPECT(elas_lowrank_ffn_fwd_noalloc(a, a, a, a, a, 8, 64, 64, 16, 64u, a, a, a, am, a, nullptr) == ELAS_ERR_FLAGS);
  EXPECT(elas_lowrank_ffn_fwd_noalloc(a, a, a, a, a, 1024, 65536, 65536, 512, 0, a, a, a, am, a, nullptr) ==
         ELAS_ERR_WORKSPACE);
  EXPECT(elas_lowrank_ffn_fwd_noalloc(a, nullptr, a, a, a, 8, 64, 64, 16, 0, a, a, a, am, a, nullptr) == ELAS_ERR_NULL);

  // backward
  EXPECT(elas_lowrank_ffn_bwd(a, a, a, a, a, a, 8, 64, 64, 16, ELAS_MODE_DENSE | ELAS_BWD_STE, a, a, am, a, a, af, af, af,
                              af, A, 1 << 30, nullptr) == ELAS_ERR_FLAGS);
  EXPECT(elas_lowrank_ffn_bwd(a, a, a, a, a, a, 8, 64, 64, 16, 16u, a, a, am, a, a, af, af, af, af, A, 1 << 30, nullptr) ==
         ELAS_ERR_FLAGS);
  EXPECT(elas_lowrank_ffn_bwd(a, a, a, a, a, a, 8, 64, 64, 12, 0, a, a, am, a, a, af, af, af, af, A, 1 << 30, nullptr) ==
         ELAS_ERR_SHAPE);
  EXPECT(elas_lowrank_ffn_bwd(a, a, a, a, a, a, 8, 64, 64, 16, 0, a, a, nullptr, a, a, af, af, af, af, A, 1 << 30,
                              nullptr) == ELAS_ERR_NULL);
  EXPECT(elas_lowrank_ffn_bwd(a, a, a, a, a, a, 8, 64, 64, 16, 0, a, a, am, a, a, af, af, nullptr, af, A, 1 << 30,
                              nullptr) == ELAS_ERR_NULL);
  EXPECT(elas_lowrank_ffn_bwd(a, a, a, a, a, a, 4096, 2048, 5464, 512, 0, a, a, am, a, a, af, af, af, af, A, 1024,
                              nullptr) == ELAS_ERR_WORKSPACE);
  EXPECT(elas_lowrank_ffn_bwd(nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0, 64, 64, 16, 0, nullptr, nullptr,
                              nullptr, nullptr, nullptr, nullptr, af, af, af, A, 0, nullptr) == ELAS_ERR_NULL);

  // full-rank forward
  EXPECT(elas_fullrank_ffn_fwd(a, a, a, 8, 64, 20, a, a, nullptr) == ELAS_ERR_SHAPE);
  EXPECT(elas_fullrank_ffn_fwd(a, nullptr, a, 8, 64, 64, a, a, nullptr) == ELAS_ERR_NULL);

  // workspace planning over many shapes and modes (small-T split-K, stream-K, dense, STE, AB factors)
  const int64_t Ts[] = {0, 1, 31, 255, 256, 257, 1000, 2048, 4096, 16417, 65536, 262144};
  const int64_t shapes[][3] = {{512, 1376, 128}, {768, 2048, 256}, {1024, 2736, 256}, {2048, 5464, 512},
                               {8, 8, 8}, {65536, 64, 8}, {64, 65536, 16}};
  size_t sum = 0;
  for (const auto& sh : shapes)
    for (int64_t T : Ts)
      for (uint32_t f : {0u, (uint32_t)ELAS_MODE_DENSE, (uint32_t)ELAS_FACTORS_AB}) {
        const size_t wf = elas_lowrank_ffn_fwd_workspace_bytes(T, sh[0], sh[1], sh[2], f);
        const size_t wb = elas_lowrank_ffn_bwd_workspace_bytes(T, sh[0], sh[1], sh[2], f == ELAS_FACTORS_AB ? ELAS_BWD_STE : f);
        EXPECT(wf % 256 == 0 && wb % 256 == 0);
        sum += wf + wb;
      }
  EXPECT(sum > 0);
  EXPECT(elas_spmm_24_workspace_bytes(10, 64, 32, ELAS_B_NK) == 0 && elas_spmm_24_workspace_bytes(10, 64, 32, ELAS_B_KN) >= 4096);

  // canonical converters against the layout formula, random contents
  std::mt19937 rng(5);
  for (int64_t M : {1, 255, 256, 600}) {
    for (int64_t N : {8, 64, 200, 5464}) {
      const int64_t ldv = elas_vals_ld(N), ldm = elas_meta_ld(N);
      std::vector<uint16_t> tv(M * ldv), cv(M * (N / 2));
      std::vector<uint8_t> tm(M * ldm), cm(M * (N / 8));
      for (auto& x : tv) x = (uint16_t)rng();
      for (auto& x : tm) x = (uint8_t)rng();
      EXPECT(elas_vals_to_canonical(tv.data(), M, N, cv.data()) == ELAS_OK);
      EXPECT(elas_meta_to_canonical(tm.data(), M, N, cm.data()) == ELAS_OK);
      for (int64_t i = 0; i < M; ++i) {
        const int64_t b = i / 256, R = M - b * 256 < 256 ? M - b * 256 : 256;
        for (int64_t j = 0; j < N / 2; ++j)
          EXPECT(cv[i * (N / 2) + j] == tv[b * 256 * ldv + (j / 32) * R * 32 + (i % 256) * 32 + j % 32]);
        for (int64_t j = 0; j < N / 8; ++j)
          EXPECT(cm[i * (N / 8) + j] == tm[b * 256 * ldm + (j / 8) * R * 8 + (i % 256) * 8 + j % 8]);
      }
    }
  }
  EXPECT(elas_meta_to_canonical(nullptr, 3, 64, nullptr) == ELAS_ERR_NULL);
  EXPECT(elas_vals_to_canonical(a, 3, 12, a) == ELAS_ERR_SHAPE);

  // debug and timing switches (no launches recorded)
  const int prev = elas_debug_sync(-1);
  EXPECT(elas_debug_sync(1) == prev && elas_debug_sync(0) == 1 && elas_debug_sync(prev) == 0);
  EXPECT(elas_timing_enable(1) == ELAS_OK && elas_timing_only("k1_up_gemm") == ELAS_OK && elas_timing_only(nullptr) == ELAS_OK);
  EXPECT(elas_timing_collect() == 0 && elas_timing_entry(0, nullptr, 0, nullptr, nullptr) == ELAS_ERR_SHAPE);
  EXPECT(elas_timing_enable(0) == ELAS_OK);

  printf("abi driver: %d failures\n", g_fail);
  return g_fail ? 1 : 0;
}
