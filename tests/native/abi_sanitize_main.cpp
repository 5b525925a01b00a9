// Drives the host side of libentropyinfer's C ABI (argument checks, size
// helpers, status strings) in a build with AddressSanitizer and
// UndefinedBehaviorSanitizer on host code.  Every call below is rejected
// (or is empty) before any launch, so no GPU is needed and no fake pointer is
// dereferenced; any out-of-bounds access or undefined operation (an integer
// overflow in a size computation, say) aborts the program.
#include <climits>
#include <initializer_list>
#include <cmath>
#include <cstdio>
#include <cstring>

#include "entropyinfer.h"

static int failures = 0;
#define EXPECT(cond)                                         \
  do {                                                       \
    if (!(cond)) {                                           \
      std::printf("FAILED: %s (line %d)\n", #cond, __LINE__); \
      ++failures;                                            \
    }                                                        \
  } while (0)

int main() {
  uint16_t* F16 = reinterpret_cast<uint16_t*>(0x1000);   // never dereferenced
  float* FF = reinterpret_cast<float*>(0x1000);
  int32_t* FI = reinterpret_cast<int32_t*>(0x1000);
  uint8_t* FU = reinterpret_cast<uint8_t*>(0x1000);
  void* FV = reinterpret_cast<void*>(0x1000);

  EXPECT(ei_abi_version() > 0);
  for (int st = -7; st <= 1; ++st) EXPECT(ei_status_str((ei_status)st) != nullptr);

  const ei_tiling t{128, 64};
  const ei_budget_params p{1e-5f, 0.5, 0.4, 2048, 3};
  const ei_dims good{1, 32, 8, 131072, 128};
  EXPECT(ei_num_segments(good, t) == 1024 && ei_num_blocks(good, t) == 2048);
  EXPECT(ei_kmax(t, p) == 98);
  EXPECT(ei_probe_workspace_bytes(good, t) > 0 && ei_prefill_workspace_bytes(good, t) > 0);

  // extreme and invalid sizes: the helpers return 0 / -1 rather than overflow
  const ei_dims huge[] = {{INT_MAX, INT_MAX, 1, INT_MAX, 128}, {1, INT_MAX, INT_MAX, 1 << 30, 128},
                          {-1, 4, 1, 1024, 128},           {1, 4, 0, 1024, 128},
                          {1, 4, 3, 1024, 128},            {1, 4, 1, -5, 128},
                          {1, 4, 1, 1024, 64},             {1, 4, 1, INT_MAX, 128}};
  const ei_tiling tilings[] = {{128, 64}, {0, 64}, {128, 0}, {192, 64}, {128, 96}, {-128, 64},
                               {INT_MAX, 64}, {2048, 128}};
  const ei_budget_params params[] = {p, {1e-5f, 0.5, 0.4, -1, 3}, {1e-5f, 0.5, 0.4, 2048, 0},
                                     {NAN, 0.5, 0.4, 2048, 3}, {1e-5f, NAN, 0.4, 2048, 3},
                                     {1e-5f, 0.5, 0.4, INT_MAX, INT_MAX}};
  size_t sink = 0;
  for (const ei_dims& d : huge)
    for (const ei_tiling& tl : tilings) {
      sink += (size_t)ei_num_segments(d, tl) + (size_t)ei_num_blocks(d, tl);
      sink += ei_probe_workspace_bytes(d, tl) + ei_prefill_workspace_bytes(d, tl);
      sink += ei_probe_select_workspace_bytes(d, tl);
      for (const ei_budget_params& pp : params) sink += (size_t)ei_kmax(tl, pp);
    }
  std::printf("helpers swept (%zu)\n", sink % 7);

  const ei_dims d{1, 4, 1, 1024, 128};
  const int32_t km = ei_kmax(t, p);
  const size_t ws = ei_probe_workspace_bytes(d, t);
  // probe
  EXPECT(ei_entropy_probe(nullptr, F16, d, t, 1.0, FF, FF, FV, ws, nullptr) == EI_ERR_NULL);
  EXPECT(ei_entropy_probe(F16, F16, d, t, 1.0, FF, FF, FV, ws - 1, nullptr) == EI_ERR_WORKSPACE);
  EXPECT(ei_entropy_probe(F16, F16, d, t, 1.0, FF, FF, nullptr, ws, nullptr) == EI_ERR_WORKSPACE);
  for (const ei_dims& dd : huge)
    EXPECT(ei_entropy_probe(F16, F16, dd, t, 1.0, FF, FF, FV, ws, nullptr) < 0);
  for (const ei_tiling& tl : tilings)
    if (tl.seg_len != 128 && tl.seg_len != 2048)
      EXPECT(ei_entropy_probe(F16, F16, d, tl, 1.0, FF, FF, FV, ws, nullptr) < 0);
  EXPECT(ei_entropy_probe(F16, F16, ei_dims{0, 4, 1, 1024, 128}, t, 1.0, FF, FF, FV, ws,
                          nullptr) == EI_OK);
  // selection
  EXPECT(ei_select_blocks(nullptr, FF, d, t, p, km, FU, FI, FI, FI, nullptr) == EI_ERR_NULL);
  EXPECT(ei_select_blocks(FF, FF, d, t, p, km - 1, FU, FI, FI, FI, nullptr) == EI_ERR_SHAPE);
  for (const ei_budget_params& pp : params)
    if (&pp != &params[0] && &pp != &params[5])
      EXPECT(ei_select_blocks(FF, FF, d, t, pp, km, FU, FI, FI, FI, nullptr) < 0);
  for (int mode : {-1, 3, INT_MAX})
    EXPECT(ei_select_blocks_mode(FF, FF, d, t, p, mode, km, FU, FI, FI, FI, nullptr) < 0);
  // fused probe -> select
  const size_t fws = ei_probe_select_workspace_bytes(d, t);
  EXPECT(fws > ws);
  EXPECT(ei_probe_select_fused(F16, F16, d, t, 1.0, p, 0, km, FF, FU, FI, FI, FI, FV, fws - 1,
                               nullptr) == EI_ERR_WORKSPACE);
  EXPECT(ei_probe_select_fused(F16, nullptr, d, t, 1.0, p, 0, km, FF, FU, FI, FI, FI, FV, fws,
                               nullptr) == EI_ERR_NULL);
  EXPECT(ei_probe_select_fused(F16, F16, d, t, 1.0, p, 3, km, FF, FU, FI, FI, FI, FV, fws,
                               nullptr) == EI_ERR_SHAPE);
  EXPECT(ei_probe_select_fused(F16, F16, d, t, NAN, p, 0, km, FF, FU, FI, FI, FI, FV, fws,
                               nullptr) == EI_ERR_SHAPE);
  EXPECT(ei_probe_select_fused(F16, F16, d, t, 1.0, p, 0, km - 1, FF, FU, FI, FI, FI, FV, fws,
                               nullptr) == EI_ERR_SHAPE);
  {
    const ei_dims longer{1, 4, 1, 131072 + 129, 128};   // 2050 past blocks in the last segment
    EXPECT(ei_probe_select_fused(F16, F16, longer, t, 1.0, p, 0, km, FF, FU, FI, FI, FI, FV,
                                 ei_probe_select_workspace_bytes(longer, t),
                                 nullptr) == EI_ERR_UNSUPPORTED);
  }
  for (const ei_dims& dd : huge)
    EXPECT(ei_probe_select_fused(F16, F16, dd, t, 1.0, p, 0, km, FF, FU, FI, FI, FI, FV, fws,
                                 nullptr) < 0);
  // attention
  EXPECT(ei_sparse_prefill_attn(F16, F16, F16, d, t, NAN, FI, FI, km, F16, nullptr, 0,
                                nullptr) == EI_ERR_SHAPE);
  EXPECT(ei_sparse_prefill_attn(F16, F16, F16, d, t, 0.088f, nullptr, FI, km, F16, nullptr, 0,
                                nullptr) == EI_ERR_NULL);
  EXPECT(ei_sparse_prefill_attn(F16, F16, F16, d, t, 0.088f, FI, FI, 0, F16, nullptr, 0,
                                nullptr) < 0);
  EXPECT(ei_sparse_prefill_attn(F16, F16, F16, d, t, 0.088f, FI, FI, km, F16, FV,
                                EI_ATTN_WORKSPACE_BYTES - 1, nullptr) == EI_ERR_WORKSPACE);
  EXPECT(ei_dense_prefill_attn(F16, nullptr, F16, d, 0.088f, 1, F16, nullptr) == EI_ERR_NULL);
  EXPECT(ei_dense_prefill_attn(F16, F16, F16, d, NAN, 1, F16, nullptr) == EI_ERR_SHAPE);
  for (const ei_dims& dd : huge)
    EXPECT(ei_dense_prefill_attn(F16, F16, F16, dd, 0.088f, 1, F16, nullptr) < 0);
  // the one-call path
  const size_t pws = ei_prefill_workspace_bytes(d, t);
  EXPECT(pws == ws + EI_ATTN_WORKSPACE_BYTES);
  EXPECT(ei_entropy_guided_prefill(F16, F16, F16, d, t, 1.0, p, 0, km, 0.088f, FF, FF, FU, FI,
                                   FI, FI, F16, FV, pws - 1, nullptr) == EI_ERR_WORKSPACE);
  EXPECT(ei_entropy_guided_prefill(F16, F16, F16, d, t, 1.0, p, 7, km, 0.088f, FF, FF, FU, FI,
                                   FI, FI, F16, FV, pws, nullptr) == EI_ERR_SHAPE);
  EXPECT(ei_entropy_guided_prefill(F16, F16, nullptr, d, t, 1.0, p, 0, km, 0.088f, FF, FF, FU,
                                   FI, FI, FI, F16, FV, pws, nullptr) == EI_ERR_NULL);
  EXPECT(ei_entropy_guided_prefill_noalloc(F16, F16, F16, ei_dims{1, 64, 8, 262144, 128}, t,
                                           1.0, p, 0, km, 0.088f, FF, FF, FU, FI, FI, FI, F16,
                                           nullptr) == EI_ERR_WORKSPACE);

  // scales: softmax_scale finite and > 0, probe_scale finite
  for (float sc : {0.0f, -0.088f, INFINITY, -INFINITY, NAN}) {
    EXPECT(ei_sparse_prefill_attn(F16, F16, F16, d, t, sc, FI, FI, km, F16, nullptr, 0,
                                  nullptr) == EI_ERR_SHAPE);
    EXPECT(ei_dense_prefill_attn(F16, F16, F16, d, sc, 0, F16, nullptr) == EI_ERR_SHAPE);
    EXPECT(ei_entropy_guided_prefill(F16, F16, F16, d, t, 1.0, p, 0, km, sc, FF, FF, FU, FI, FI,
                                     FI, F16, FV, pws, nullptr) == EI_ERR_SHAPE);
  }
  for (double ps : {(double)INFINITY, (double)NAN})
    EXPECT(ei_entropy_probe(F16, F16, d, t, ps, FF, FF, FV, ws, nullptr) == EI_ERR_SHAPE);

  std::printf("abi sanitized run: %s\n", failures ? "FAILED" : "ok");
  return failures ? 1 : 0;
}
