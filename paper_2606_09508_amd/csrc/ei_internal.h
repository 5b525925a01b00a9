// Internal declarations shared by the HIP translation units of
// libentropyinfer.so: device helpers and the host-side launchers that the
// C ABI layer (ei_api.hip) calls after validating its arguments.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ei {

constexpr int kHeadDim = 128;
constexpr int kWave = 64;

// ----------------------------------------------------------------------------
// Device helpers
// ----------------------------------------------------------------------------

// The two bf16 halves of a 32-bit word, widened exactly to fp32.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float wave_max_f32(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// Max over the 64 lanes: butterflies within rows of 16 lanes by DPP, then two
// cross-row exchanges.
#define EI_DPP_MOV(v, ctrl) \
  __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, (v)), (ctrl), 0xF, 0xF, false))
__device__ __forceinline__ float wave_max_f32_dpp(float v) {
  v = fmaxf(v, EI_DPP_MOV(v, 0xB1));    // quad_perm [1,0,3,2]
  v = fmaxf(v, EI_DPP_MOV(v, 0x4E));    // quad_perm [2,3,0,1]
  v = fmaxf(v, EI_DPP_MOV(v, 0x141));   // row_half_mirror
  v = fmaxf(v, EI_DPP_MOV(v, 0x140));   // row_mirror
  v = fmaxf(v, __shfl_xor(v, 16));
  v = fmaxf(v, __shfl_xor(v, 32));
  return v;
}

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    uint32_t t = __shfl_xor(v, o);
    v = t > v ? t : v;
  }
  return v;
}

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    uint32_t t = __shfl_xor(v, o);
    v = t < v ? t : v;
  }
  return v;
}

__device__ __forceinline__ int popc64(uint64_t m) { return __popcll(m); }

// Wave-wide primitives without LDS round trips: DPP within rows of 16 lanes,
// v_readlane across rows.
#define EI_DPP_U32(v, ctrl, rmask, bctrl) \
  ((uint32_t)__builtin_amdgcn_update_dpp(0, (int)(v), (ctrl), (rmask), 0xF, (bctrl)))
__device__ __forceinline__ uint32_t rl_u32(uint32_t v, int l) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, l);
}
__device__ __forceinline__ uint32_t wave_max_u32_f(uint32_t v) {
  uint32_t t;
  t = EI_DPP_U32(v, 0xB1, 0xF, false); v = t > v ? t : v;    // quad_perm [1,0,3,2]
  t = EI_DPP_U32(v, 0x4E, 0xF, false); v = t > v ? t : v;    // quad_perm [2,3,0,1]
  t = EI_DPP_U32(v, 0x141, 0xF, false); v = t > v ? t : v;   // row_half_mirror
  t = EI_DPP_U32(v, 0x140, 0xF, false); v = t > v ? t : v;   // row_mirror
  const uint32_t a = rl_u32(v, 0), b = rl_u32(v, 16), c = rl_u32(v, 32), d = rl_u32(v, 48);
  const uint32_t ab = a > b ? a : b, cd = c > d ? c : d;
  return ab > cd ? ab : cd;
}
__device__ __forceinline__ uint32_t wave_min_u32_f(uint32_t v) {
  uint32_t t;
  t = EI_DPP_U32(v, 0xB1, 0xF, false); v = t < v ? t : v;
  t = EI_DPP_U32(v, 0x4E, 0xF, false); v = t < v ? t : v;
  t = EI_DPP_U32(v, 0x141, 0xF, false); v = t < v ? t : v;
  t = EI_DPP_U32(v, 0x140, 0xF, false); v = t < v ? t : v;
  const uint32_t a = rl_u32(v, 0), b = rl_u32(v, 16), c = rl_u32(v, 32), d = rl_u32(v, 48);
  const uint32_t ab = a < b ? a : b, cd = c < d ? c : d;
  return ab < cd ? ab : cd;
}
// Inclusive prefix sum over the 64 lanes (lanes without a source add 0).
__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t x) {
  x += EI_DPP_U32(x, 0x111, 0xF, true);   // row_shr:1
  x += EI_DPP_U32(x, 0x112, 0xF, true);   // row_shr:2
  x += EI_DPP_U32(x, 0x114, 0xF, true);   // row_shr:4
  x += EI_DPP_U32(x, 0x118, 0xF, true);   // row_shr:8
  x += EI_DPP_U32(x, 0x142, 0xA, true);   // row_bcast:15 into rows 1, 3
  x += EI_DPP_U32(x, 0x143, 0xC, true);   // row_bcast:31 into rows 2, 3
  return x;
}


// ----------------------------------------------------------------------------
// Host launchers (arguments already validated; B, N > 0)
// ----------------------------------------------------------------------------

struct ProbeShape {
  int B, Hq, Hkv, N, Ls, Lb, CS, CB, r;
};

// Workspace of the probe: the pooled query and key vectors' limb records,
// residual parts and scales (layout in ei_probe.hip), 256-byte aligned parts.
size_t probe_workspace_bytes(const ProbeShape& s);
// Whether the probe kernels support the shape (every validated shape).
bool probe_supported(const ProbeShape& s);

hipError_t launch_probe(const uint16_t* q, const uint16_t* k, const ProbeShape& s,
                        double probe_scale, float* log_scores, float* entropy, void* workspace,
                        hipStream_t stream);

struct SelectShape {
  int B, Hq, N, Ls, Lb, CS, CB, r, kmax;
  float e_t;
  double alpha, delta_t;
  int Bh, mult;
  int mode;   // ei_classify_mode
  int G;      // query heads per KV head
};

bool select_supported(const SelectShape& s);

hipError_t launch_select(const float* log_scores, const float* entropy, const SelectShape& s,
                         uint8_t* rigid, int32_t* budget_blocks, int32_t* block_idx,
                         int32_t* block_cnt, hipStream_t stream);
// Classification and budgets only (the first kernel of launch_select).
hipError_t launch_budget(const float* entropy, const SelectShape& s, uint8_t* rigid,
                         int32_t* budget_blocks, hipStream_t stream);

// Fused probe -> select (Algorithms 1-3 and the top-k, without ln A in
// memory): workspace of probe_select_workspace_bytes (the probe's records
// plus 64 bytes per (b, h, s)); supported while every past-block row fits the
// LDS rows of the second scores kernel ((C_S - 1) r <= 2048).
size_t probe_select_workspace_bytes(const ProbeShape& s);
bool probe_select_supported(const ProbeShape& s);
hipError_t launch_probe_select(const uint16_t* q, const uint16_t* k, const ProbeShape& s,
                               double probe_scale, const SelectShape& ss, float* entropy,
                               uint8_t* rigid, int32_t* budget_blocks, int32_t* block_idx,
                               int32_t* block_cnt, void* workspace, hipStream_t stream);

struct AttnShape {
  int B, Hq, Hkv, N, Ls, Lb, CS, CB, kmax;
  float softmax_scale;
};

enum AttnMode { kSparse = 0, kDenseCausal = 1, kDenseFull = 2 };

// GQA-union tiles (two query heads of a KV group per workgroup): limits of
// the merged list held in LDS.
constexpr int kUnionMaxList = 128;     // kmax
constexpr int kUnionMaxBlocks = 8192;  // C_B
bool attention_union_supported(const AttnShape& s);
hipError_t launch_attention_union(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                  const AttnShape& s, const int32_t* block_idx,
                                  const int32_t* block_cnt, uint16_t* o, hipStream_t stream);

// sched_ws: the sparse kernel's scheduling workspace (kAttnSchedBytes, 4-byte
// aligned) for its persistent grid, or null for the static grid.
constexpr size_t kAttnSchedBytes = 256;
hipError_t launch_attention(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                            const AttnShape& s, AttnMode mode, const int32_t* block_idx,
                            const int32_t* block_cnt, uint16_t* o, void* sched_ws,
                            hipStream_t stream);

}  // namespace ei
