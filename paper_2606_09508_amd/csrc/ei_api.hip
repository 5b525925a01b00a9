// C ABI of libentropyinfer.so: argument validation on the host, then the
// launches of ei_probe.hip, ei_select.hip and ei_attn.hip.  Nothing is
// launched unless every check passes; no exception crosses the ABI.
#include "../../include/entropyinfer.h"
#include "ei_internal.h"

#include <limits.h>

#include <initializer_list>

namespace {

constexpr int32_t kAbiVersion = 7;
static_assert(EI_ATTN_WORKSPACE_BYTES == ei::kAttnSchedBytes, "attention workspace size");

struct Sizes {
  int64_t B, Hq, Hkv, N, D, CS, CB, r;
};

ei_status check_dims(const ei_dims& d) {
  if (d.batch < 0 || d.seq_len < 0 || d.n_q_heads <= 0 || d.n_kv_heads <= 0 || d.head_dim <= 0)
    return EI_ERR_SHAPE;
  if (d.n_q_heads % d.n_kv_heads) return EI_ERR_SHAPE;
  // element offsets are formed in 64-bit, (batch, head) indices in 32-bit
  if ((int64_t)d.batch * d.n_q_heads > INT_MAX / 2) return EI_ERR_SHAPE;
  // every grid (workgroups per (batch, head, 128-row tile or segment)) fits
  // in 31 bits
  if ((int64_t)d.batch * d.n_q_heads * (((int64_t)d.seq_len + 127) / 128) > INT_MAX)
    return EI_ERR_SHAPE;
  if (d.head_dim != ei::kHeadDim) return EI_ERR_UNSUPPORTED;
  return EI_OK;
}

ei_status check_tiling(const ei_tiling& t) {
  if (t.block_len != 64 && t.block_len != 128) return EI_ERR_UNSUPPORTED;
  if (t.seg_len <= 0 || t.seg_len % 128 || t.seg_len % t.block_len) return EI_ERR_SHAPE;
  return EI_OK;
}

// The attention kernels mask scores to -inf before scaling and take the row
// maximum of the raw scores, which is the maximum of the scaled ones only for
// a positive scale: softmax_scale must be finite and > 0.
bool scale_ok(float s) { return s > 0.0f && s <= 3.402823466e38f; }
// probe_scale multiplies binary64 logits; any finite value (0 and negative
// values included) is meaningful.
bool probe_scale_ok(double s) { return s == s && s - s == 0.0; }

Sizes sizes(const ei_dims& d, const ei_tiling* t) {
  Sizes s{d.batch, d.n_q_heads, d.n_kv_heads, d.seq_len, d.head_dim, 0, 0, 0};
  if (t) {
    s.CS = (s.N + t->seg_len - 1) / t->seg_len;
    s.CB = (s.N + t->block_len - 1) / t->block_len;
    s.r = t->seg_len / t->block_len;
  }
  return s;
}

ei_status check_params(const ei_budget_params& p) {
  if (p.base_budget_tokens < 0 || p.max_budget_mult < 1) return EI_ERR_SHAPE;
  if (!(p.alpha == p.alpha) || !(p.delta_t == p.delta_t)) return EI_ERR_SHAPE;
  if ((int64_t)p.max_budget_mult * p.base_budget_tokens > INT_MAX / 2) return EI_ERR_SHAPE;
  return EI_OK;
}

int32_t kmax_of(const ei_tiling& t, const ei_budget_params& p) {
  return (int32_t)((int64_t)p.max_budget_mult * p.base_budget_tokens / t.block_len +
                   t.seg_len / t.block_len);
}

ei_status from_hip(hipError_t e) { return e == hipSuccess ? EI_OK : EI_ERR_LAUNCH; }

// The kernels move bf16 tensors and the workspace in 16-byte vectors (and by
// LDS DMA), fp32 / int32 arrays in 4-byte words.
bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }
bool aligned16(std::initializer_list<const void*> ps) {
  for (const void* p : ps)
    if (!aligned(p, 16)) return false;
  return true;
}
bool aligned4(std::initializer_list<const void*> ps) {
  for (const void* p : ps)
    if (!aligned(p, 4)) return false;
  return true;
}

}  // namespace

extern "C" {

int32_t ei_abi_version(void) { return kAbiVersion; }

const char* ei_status_str(ei_status status) {
  switch (status) {
    case EI_OK: return "EI_OK";
    case EI_ERR_NULL: return "EI_ERR_NULL: a required pointer is NULL";
    case EI_ERR_SHAPE: return "EI_ERR_SHAPE: inconsistent or out-of-range sizes";
    case EI_ERR_UNSUPPORTED: return "EI_ERR_UNSUPPORTED: valid but not supported by this library";
    case EI_ERR_WORKSPACE: return "EI_ERR_WORKSPACE: workspace missing or too small";
    case EI_ERR_LAUNCH: return "EI_ERR_LAUNCH: a kernel launch failed";
  }
  return "unknown ei_status";
}

int64_t ei_num_segments(ei_dims dims, ei_tiling tiling) {
  if (check_dims(dims) == EI_ERR_SHAPE || check_tiling(tiling) != EI_OK) return -1;
  return sizes(dims, &tiling).CS;
}

int64_t ei_num_blocks(ei_dims dims, ei_tiling tiling) {
  if (check_dims(dims) == EI_ERR_SHAPE || check_tiling(tiling) != EI_OK) return -1;
  return sizes(dims, &tiling).CB;
}

int32_t ei_kmax(ei_tiling tiling, ei_budget_params params) {
  if (check_tiling(tiling) != EI_OK || check_params(params) != EI_OK) return -1;
  return kmax_of(tiling, params);
}

size_t ei_probe_workspace_bytes(ei_dims dims, ei_tiling tiling) {
  if (check_dims(dims) != EI_OK || check_tiling(tiling) != EI_OK) return 0;
  const Sizes z = sizes(dims, &tiling);
  const ei::ProbeShape ps{(int)z.B, (int)z.Hq, (int)z.Hkv, (int)z.N, tiling.seg_len,
                          tiling.block_len, (int)z.CS, (int)z.CB, (int)z.r};
  return ei::probe_workspace_bytes(ps);
}

ei_status ei_entropy_probe(const uint16_t* q, const uint16_t* k, ei_dims dims, ei_tiling tiling,
                           double probe_scale, float* log_scores, float* entropy,
                           void* workspace, size_t workspace_bytes, void* stream) {
  ei_status st = check_dims(dims);
  if (st != EI_OK) return st;
  if ((st = check_tiling(tiling)) != EI_OK) return st;
  if (!probe_scale_ok(probe_scale)) return EI_ERR_SHAPE;
  const Sizes z = sizes(dims, &tiling);
  if (z.B == 0 || z.N == 0) return EI_OK;
  if (!q || !k || !log_scores || !entropy) return EI_ERR_NULL;
  if (!aligned16({q, k}) || !aligned4({log_scores, entropy})) return EI_ERR_UNSUPPORTED;
  const ei::ProbeShape ps{(int)z.B, (int)z.Hq, (int)z.Hkv, (int)z.N, tiling.seg_len,
                          tiling.block_len, (int)z.CS, (int)z.CB, (int)z.r};
  if (!ei::probe_supported(ps)) return EI_ERR_UNSUPPORTED;
  if (!workspace || workspace_bytes < ei::probe_workspace_bytes(ps))
    return EI_ERR_WORKSPACE;
  if (!aligned16({workspace})) return EI_ERR_UNSUPPORTED;
  return from_hip(ei::launch_probe(q, k, ps, probe_scale, log_scores, entropy, workspace,
                                   (hipStream_t)stream));
}

ei_status ei_select_blocks(const float* log_scores, const float* entropy, ei_dims dims,
                           ei_tiling tiling, ei_budget_params params, int32_t kmax,
                           uint8_t* head_is_rigid, int32_t* budget_blocks, int32_t* block_idx,
                           int32_t* block_cnt, void* stream) {
  return ei_select_blocks_mode(log_scores, entropy, dims, tiling, params, EI_CLASSIFY_HEAD,
                               kmax, head_is_rigid, budget_blocks, block_idx, block_cnt, stream);
}

ei_status ei_select_blocks_mode(const float* log_scores, const float* entropy, ei_dims dims,
                                ei_tiling tiling, ei_budget_params params, int32_t mode,
                                int32_t kmax, uint8_t* head_is_rigid, int32_t* budget_blocks,
                                int32_t* block_idx, int32_t* block_cnt, void* stream) {
  if (mode < EI_CLASSIFY_HEAD || mode > EI_CLASSIFY_SEGMENT) return EI_ERR_SHAPE;
  ei_status st = check_dims(dims);
  if (st == EI_ERR_SHAPE) return st;   // head_dim is not read by the selection
  if ((st = check_tiling(tiling)) != EI_OK) return st;
  if ((st = check_params(params)) != EI_OK) return st;
  if (kmax < kmax_of(tiling, params)) return EI_ERR_SHAPE;
  const Sizes z = sizes(dims, &tiling);
  if (z.B == 0 || z.N == 0) return EI_OK;
  if (!log_scores || !entropy || !head_is_rigid || !budget_blocks || !block_idx || !block_cnt)
    return EI_ERR_NULL;
  if (!aligned4({log_scores, entropy, budget_blocks, block_idx, block_cnt}))
    return EI_ERR_UNSUPPORTED;
  const ei::SelectShape ss{(int)z.B, (int)z.Hq, (int)z.N, tiling.seg_len, tiling.block_len,
                           (int)z.CS, (int)z.CB, (int)z.r, kmax, params.entropy_threshold,
                           params.alpha, params.delta_t, params.base_budget_tokens,
                           params.max_budget_mult, (int)mode, (int)(z.Hq / z.Hkv)};
  if (!ei::select_supported(ss)) return EI_ERR_UNSUPPORTED;
  return from_hip(ei::launch_select(log_scores, entropy, ss, head_is_rigid, budget_blocks,
                                    block_idx, block_cnt, (hipStream_t)stream));
}

size_t ei_probe_select_workspace_bytes(ei_dims dims, ei_tiling tiling) {
  if (check_dims(dims) != EI_OK || check_tiling(tiling) != EI_OK) return 0;
  const Sizes z = sizes(dims, &tiling);
  const ei::ProbeShape ps{(int)z.B, (int)z.Hq, (int)z.Hkv, (int)z.N, tiling.seg_len,
                          tiling.block_len, (int)z.CS, (int)z.CB, (int)z.r};
  return ei::probe_select_workspace_bytes(ps);
}

ei_status ei_probe_select_fused(const uint16_t* q, const uint16_t* k, ei_dims dims,
                                ei_tiling tiling, double probe_scale, ei_budget_params params,
                                int32_t mode, int32_t kmax, float* entropy,
                                uint8_t* head_is_rigid, int32_t* budget_blocks,
                                int32_t* block_idx, int32_t* block_cnt, void* workspace,
                                size_t workspace_bytes, void* stream) {
  ei_status st = check_dims(dims);
  if (st != EI_OK) return st;
  if ((st = check_tiling(tiling)) != EI_OK) return st;
  if ((st = check_params(params)) != EI_OK) return st;
  if (mode < EI_CLASSIFY_HEAD || mode > EI_CLASSIFY_SEGMENT) return EI_ERR_SHAPE;
  if (!probe_scale_ok(probe_scale)) return EI_ERR_SHAPE;
  if (kmax < kmax_of(tiling, params)) return EI_ERR_SHAPE;
  const Sizes z = sizes(dims, &tiling);
  if (z.B == 0 || z.N == 0) return EI_OK;
  if (!q || !k || !entropy || !head_is_rigid || !budget_blocks || !block_idx || !block_cnt)
    return EI_ERR_NULL;
  if (!aligned16({q, k}) || !aligned4({entropy, budget_blocks, block_idx, block_cnt}))
    return EI_ERR_UNSUPPORTED;
  const ei::ProbeShape ps{(int)z.B, (int)z.Hq, (int)z.Hkv, (int)z.N, tiling.seg_len,
                          tiling.block_len, (int)z.CS, (int)z.CB, (int)z.r};
  const ei::SelectShape ss{(int)z.B, (int)z.Hq, (int)z.N, tiling.seg_len, tiling.block_len,
                           (int)z.CS, (int)z.CB, (int)z.r, kmax, params.entropy_threshold,
                           params.alpha, params.delta_t, params.base_budget_tokens,
                           params.max_budget_mult, (int)mode, (int)(z.Hq / z.Hkv)};
  if (!ei::probe_supported(ps) || !ei::probe_select_supported(ps)) return EI_ERR_UNSUPPORTED;
  if (!workspace || workspace_bytes < ei::probe_select_workspace_bytes(ps))
    return EI_ERR_WORKSPACE;
  if (!aligned16({workspace})) return EI_ERR_UNSUPPORTED;
  return from_hip(ei::launch_probe_select(q, k, ps, probe_scale, ss, entropy, head_is_rigid,
                                          budget_blocks, block_idx, block_cnt, workspace,
                                          (hipStream_t)stream));
}

ei_status ei_sparse_prefill_attn(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                 ei_dims dims, ei_tiling tiling, float softmax_scale,
                                 const int32_t* block_idx, const int32_t* block_cnt,
                                 int32_t kmax, uint16_t* o, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  ei_status st = check_dims(dims);
  if (st != EI_OK) return st;
  if ((st = check_tiling(tiling)) != EI_OK) return st;
  if (kmax <= 0 || !scale_ok(softmax_scale)) return EI_ERR_SHAPE;
  const Sizes z = sizes(dims, &tiling);
  if (z.B == 0 || z.N == 0) return EI_OK;
  if (!q || !k || !v || !block_idx || !block_cnt || !o) return EI_ERR_NULL;
  if (!aligned16({q, k, v, o}) || !aligned4({block_idx, block_cnt})) return EI_ERR_UNSUPPORTED;
  if (workspace && workspace_bytes < EI_ATTN_WORKSPACE_BYTES) return EI_ERR_WORKSPACE;
  if (workspace && !aligned16({workspace})) return EI_ERR_UNSUPPORTED;
  const ei::AttnShape as{(int)z.B, (int)z.Hq, (int)z.Hkv, (int)z.N, tiling.seg_len,
                         tiling.block_len, (int)z.CS, (int)z.CB, kmax, softmax_scale};
  return from_hip(ei::launch_attention(q, k, v, as, ei::kSparse, block_idx, block_cnt, o,
                                       workspace, (hipStream_t)stream));
}

ei_status ei_sparse_prefill_attn_gqa_union(const uint16_t* q, const uint16_t* k,
                                           const uint16_t* v, ei_dims dims, ei_tiling tiling,
                                           float softmax_scale, const int32_t* block_idx,
                                           const int32_t* block_cnt, int32_t kmax, uint16_t* o,
                                           void* stream) {
  ei_status st = check_dims(dims);
  if (st != EI_OK) return st;
  if ((st = check_tiling(tiling)) != EI_OK) return st;
  if (kmax <= 0 || !scale_ok(softmax_scale)) return EI_ERR_SHAPE;
  const Sizes z = sizes(dims, &tiling);
  if (z.B == 0 || z.N == 0) return EI_OK;
  if (!q || !k || !v || !block_idx || !block_cnt || !o) return EI_ERR_NULL;
  if (!aligned16({q, k, v, o}) || !aligned4({block_idx, block_cnt})) return EI_ERR_UNSUPPORTED;
  const ei::AttnShape as{(int)z.B, (int)z.Hq, (int)z.Hkv, (int)z.N, tiling.seg_len,
                         tiling.block_len, (int)z.CS, (int)z.CB, kmax, softmax_scale};
  if (!ei::attention_union_supported(as)) return EI_ERR_UNSUPPORTED;
  return from_hip(ei::launch_attention_union(q, k, v, as, block_idx, block_cnt, o,
                                             (hipStream_t)stream));
}

size_t ei_prefill_workspace_bytes(ei_dims dims, ei_tiling tiling) {
  // the probe workspace (a multiple of 256 bytes), then the attention's
  // scheduling counters
  const size_t p = ei_probe_workspace_bytes(dims, tiling);
  return p ? p + EI_ATTN_WORKSPACE_BYTES : 0;
}

ei_status ei_entropy_guided_prefill(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                    ei_dims dims, ei_tiling tiling, double probe_scale,
                                    ei_budget_params params, int32_t mode, int32_t kmax,
                                    float softmax_scale, float* log_scores, float* entropy,
                                    uint8_t* head_is_rigid, int32_t* budget_blocks,
                                    int32_t* block_idx, int32_t* block_cnt, uint16_t* o,
                                    void* workspace, size_t workspace_bytes, void* stream) {
  // validate the whole problem as the three calls would
  ei_status st = check_dims(dims);
  if (st != EI_OK) return st;
  if ((st = check_tiling(tiling)) != EI_OK) return st;
  if ((st = check_params(params)) != EI_OK) return st;
  if (mode < EI_CLASSIFY_HEAD || mode > EI_CLASSIFY_SEGMENT) return EI_ERR_SHAPE;
  if (!probe_scale_ok(probe_scale) || !scale_ok(softmax_scale)) return EI_ERR_SHAPE;
  if (kmax < kmax_of(tiling, params)) return EI_ERR_SHAPE;
  const Sizes z = sizes(dims, &tiling);
  if (z.B == 0 || z.N == 0) return EI_OK;
  if (!q || !k || !v || !log_scores || !entropy || !head_is_rigid || !budget_blocks ||
      !block_idx || !block_cnt || !o)
    return EI_ERR_NULL;
  if (!aligned16({q, k, v, o}) ||
      !aligned4({log_scores, entropy, budget_blocks, block_idx, block_cnt}))
    return EI_ERR_UNSUPPORTED;
  const ei::ProbeShape ps{(int)z.B, (int)z.Hq, (int)z.Hkv, (int)z.N, tiling.seg_len,
                          tiling.block_len, (int)z.CS, (int)z.CB, (int)z.r};
  if (!ei::probe_supported(ps)) return EI_ERR_UNSUPPORTED;
  const ei::SelectShape ss{(int)z.B, (int)z.Hq, (int)z.N, tiling.seg_len, tiling.block_len,
                           (int)z.CS, (int)z.CB, (int)z.r, kmax, params.entropy_threshold,
                           params.alpha, params.delta_t, params.base_budget_tokens,
                           params.max_budget_mult, (int)mode, (int)(z.Hq / z.Hkv)};
  if (!ei::select_supported(ss)) return EI_ERR_UNSUPPORTED;
  const size_t probe_bytes = ei::probe_workspace_bytes(ps);
  if (!workspace || workspace_bytes < probe_bytes + EI_ATTN_WORKSPACE_BYTES)
    return EI_ERR_WORKSPACE;
  if (!aligned16({workspace})) return EI_ERR_UNSUPPORTED;
  const ei::AttnShape as{(int)z.B, (int)z.Hq, (int)z.Hkv, (int)z.N, tiling.seg_len,
                         tiling.block_len, (int)z.CS, (int)z.CB, kmax, softmax_scale};
  // The three stages over the whole layer, in order on one stream.  (Running
  // the probe of one KV group beside the attention of the previous one
  // measured slower: both are bound by vector ALU work, and eight per-group
  // attention launches add their tails.)
  hipStream_t s0 = (hipStream_t)stream;
  hipError_t err = ei::launch_probe(q, k, ps, probe_scale, log_scores, entropy, workspace, s0);
  if (err == hipSuccess)
    err = ei::launch_select(log_scores, entropy, ss, head_is_rigid, budget_blocks, block_idx,
                            block_cnt, s0);
  if (err == hipSuccess)
    err = ei::launch_attention(q, k, v, as, ei::kSparse, block_idx, block_cnt, o,
                               (unsigned char*)workspace + probe_bytes, s0);
  return from_hip(err);
}

ei_status ei_dense_prefill_attn(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                ei_dims dims, float softmax_scale, int32_t causal, uint16_t* o,
                                void* stream) {
  ei_status st = check_dims(dims);
  if (st != EI_OK) return st;
  if (!scale_ok(softmax_scale)) return EI_ERR_SHAPE;
  const Sizes z = sizes(dims, nullptr);
  if (z.B == 0 || z.N == 0) return EI_OK;
  if (!q || !k || !v || !o) return EI_ERR_NULL;
  if (!aligned16({q, k, v, o})) return EI_ERR_UNSUPPORTED;
  const ei::AttnShape as{(int)z.B, (int)z.Hq, (int)z.Hkv, (int)z.N, 128, 64, 0, 0, 0,
                         softmax_scale};
  return from_hip(ei::launch_attention(q, k, v, as,
                                       causal ? ei::kDenseCausal : ei::kDenseFull, nullptr,
                                       nullptr, o, nullptr, (hipStream_t)stream));
}

}  // extern "C"
