/*
 * entropyinfer.h -- C ABI of libentropyinfer.so, the MI355X (gfx950) prefill
 * hot path of EntropyInfer ("From Rigid to Dynamic: Entropy-Guided Adaptive
 * Inference for Long-Context LLMs"):
 *
 *   ei_entropy_probe        Algorithms 1-2 and the row entropy (Section 4.2)
 *   ei_select_blocks        Algorithm 3 (rigid / dynamic heads, budgets) and
 *                           per-segment top-k key-block selection (Section 4.2,
 *                           Appendix A Eq. t_topk)
 *   ei_probe_select_fused   the two above without ln A in memory
 *   ei_sparse_prefill_attn  causal GQA attention over the selected blocks
 *                           (Appendix A Eq. t_spa); _gqa_union: the same with
 *                           two query heads of a KV group per tile
 *   ei_dense_prefill_attn   dense (causal) GQA attention, the full-attention
 *                           baseline the paper compares against
 *
 * Conventions shared by every entry point
 *  - Tensors are contiguous, row-major, in device memory owned by the caller;
 *    the library never allocates, frees or keeps a pointer after returning.
 *  - bf16 tensors are passed as uint16_t bit patterns.
 *  - Q is [B][Hq][N][D], K and V are [B][Hkv][N][D]; query head h reads key
 *    head h / (Hq / Hkv) (grouped-query attention).  D must be 128.
 *  - Segment size L_S and block size L_B (Section 4.1): L_B is 64 or 128
 *    (another L_B: EI_ERR_UNSUPPORTED), L_S a positive multiple of 128 and of
 *    L_B (else EI_ERR_SHAPE).  C_S = ceil(N / L_S) segments, C_B =
 *    ceil(N / L_B) key blocks, r = L_S / L_B.  A ragged tail (N not a
 *    multiple of L_S) forms a short last segment / block.
 *  - Scales: softmax_scale must be finite and > 0, probe_scale finite (else
 *    EI_ERR_SHAPE).
 *  - `stream` is a hipStream_t (NULL = the default stream).  Calls are
 *    asynchronous; outputs are valid once the stream is synchronised.
 *  - Every argument is validated on the host before anything is launched; a
 *    failed check returns a negative ei_status and launches nothing.
 *    B == 0 or N == 0 is valid and launches nothing.
 *  - Alignment: bf16 tensors (Q, K, V, O) and workspaces start on a 16-byte
 *    boundary, fp32 / int32 arrays on a 4-byte one (hipMalloc returns
 *    256-byte aligned memory); a pointer that is not returns
 *    EI_ERR_UNSUPPORTED.
 *  - Outputs must not alias inputs.  Identical inputs give bitwise-identical
 *    outputs (the only atomics are integer counts: in LDS, and the sparse
 *    attention's work-queue counters in its workspace, which decide which
 *    workgroup computes a tile but not what it computes).  No global state
 *    (except the no-allocation variant's scratch array), no logging; calls
 *    on different streams may run concurrently when they do not share a
 *    workspace.
 */
#ifndef ENTROPYINFER_H
#define ENTROPYINFER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  EI_OK = 0,
  EI_ERR_NULL = -1,        /* a required pointer is NULL */
  EI_ERR_SHAPE = -2,       /* inconsistent or out-of-range sizes */
  EI_ERR_UNSUPPORTED = -3, /* valid but not implemented here (e.g. D != 128,
                              a misaligned pointer) */
  EI_ERR_WORKSPACE = -4,   /* workspace missing or smaller than required */
  EI_ERR_LAUNCH = -5       /* a kernel launch failed (hipGetLastError) */
} ei_status;

/* Problem sizes: batch B, query heads Hq, key/value heads Hkv, sequence N,
 * head dimension D.  Every launch's grid is bounded by B * Hq * ceil(N / 128)
 * workgroups, which must not exceed 2^31 - 1 (else EI_ERR_SHAPE). */
typedef struct {
  int32_t batch, n_q_heads, n_kv_heads, seq_len, head_dim;
} ei_dims;

/* Segment size L_S and key-block size L_B (Section 4.1). */
typedef struct {
  int32_t seg_len, block_len;
} ei_tiling;

/* Algorithm 3's constants, exposed as parameters: entropy threshold e_t
 * (1e-5), budget coefficient alpha (0.5), fluctuation threshold Delta_t
 * (0.4), base budget B_h in tokens (2048, Section 5.1.3) and the cap
 * multiplier (3: B_i <= 3 B_h, Appendix A). */
typedef struct {
  float entropy_threshold;
  double alpha;
  double delta_t;
  int32_t base_budget_tokens;
  int32_t max_budget_mult;
} ei_budget_params;

/* Classification of ei_select_blocks_mode.  The block ranking is per query
 * head in every mode; a uniform budget for all heads (the fixed k of
 * CritiPrefill, Section 2) is EI_CLASSIFY_HEAD with entropy_threshold = +inf. */
typedef enum {
  EI_CLASSIFY_HEAD = 0,      /* Algorithm 3 per query head: the method */
  EI_CLASSIFY_GQA_GROUP = 1, /* Algorithm 3 on the mean entropy of each GQA group
                                (the per-group aggregation of Section 3); every
                                head of the group takes the group's budgets */
  EI_CLASSIFY_SEGMENT = 2    /* rigid rule per segment: a segment with
                                e_s < e_t takes B_h, every other segment
                                s >= 1 follows Algorithm 3's update from B_{s-1} */
} ei_classify_mode;

/* Version of this interface (incremented on any change of a signature). */
int32_t ei_abi_version(void);

/* Human-readable name of a status code (static storage). */
const char* ei_status_str(ei_status status);

/* C_S = ceil(N / L_S) and C_B = ceil(N / L_B); -1 on invalid sizes. */
int64_t ei_num_segments(ei_dims dims, ei_tiling tiling);
int64_t ei_num_blocks(ei_dims dims, ei_tiling tiling);

/* Entries per (b, h, s) row of the selection lists:
 * floor(mult * B_h / L_B) + L_S / L_B; -1 on invalid parameters. */
int32_t ei_kmax(ei_tiling tiling, ei_budget_params params);

/* Workspace bytes ei_entropy_probe needs (the pooled Q and K representation
 * vectors of Algorithm 1 as fixed-point limbs, residual parts and scales);
 * 0 on invalid sizes. */
size_t ei_probe_workspace_bytes(ei_dims dims, ei_tiling tiling);

/*
 * ei_entropy_probe -- Algorithms 1 and 2 and the row entropy (Section 4.2).
 *
 * For query head h, segment s and visible key block j < n_vis(s) =
 * min((s+1) r, C_B) (block-causal, including the segment's own blocks):
 * Q_max / Q_min are the element-wise max / min of the segment's query rows,
 * K_max / K_min those of the block's key rows (Algorithm 1); the four logits
 * x_ab = probe_scale * <Q_a, K_b> are formed exactly as integer dot products
 * of 7-bit limbs of the vectors' fixed-point forms (int8 matrix cores), plus
 * the products of the parts below the fixed-point grid where those can move
 * a logit by 2^-30 or more, in binary64; S1..S4 are their softmaxes over j;
 * A = max((S1 + S2) / 2,
 * (S3 + S4) / 2) (Algorithm 2, used without renormalisation); the entropy is
 * -sum_j A ln A (natural log, Section 3).
 *
 *   q, k         bf16 [B][Hq][N][D], [B][Hkv][N][D]
 *   probe_scale  multiplies the logits (finite); 1.0 is Algorithm 2 as printed
 *   log_scores   out, fp32 [B][Hq][C_S][C_B]: ln A for j < n_vis(s); entries
 *                with j >= n_vis(s) are left untouched
 *   entropy      out, fp32 [B][Hq][C_S]
 *   workspace    device scratch of at least ei_probe_workspace_bytes()
 *
 * A non-finite element of Q or K makes every logit it enters, and so its
 * rows' ln A and entropy, NaN.
 *
 * Errors: EI_ERR_NULL, EI_ERR_SHAPE, EI_ERR_UNSUPPORTED (D != 128),
 * EI_ERR_WORKSPACE, EI_ERR_LAUNCH.
 */
ei_status ei_entropy_probe(const uint16_t* q, const uint16_t* k, ei_dims dims,
                           ei_tiling tiling, double probe_scale, float* log_scores,
                           float* entropy, void* workspace, size_t workspace_bytes,
                           void* stream);

/*
 * ei_select_blocks -- head classification, budget allocation (Algorithm 3)
 * and top-k block selection (Section 4.2).
 *
 * Head (b, h) is rigid iff every entropy[b][h][s] < e_t; a NaN entropy makes
 * it dynamic.  Budgets in tokens, binary64, no FMA contraction: rigid
 * B_s = B_h; dynamic B_0 = B_h and B_s = clamp(B_{s-1} + (alpha B_h) *
 * (|e_s - e_{s-1}| / e_{s-1} - Delta_t), B_h, mult B_h) with 0/0 -> 0,
 * x/0 -> +inf and NaN -> B_h.  k_s = min(floor(B_s / L_B), s r) past blocks
 * are kept: those with the largest log_scores (binary32 total order, NaN
 * lowest, -0 == +0, equal scores -> higher block index), plus the segment's
 * own blocks s r .. min((s+1) r, C_B) - 1, which are not charged.
 *
 *   log_scores, entropy  fp32 as written by ei_entropy_probe (only
 *                        j < s r is read)
 *   kmax                 entries per row, >= ei_kmax(tiling, params)
 *   head_is_rigid        out, u8 [B][Hq]
 *   budget_blocks        out, i32 [B][Hq][C_S] = k_s
 *   block_idx            out, i32 [B][Hq][C_S][kmax], strictly ascending,
 *                        padded with -1
 *   block_cnt            out, i32 [B][Hq][C_S] = k_s + own blocks
 *
 * Errors: EI_ERR_NULL, EI_ERR_SHAPE (including kmax too small or a negative
 * budget), EI_ERR_UNSUPPORTED (C_B beyond the selector's register tile),
 * EI_ERR_LAUNCH.
 */
ei_status ei_select_blocks(const float* log_scores, const float* entropy, ei_dims dims,
                           ei_tiling tiling, ei_budget_params params, int32_t kmax,
                           uint8_t* head_is_rigid, int32_t* budget_blocks,
                           int32_t* block_idx, int32_t* block_cnt, void* stream);

/*
 * ei_select_blocks_mode -- ei_select_blocks with the classification variant
 * `mode` (an ei_classify_mode; EI_CLASSIFY_HEAD is ei_select_blocks).
 * EI_CLASSIFY_GQA_GROUP averages the entropies of the n_q_heads / n_kv_heads
 * query heads of each group per segment (binary64 sum in head order, divided
 * by the group size, rounded to binary32) and runs the head rule on the mean;
 * head_is_rigid then holds the group's flag for each of its heads.
 * EI_CLASSIFY_SEGMENT sets B_s = B_h for every segment with e_s < e_t and
 * otherwise applies the clamped update from B_{s-1}; head_is_rigid is set iff
 * every segment is below e_t (then all budgets equal ei_select_blocks').
 *
 * Errors: as ei_select_blocks, plus EI_ERR_SHAPE for an unknown mode.
 */
ei_status ei_select_blocks_mode(const float* log_scores, const float* entropy, ei_dims dims,
                                ei_tiling tiling, ei_budget_params params, int32_t mode,
                                int32_t kmax, uint8_t* head_is_rigid, int32_t* budget_blocks,
                                int32_t* block_idx, int32_t* block_cnt, void* stream);

/* Workspace bytes ei_probe_select_fused needs: ei_probe_workspace_bytes plus
 * 64 bytes per (b, h, s) of softmax statistics; 0 on invalid sizes. */
size_t ei_probe_select_workspace_bytes(ei_dims dims, ei_tiling tiling);

/*
 * ei_probe_select_fused -- ei_entropy_probe followed by ei_select_blocks_mode
 * without the observation matrix ln A in memory (Appendix A: the top-k of
 * Eq. t_topk consumes the C_S x C_B matrix of Eq. t_obs; Section 5's latency
 * study puts the method's extra cost on its per-head work).  After pooling:
 * the entropies, with each (b, h, s) row's softmax statistics kept in the
 * workspace; the classification and budgets of Algorithm 3; then the logits
 * formed once more, ln A of the past blocks held in LDS and the top-k taken
 * there.  entropy, head_is_rigid, budget_blocks, block_idx and block_cnt are
 * bitwise those of the two calls with the same arguments.
 *
 *   q, k, probe_scale    as ei_entropy_probe
 *   params, mode, kmax   as ei_select_blocks_mode
 *   entropy, head_is_rigid, budget_blocks, block_idx, block_cnt
 *                        out, as the two calls (ln A is not produced)
 *   workspace            at least ei_probe_select_workspace_bytes()
 *
 * Errors: those of the two calls; EI_ERR_UNSUPPORTED also when a segment has
 * more than 2048 past blocks ((C_S - 1) L_S / L_B > 2048: the LDS rows of the
 * selection kernel hold at most that many).
 */
ei_status ei_probe_select_fused(const uint16_t* q, const uint16_t* k, ei_dims dims,
                                ei_tiling tiling, double probe_scale, ei_budget_params params,
                                int32_t mode, int32_t kmax, float* entropy,
                                uint8_t* head_is_rigid, int32_t* budget_blocks,
                                int32_t* block_idx, int32_t* block_cnt, void* workspace,
                                size_t workspace_bytes, void* stream);

/*
 * ei_sparse_prefill_attn -- block-sparse causal GQA attention (Section 4.2,
 * Appendix A Eq. t_spa).  Query i of segment s attends to the keys of the
 * blocks block_idx[b][h][s][0 .. block_cnt) that are <= i:
 * O_i = sum_j softmax_j(softmax_scale <q_i, k_j>) v_j, fp32 accumulation and
 * online softmax, bf16 output.
 *
 *   q, k, v        bf16 [B][Hq][N][D], [B][Hkv][N][D], [B][Hkv][N][D]
 *   softmax_scale  usually 1 / sqrt(D); finite and > 0
 *   block_idx      i32 [B][Hq][C_S][kmax] strictly ascending block indices
 *   block_cnt      i32 [B][Hq][C_S]
 *   o              out, bf16 [B][Hq][N][D]
 *
 * A list is read up to block_cnt (clamped to [0, kmax]) and stops at the
 * first entry that is negative, >= C_B or not above its predecessor, so a
 * malformed list never leads to an out-of-bounds access.  A query with no
 * visible key gets a zero row.  The probabilities are formed against a
 * running maximum that may trail the row's maximum by up to 32 (base 2), so
 * each is at most 2^32 before it is accumulated: O stays finite while
 * 2^32 * (keys attended) * max |v| is inside the fp32 range (|v| < 2^79 at
 * 2^17 keys).  A sub-block in which a lane's probabilities sum past 2^32
 * (or overflow) is formed again after the row maximum is raised.
 *
 *   workspace      NULL, or EI_ATTN_WORKSPACE_BYTES of device memory for the
 *                  kernel's work-queue counters (zeroed on `stream` by the
 *                  call itself; a workspace must not be shared by calls that
 *                  may run at the same time)
 *
 * Scheduling (results are bitwise the same either way): with a workspace
 * and B * Hkv a multiple or a divisor of 8, the kernel is persistent (two
 * workgroups per CU), each XCD working through a queue of the (tile, query
 * head) items of its own KV groups (or of its share of one group's tiles),
 * heaviest tiles first, then taking items from the other XCDs' queues; K/V
 * blocks then stay in the L2 of the XCD whose tiles select them.  Otherwise
 * one workgroup per (tile, query head) on a static grid.
 *
 * Errors: EI_ERR_NULL, EI_ERR_SHAPE (also kmax <= 0 or a softmax_scale that is
 * not finite and positive), EI_ERR_UNSUPPORTED (also a workspace not 16-byte
 * aligned), EI_ERR_WORKSPACE (a workspace under EI_ATTN_WORKSPACE_BYTES),
 * EI_ERR_LAUNCH.
 */
#define EI_ATTN_WORKSPACE_BYTES ((size_t)256)
ei_status ei_sparse_prefill_attn(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                 ei_dims dims, ei_tiling tiling, float softmax_scale,
                                 const int32_t* block_idx, const int32_t* block_cnt,
                                 int32_t kmax, uint16_t* o, void* workspace,
                                 size_t workspace_bytes, void* stream);

/*
 * ei_sparse_prefill_attn_gqa_union -- the same attention as
 * ei_sparse_prefill_attn with GQA-union tiles (Section 5's end-to-end latency
 * study puts the method's extra cost over uniform budgets on its per-head
 * budgets, whose heads no longer share K/V loads): one workgroup takes a
 * query tile of two query heads of the same KV head,
 * copies each block of the union of their lists once and lets each head
 * compute only its own blocks.  Same arguments (without a workspace: a static
 * grid) and bitwise the same output as ei_sparse_prefill_attn.
 *
 * Errors: as ei_sparse_prefill_attn; EI_ERR_UNSUPPORTED also when
 * kmax > 128 or C_B > 8192 (the merged list lives in LDS).
 */
ei_status ei_sparse_prefill_attn_gqa_union(const uint16_t* q, const uint16_t* k,
                                           const uint16_t* v, ei_dims dims, ei_tiling tiling,
                                           float softmax_scale, const int32_t* block_idx,
                                           const int32_t* block_cnt, int32_t kmax, uint16_t* o,
                                           void* stream);

/*
 * ei_dense_prefill_attn -- dense GQA attention (Section 2's A_h V), causal
 * (keys j <= i) when `causal` is non-zero, else over all N keys; same tile
 * code and numerics as ei_sparse_prefill_attn.
 *
 * Errors: EI_ERR_NULL, EI_ERR_SHAPE (also a softmax_scale that is not finite
 * and positive), EI_ERR_UNSUPPORTED, EI_ERR_LAUNCH.
 */
ei_status ei_dense_prefill_attn(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                ei_dims dims, float softmax_scale, int32_t causal,
                                uint16_t* o, void* stream);

/* Workspace bytes ei_entropy_guided_prefill needs: ei_probe_workspace_bytes
 * followed by EI_ATTN_WORKSPACE_BYTES for the attention; 0 on invalid sizes. */
size_t ei_prefill_workspace_bytes(ei_dims dims, ei_tiling tiling);

/*
 * ei_entropy_guided_prefill -- the whole prefill path of one layer (Section
 * 4.2): ei_entropy_probe, ei_select_blocks_mode and ei_sparse_prefill_attn
 * over all heads, in this order on `stream`, with the arguments validated
 * once for all three.  The outputs are bitwise those of the three calls.
 *
 *   q, k, v            as ei_sparse_prefill_attn
 *   probe_scale        as ei_entropy_probe; softmax_scale as the attention
 *   params, mode, kmax as ei_select_blocks_mode
 *   log_scores, entropy, head_is_rigid, budget_blocks, block_idx, block_cnt,
 *   o                  outputs of the three calls (same layouts)
 *   workspace          at least ei_prefill_workspace_bytes(): the probe's
 *                      workspace, then the attention's (persistent schedule)
 *
 * Errors: those of the three calls.
 */
ei_status ei_entropy_guided_prefill(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                    ei_dims dims, ei_tiling tiling, double probe_scale,
                                    ei_budget_params params, int32_t mode, int32_t kmax,
                                    float softmax_scale, float* log_scores, float* entropy,
                                    uint8_t* head_is_rigid, int32_t* budget_blocks,
                                    int32_t* block_idx, int32_t* block_cnt, uint16_t* o,
                                    void* workspace, size_t workspace_bytes, void* stream);

/* Device scratch that ei_entropy_guided_prefill_noalloc holds on every device
 * it runs on, until the process ends (128 MiB: the workspace of a layer of 64
 * query and 8 KV heads at 131072 tokens is 123 MiB). */
#define EI_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)

/*
 * ei_entropy_guided_prefill_noalloc -- ei_entropy_guided_prefill for callers
 * that cannot allocate device memory: work captured into a HIP graph, tight
 * serving loops, harnesses that forbid hipMalloc.  The same arguments and
 * bitwise the same outputs, without the workspace: the workspace (the probe's
 * and the attention's) is a static device array of EI_NOALLOC_SCRATCH_BYTES per
 * device (looked up on the first call on a device, with that device current).  The call allocates and
 * frees nothing.  Every call on a device shares that device's array, so calls
 * that overlap on one device (on different streams, or from several threads)
 * race and must be serialised by the caller.
 *
 * Errors: those of ei_entropy_guided_prefill; EI_ERR_WORKSPACE when the
 * problem needs more than EI_NOALLOC_SCRATCH_BYTES (ei_prefill_workspace_bytes
 * tells), EI_ERR_LAUNCH if the scratch array's address cannot be looked up.
 */
ei_status ei_entropy_guided_prefill_noalloc(const uint16_t* q, const uint16_t* k,
                                            const uint16_t* v, ei_dims dims, ei_tiling tiling,
                                            double probe_scale, ei_budget_params params,
                                            int32_t mode, int32_t kmax, float softmax_scale,
                                            float* log_scores, float* entropy,
                                            uint8_t* head_is_rigid, int32_t* budget_blocks,
                                            int32_t* block_idx, int32_t* block_cnt, uint16_t* o,
                                            void* stream);

#ifdef __cplusplus
}
#endif

#endif /* ENTROPYINFER_H */
