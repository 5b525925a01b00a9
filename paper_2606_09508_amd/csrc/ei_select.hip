// Head classification and budget allocation (Algorithm 3) and per-segment
// top-k key-block selection (Section 4.2, Appendix A Eq. t_topk).
//
//  budget_kernel  one workgroup per (b, query head): the rigid test over all
//                 segment entropies, the ratios |e_s - e_{s-1}| / e_{s-1} in
//                 parallel, the clamped budget recurrence (inherently
//                 sequential; one wave, increments broadcast from LDS) and
//                 k_s = min(floor(B_s / L_B), s r).
//                 Variants: the entropies may be the GQA group's means
//                 (binary64 sum in head order / G, rounded to binary32), and
//                 the rigid rule may apply per segment (B_s = B_h wherever
//                 e_s < e_t).
//                 binary64 with FP contraction off, in the order the budget
//                 recurrence is written, so the result is bit-identical to any
//                 other IEEE evaluation in that order.
//  topk_kernel    one wave per (b, h, s) row, reading the row's ln A from
//                 HBM; the selection itself (radix select of the k-th largest
//                 score, ties to the highest block index, ascending output)
//                 is topk::select_row in ei_topk.h.
#include "../../include/entropyinfer.h"
#include "ei_internal.h"
#include "ei_topk.h"

#include <math.h>

#pragma clang fp contract(off)

namespace ei {
namespace {

constexpr int kThreads = 256;
constexpr int kChunk = 1024;

__global__ __launch_bounds__(kThreads) void budget_kernel(
    const float* __restrict__ entropy, int Hq, int CS, int r, int Lb, float e_t, double alpha,
    double delta_t, int Bh, int mult, int mode, int G, uint8_t* __restrict__ rigid_out,
    int32_t* __restrict__ k_out) {
  __shared__ double delta[kChunk];   // -inf: the segment restarts at B_h
  __shared__ double Bs[kChunk];
  const int64_t bh = blockIdx.x;
  int32_t* ko = k_out + bh * CS;
  const int tid = threadIdx.x;
  // the entropy row this head's budgets follow
  const bool group = mode == EI_CLASSIFY_GQA_GROUP;
  const float* e = entropy + (group ? bh - (bh % Hq) % G : bh) * CS;
  auto E = [&](int s) -> float {
    if (!group) return e[s];
    double sum = 0.0;
    for (int h = 0; h < G; ++h) sum += (double)e[(int64_t)h * CS + s];
    return (float)(sum / (double)G);
  };

  int below = 1;
  for (int s = tid; s < CS; s += kThreads)
    if (!(E(s) < e_t)) below = 0;
  below = __syncthreads_and(below);
  const double B0 = (double)Bh;
  const double cap = (double)mult * B0;
  const double a = alpha * B0;
  if (tid == 0) rigid_out[bh] = (uint8_t)(below ? 1 : 0);
  if (below) {
    const int64_t kb = (int64_t)floor(B0 / (double)Lb);
    for (int s = tid; s < CS; s += kThreads)
      ko[s] = (int32_t)min(kb, (int64_t)s * r);
    return;
  }
  double Bprev = B0;   // meaningful in wave 0 only
  for (int c0 = 0; c0 < CS; c0 += kChunk) {
    const int n = min(kChunk, CS - c0);
    // the increments are padded with zeros to a whole number of waves
    const int npad = (n + kWave - 1) / kWave * kWave;
    for (int i = tid; i < npad; i += kThreads) {
      if (i >= n) {
        delta[i] = 0.0;
        continue;
      }
      const int s = c0 + i;
      const float es = E(s);
      // B_0 = B_h, and a rigid segment of the per-segment rule takes B_h:
      // B_prev + (-inf) is clamped to exactly B_h below
      if (s == 0 || (mode == EI_CLASSIFY_SEGMENT && es < e_t)) {
        delta[i] = -INFINITY;
        continue;
      }
      const double ep = (double)E(s - 1), ec = (double)es;
      const double num = fabs(ec - ep);
      const double ratio = (num == 0.0 && ep == 0.0) ? 0.0 : num / ep;
      const double t = ratio - delta_t;
      delta[i] = a * t;
    }
    __syncthreads();
    if (tid < kWave) {
      // Wave 0 runs the recurrence 64 segments at a time, every lane reading
      // each increment from LDS as a broadcast (the loads of a group are
      // independent of the chain and issue ahead of it), so the dependent
      // chain is the add and the two clamps.  The clamps as fmax / fmin give
      // the same value as the comparisons in every case (NaN and -inf -> B_0,
      // +inf -> 3 B_0).  Every lane carries the same B_prev and writes the
      // same value; past the chunk's end the steps run on the zero padding
      // and their results are not read.
      for (int i0 = 0; i0 < n; i0 += kWave) {
#pragma unroll
        for (int j = 0; j < kWave; ++j) {
          Bprev = fmin(fmax(Bprev + delta[i0 + j], B0), cap);
          Bs[i0 + j] = Bprev;
        }
      }
    }
    __syncthreads();
    for (int i = tid; i < n; i += kThreads) {
      const int s = c0 + i;
      const int64_t kb = (int64_t)floor(Bs[i] / (double)Lb);
      ko[s] = (int32_t)min(kb, (int64_t)s * r);
    }
    __syncthreads();
  }
}

constexpr int kWavesPerGroup = kThreads / kWave;

template <int SLOTS>
__global__ __launch_bounds__(kThreads, SLOTS <= 32 ? 6 : 1) void topk_kernel(
    const float* __restrict__ log_scores, const int32_t* __restrict__ kblocks, int64_t rows,
    int CS, int CB, int r, int kmax, int32_t* __restrict__ idx, int32_t* __restrict__ cnt) {
  // per-wave scratch: bucket counts (16-bit halves of 32-bit words: a row has
  // at most 8192 keys) and the compacted keys of T's bucket
  __shared__ __attribute__((aligned(16))) uint32_t hist_all[kWavesPerGroup][topk::kHistWords];
  __shared__ uint32_t cand_all[kWavesPerGroup][topk::kCandWords];
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const int64_t row = (int64_t)blockIdx.x * kWavesPerGroup + wv;
  if (row >= rows) return;   // no workgroup barriers below
  const int lane = threadIdx.x & (kWave - 1);
  const float* L = log_scores + row * (int64_t)CB;
  topk::select_row<SLOTS>([&](int j) { return L[j]; }, (int)(row % CS), r, CB, kmax,
                          kblocks[row], idx + row * (int64_t)kmax, cnt + row, hist_all[wv],
                          cand_all[wv], lane);
}

template <int SLOTS>
hipError_t launch_topk_t(const float* log_scores, const int32_t* kb, const SelectShape& s,
                         int32_t* idx, int32_t* cnt, hipStream_t stream) {
  const int64_t rows = (int64_t)s.B * s.Hq * s.CS;
  const int64_t grid = (rows + (kThreads / kWave) - 1) / (kThreads / kWave);
  hipLaunchKernelGGL(topk_kernel<SLOTS>, dim3((unsigned)grid), dim3(kThreads), 0, stream,
                     log_scores, kb, rows, s.CS, s.CB, s.r, s.kmax, idx, cnt);
  return hipGetLastError();
}

}  // namespace

// the longest row (128 slots per lane) must fit the histogram's 16-bit counters
static_assert(128 * kWave < (1 << 16), "a row's keys must fit one 16-bit bucket counter");
bool select_supported(const SelectShape& s) { return s.CB <= 128 * kWave; }

hipError_t launch_budget(const float* entropy, const SelectShape& s, uint8_t* rigid,
                         int32_t* budget_blocks, hipStream_t stream) {
  hipLaunchKernelGGL(budget_kernel, dim3((unsigned)(s.B * s.Hq)), dim3(kThreads), 0, stream,
                     entropy, s.Hq, s.CS, s.r, s.Lb, s.e_t, s.alpha, s.delta_t, s.Bh, s.mult,
                     s.mode, s.G, rigid, budget_blocks);
  return hipGetLastError();
}

hipError_t launch_select(const float* log_scores, const float* entropy, const SelectShape& s,
                         uint8_t* rigid, int32_t* budget_blocks, int32_t* block_idx,
                         int32_t* block_cnt, hipStream_t stream) {
  hipError_t e = launch_budget(entropy, s, rigid, budget_blocks, stream);
  if (e != hipSuccess) return e;
  const int npast_max = (s.CS - 1) * s.r;
  if (npast_max <= 8 * kWave)
    return launch_topk_t<8>(log_scores, budget_blocks, s, block_idx, block_cnt, stream);
  if (npast_max <= 32 * kWave)
    return launch_topk_t<32>(log_scores, budget_blocks, s, block_idx, block_cnt, stream);
  if (npast_max <= 64 * kWave)
    return launch_topk_t<64>(log_scores, budget_blocks, s, block_idx, block_cnt, stream);
  return launch_topk_t<128>(log_scores, budget_blocks, s, block_idx, block_cnt, stream);
}

}  // namespace ei
