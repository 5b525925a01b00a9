// Head classification and budget allocation (Algorithm 3) and per-segment
// top-k key-block selection (Section 4.2, Appendix A Eq. t_topk).
//
//  budget_kernel  one workgroup per (b, query head): the rigid test over all
//                 segment entropies, the ratios |e_s - e_{s-1}| / e_{s-1} in
//                 parallel, the clamped budget recurrence and
//                 k_s = min(floor(B_s / L_B), s r).  The recurrence runs in
//                 one wave, each lane owning a run of consecutive steps:
//                 since one step x -> min(max(x + d, B_h), m B_h) is
//                 monotone, a run evaluated from both ends of an interval
//                 holding its true start bounds its true values.  Each round
//                 every lane runs its steps from both ends of its interval
//                 and hands the two ends reached to the next lane; an
//                 interval that has shrunk to one value is the true start.
//                 Runs that meet a clamp from both ends settle the next lane
//                 at once, and after at most 63 rounds every start is known
//                 (the sequential order, in the worst case).
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
constexpr int kRunMax = kChunk / kWave;   // steps per lane in the budget recurrence

// Lane l receives lane l - 1's v (lane 0 keeps its own): a DPP wave shift.
__device__ __forceinline__ double shift_up1(double v) {
  const int2 w = __builtin_bit_cast(int2, v);
  const int lo = __builtin_amdgcn_update_dpp(w.x, w.x, 0x138, 0xf, 0xf, false);   // wave_shr:1
  const int hi = __builtin_amdgcn_update_dpp(w.y, w.y, 0x138, 0xf, 0xf, false);
  return __builtin_bit_cast(double, make_int2(lo, hi));
}

template <bool GROUP>
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
  const float* e = entropy + (GROUP ? bh - (bh % Hq) % G : bh) * CS;
  auto E = [&](int s) -> float {
    if constexpr (!GROUP) {
      return e[s];
    } else {
      double sum = 0.0;
      for (int h = 0; h < G; ++h) sum += (double)e[(int64_t)h * CS + s];
      return (float)(sum / (double)G);
    }
  };

  const double B0 = (double)Bh;
  const double cap = (double)mult * B0;
  const double a = alpha * B0;
  // The increments of the chunk of steps at c0 (n steps) into delta.  The
  // steps are padded with zero increments to a whole number of waves (a zero
  // increment leaves a clamped value unchanged) and split into kWave runs of
  // L consecutive steps; step i = l L + j of lane l's run is held at
  // delta[j kWave + l], so every lane's reads and writes of a step are one
  // conflict-free row.  Up to four steps per thread, with selects rather
  // than branches so that their loads issue together (a padding step reads
  // an unused segment).  Returns 0 if a segment of the chunk is not below
  // e_t.
  auto increments = [&](int c0, int n) {
    const int npad = (n + kWave - 1) / kWave * kWave;
    const int L = npad / kWave;
    int low = 1;
#pragma unroll 4
    for (int p = tid; p < npad; p += kThreads) {
      const int i = (p % kWave) * L + p / kWave;
      const int s = c0 + min(i, n - 1);
      const float es = E(s), eprev = E(max(s - 1, 0));
      if (!(es < e_t)) low = 0;
      const double ep = (double)eprev, ec = (double)es;
      const double num = fabs(ec - ep);
      const double ratio = (num == 0.0 && ep == 0.0) ? 0.0 : num / ep;
      double d = a * (ratio - delta_t);
      // B_0 = B_h, and a rigid segment of the per-segment rule takes B_h:
      // B_prev + (-inf) is clamped to exactly B_h below
      d = (s == 0 || (mode == EI_CLASSIFY_SEGMENT && es < e_t)) ? -INFINITY : d;
      delta[p] = i < n ? d : 0.0;
    }
    return low;
  };

  // the rigid test over every segment, the first chunk's increments on the way
  int below = increments(0, min(kChunk, CS));
#pragma unroll 4
  for (int s = kChunk + tid; s < CS; s += kThreads)
    if (!(E(s) < e_t)) below = 0;
  below = __syncthreads_and(below);
  if (tid == 0) rigid_out[bh] = (uint8_t)(below ? 1 : 0);
  if (below) {
    const int64_t kb = (int64_t)floor(B0 / (double)Lb);
    for (int s = tid; s < CS; s += kThreads)
      ko[s] = (int32_t)min(kb, (int64_t)s * r);
    return;
  }
  double Bprev = B0;   // wave 0: B before the chunk's first step
  for (int c0 = 0; c0 < CS; c0 += kChunk) {
    const int n = min(kChunk, CS - c0);
    const int L = (n + kWave - 1) / kWave, npad = L * kWave;
    if (c0 > 0) increments(c0, n);   // the first chunk's are in delta already
    __syncthreads();
    if (tid < kWave) {
      // One step of the recurrence.  The clamps as fmax / fmin give the same
      // value as the comparisons in every case (NaN and -inf -> B_h, +inf ->
      // m B_h), and every value a step yields lies in [lo, hi].
      auto step = [&](double x, double d) { return fmin(fmax(x + d, B0), cap); };
      const double lo = step(B0, -INFINITY), hi = step(B0, INFINITY);
      const int lane = tid;
      double dv[kRunMax];   // the lane's increments (entries j >= L unused)
#pragma unroll
      for (int j = 0; j < kRunMax; ++j) dv[j] = delta[j * kWave + lane];
      // A step is monotone in x, so a run evaluated from the two ends of an
      // interval holding its true start bounds every true value of the run.
      // Each round every lane runs its steps from both ends of its start
      // interval, and its successor takes the two ends reached as its next
      // start interval.  Lane 0 starts from the carried B itself; a lane whose
      // start interval is one value (equal bit patterns) has its true start,
      // and so does its successor one round later at the latest, so after at
      // most kWave - 1 rounds every start is known.  Runs that meet a clamp
      // from both ends settle their successors much sooner.  (The one thing
      // the bounds cannot settle is the sign of a zero budget, which no k_s
      // depends on.)
      double pl = lane == 0 ? Bprev : lo, ph = lane == 0 ? Bprev : hi;
      while (__builtin_amdgcn_ballot_w64(__double_as_longlong(pl) ==
                                         __double_as_longlong(ph)) != ~0ull) {
        double xl = pl, xh = ph;
#pragma unroll
        for (int j = 0; j < kRunMax; ++j)
          if (j < L) {
            xl = step(xl, dv[j]);
            xh = step(xh, dv[j]);
          }
        xl = shift_up1(xl);
        xh = shift_up1(xh);
        if (lane > 0) {
          pl = xl;
          ph = xh;
        }
      }
      // every lane from its true start, in the recurrence's own order
      double x = pl;
#pragma unroll
      for (int j = 0; j < kRunMax; ++j)
        if (j < L) {
          x = step(x, dv[j]);
          Bs[j * kWave + lane] = x;
        }
      Bprev = __shfl(x, kWave - 1);
    }
    __syncthreads();
    for (int p = tid; p < npad; p += kThreads) {
      const int i = (p % kWave) * L + p / kWave;
      if (i >= n) continue;
      const int s = c0 + i;
      const int64_t kb = (int64_t)floor(Bs[p] / (double)Lb);
      ko[s] = (int32_t)min(kb, (int64_t)s * r);
    }
    __syncthreads();
  }
}

constexpr int kWavesPerGroup = kThreads / kWave;

template <int SLOTS>
__global__ __launch_bounds__(kThreads, SLOTS <= 16 ? 8 : SLOTS <= 32 ? 6 : 1) void topk_kernel(
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
  topk::select_row<SLOTS>([&](int j) { return L[j]; }, CB, (int)(row % CS), r, CB, kmax,
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
  if (s.mode == EI_CLASSIFY_GQA_GROUP)
    hipLaunchKernelGGL(budget_kernel<true>, dim3((unsigned)(s.B * s.Hq)), dim3(kThreads), 0,
                       stream, entropy, s.Hq, s.CS, s.r, s.Lb, s.e_t, s.alpha, s.delta_t, s.Bh,
                       s.mult, s.mode, s.G, rigid, budget_blocks);
  else
    hipLaunchKernelGGL(budget_kernel<false>, dim3((unsigned)(s.B * s.Hq)), dim3(kThreads), 0,
                       stream, entropy, s.Hq, s.CS, s.r, s.Lb, s.e_t, s.alpha, s.delta_t, s.Bh,
                       s.mult, s.mode, s.G, rigid, budget_blocks);
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
  if (npast_max <= 16 * kWave)
    return launch_topk_t<16>(log_scores, budget_blocks, s, block_idx, block_cnt, stream);
  if (npast_max <= 32 * kWave)
    return launch_topk_t<32>(log_scores, budget_blocks, s, block_idx, block_cnt, stream);
  if (npast_max <= 64 * kWave)
    return launch_topk_t<64>(log_scores, budget_blocks, s, block_idx, block_cnt, stream);
  return launch_topk_t<128>(log_scores, budget_blocks, s, block_idx, block_cnt, stream);
}

}  // namespace ei
