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
//  topk_kernel    one wave per (b, h, s) row: the row's past-block scores sit
//                 in registers as order-preserving 32-bit keys (all loads
//                 issued before any is used).  The k-th largest key T is
//                 found by radix selection: an 11-bit histogram (in LDS,
//                 16-bit counters) of the bits below the keys' common prefix
//                 picks T's bucket (a DPP prefix sum over the lanes' 32-bucket
//                 groups, then one over the chosen group's buckets); the keys
//                 of that bucket (usually few, at most 128 here) are
//                 compacted to two per lane and T's remaining bits are
//                 resolved there with two ballots per bit.  Ties at T keep
//                 the highest block indices; the chosen blocks plus the
//                 segment's own blocks are written ascending.  The kernel is
//                 bound by instruction issue: the row's index is wave-uniform
//                 and every slot loop tests its slot against the row's length
//                 as a scalar branch, so no per-slot lane masks are formed.
#include "../../include/entropyinfer.h"
#include "ei_internal.h"

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

// Order-preserving key of a binary32 score, shifted by one so that 0 marks
// an empty slot: NaN -> 1 (below -inf), -0 == +0, larger float -> larger key.
// Selects only (no branches).
__device__ __forceinline__ uint32_t score_key(float v) {
  const uint32_t u = v == 0.0f ? 0u : __float_as_uint(v);
  const uint32_t k = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (v != v ? 0u : k) + 1u;   // finite/inf keys are <= 0xff800000, so no wrap
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }

// A copy of a wave-uniform value that the optimizer cannot see through: the
// slot tests of each loop against it stay scalar branches, instead of lane
// masks computed once and kept live (in SGPRs, spilled) across the loops.
__device__ __forceinline__ int fresh_uniform(int x) {
  asm volatile("" : "+s"(x));
  return x;
}

constexpr int kWavesPerGroup = kThreads / kWave;
constexpr int kHistBits = 11;
constexpr int kHistBins = 1 << kHistBits;


// Order within one wave between its LDS writes and the reads of other lanes.
__device__ __forceinline__ void wave_lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int SLOTS>
__global__ __launch_bounds__(kThreads, SLOTS <= 32 ? 6 : 1) void topk_kernel(
    const float* __restrict__ log_scores, const int32_t* __restrict__ kblocks, int64_t rows,
    int CS, int CB, int r, int kmax, int32_t* __restrict__ idx, int32_t* __restrict__ cnt) {
  // per-wave scratch: bucket counts (16-bit halves of 32-bit words: a row has
  // at most 8192 keys) and the compacted keys of T's bucket
  __shared__ __attribute__((aligned(16))) uint32_t hist_all[kWavesPerGroup][kHistBins / 2];
  __shared__ uint32_t cand_all[kWavesPerGroup][2 * kWave];
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const int64_t row = (int64_t)blockIdx.x * kWavesPerGroup + wv;
  if (row >= rows) return;   // no workgroup barriers below
  uint32_t* hist = hist_all[wv];
  uint32_t* cand = cand_all[wv];
  const int lane = threadIdx.x & (kWave - 1);
  const int s = (int)(row % CS);
  const int npast = s * r;
  const int kk = kblocks[row];
  const float* L = log_scores + row * (int64_t)CB;
  int32_t* out = idx + row * (int64_t)kmax;
  const int nsl = (npast + kWave - 1) / kWave;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  int pos = 0;

  if (kk >= npast) {
    for (int j = lane; j < npast; j += kWave) out[j] = j;
    pos = npast;
  } else if (kk > 0) {
    uint32_t key[SLOTS];
    uint32_t kmx = 0, kmn = 0xffffffffu;
    // all loads first, unconditionally (lanes past the row read its last
    // past block, one shared line), so that they are in flight together
    float raw[SLOTS];
#pragma unroll
    for (int sl = 0; sl < SLOTS; ++sl) raw[sl] = L[min(sl * kWave + lane, npast - 1)];
#pragma unroll
    for (int sl = 0; sl < SLOTS; ++sl) {
      const int j = sl * kWave + lane;
      key[sl] = j < npast ? score_key(raw[sl]) : 0u;   // j < npast: sl < nsl
      kmx = key[sl] > kmx ? key[sl] : kmx;
      kmn = (key[sl] != 0u && key[sl] < kmn) ? key[sl] : kmn;
    }
    kmx = wave_max_u32_f(kmx);
    kmn = wave_min_u32_f(kmn);
    // T = the kk-th largest key; gt / eq = keys above / equal to T.
    uint32_t T;
    int gt = -1, eq = -1;
    if (kmx == kmn) {
      T = kmx;
      gt = 0;
      eq = npast;
    } else {
      // Valid keys share the bits above `top`; bucket them by the next
      // (up to) 11 bits.
      const int top = 31 - __clz(kmx ^ kmn);
      const uint32_t prefix = kmx & ~((top == 31) ? 0xffffffffu : ((2u << top) - 1u));
      const int shift = max(top - (kHistBits - 1), 0);
      const uint32_t dmask = (2u << (top - shift)) - 1u;
      for (int i = lane; i < kHistBins / 8; i += kWave) ((uint4*)hist)[i] = make_uint4(0, 0, 0, 0);
      wave_lds_fence();
      const int nsh = fresh_uniform(nsl);
#pragma unroll
      for (int sl = 0; sl < SLOTS; ++sl)
        if (sl < nsh && key[sl]) {
          const uint32_t bin = (key[sl] >> shift) & dmask;
          atomicAdd(&hist[bin >> 1], 1u << (16 * (bin & 1)));
        }
      wave_lds_fence();
      // Lane l owns buckets 32 l .. 32 l + 31; find the bucket holding T from
      // the top: the largest d with (keys in buckets >= d) >= kk.
      uint32_t Sp = 0;   // both halves summed at once: each stays below 2^16
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const uint4 w = ((const uint4*)(hist + 16 * lane))[qd];
        Sp += (w.x + w.y) + (w.z + w.w);
      }
      const uint32_t S = (Sp & 0xffffu) + (Sp >> 16);
      const uint32_t pre = wave_incl_scan_u32(S);   // inclusive prefix over lanes
      const uint32_t total = rl_u32(pre, kWave - 1);
      const uint32_t suf = total - pre + S;   // keys in buckets of lanes >= lane
      const uint64_t okm = ballot(suf >= (uint32_t)kk);
      const int ls = 63 - __clzll(okm);     // okm != 0: total = npast > kk
      // lane ls's 32 buckets, highest first, one per lane t < 32: T's bucket
      // is the first at which the keys above ls's buckets plus the running
      // count reach kk (lane ls itself reaches it, so the ballot is not 0)
      const uint32_t acc0 = rl_u32(suf - S, ls);
      uint32_t bt = 0u;
      if (lane < 32) {
        const int bin = 32 * ls + 31 - lane;
        bt = (hist[bin >> 1] >> (16 * (bin & 1))) & 0xffffu;
      }
      const uint32_t run = wave_incl_scan_u32(bt);
      const uint64_t hit = ballot(lane < 32 && acc0 + run >= (uint32_t)kk);
      const int tb = (int)__builtin_ctzll(hit);
      const int dstar = 32 * ls + 31 - tb;
      const uint32_t above = acc0 + rl_u32(run - bt, tb);
      const uint32_t nb = rl_u32(bt, tb);
      T = prefix | ((uint32_t)dstar << shift);
      if (shift == 0) {
        gt = (int)above;
        eq = (int)nb;
      } else if (nb <= (uint32_t)(2 * kWave)) {
        // compact the bucket's keys, two per lane, and resolve the low bits
        int cp = 0;
        const int nsc = fresh_uniform(nsl);
#pragma unroll
        for (int sl = 0; sl < SLOTS; ++sl) {
          if (sl < nsc) {
            const bool in = key[sl] != 0u && ((key[sl] >> shift) & dmask) == (uint32_t)dstar;
            const uint64_t m = ballot(in);
            if (in) cand[cp + popc64(m & lt_mask)] = key[sl];
            cp += popc64(m);
          }
        }
        wave_lds_fence();
        const uint32_t c0 = lane < (int)nb ? cand[lane] : 0u;
        const uint32_t c1 = lane + kWave < (int)nb ? cand[lane + kWave] : 0u;
        for (int bit = shift - 1; bit >= 0; --bit) {
          const uint32_t c = T | (1u << bit);
          if ((int)above + popc64(ballot(c0 >= c)) + popc64(ballot(c1 >= c)) >= kk) T = c;
        }
        gt = (int)above + popc64(ballot(c0 > T)) + popc64(ballot(c1 > T));
        eq = popc64(ballot(c0 == T)) + popc64(ballot(c1 == T));
      } else {
        // large bucket (many equal high bits): resolve over all slots
        for (int bit = shift - 1; bit >= 0; --bit) {
          const uint32_t c = T | (1u << bit);
          int n = 0;
          const int nsb = fresh_uniform(nsl);
#pragma unroll
          for (int sl = 0; sl < SLOTS; ++sl)
            if (sl < nsb) n += popc64(ballot(key[sl] >= c));
          if (n >= kk) T = c;
        }
      }
    }
    if (gt < 0) {
      gt = 0;
      eq = 0;
      const int nse = fresh_uniform(nsl);
#pragma unroll
      for (int sl = 0; sl < SLOTS; ++sl)
        if (sl < nse) {
          gt += popc64(ballot(key[sl] > T));
          eq += popc64(ballot(key[sl] == T));
        }
    }
    const int need = kk - gt;   // 1 .. eq keys equal to T, highest indices first
    int J = 0;
    if (need < eq) {
      // J = the largest index with at least `need` keys equal to T at or
      // above it.  The lane's slots holding T as a bit mask, so that the
      // search keeps no per-slot wave masks live.
      constexpr int kWords = (SLOTS + 31) / 32;
      uint32_t tm[kWords];
#pragma unroll
      for (int w = 0; w < kWords; ++w) tm[w] = 0u;
      const int nst = fresh_uniform(nsl);
#pragma unroll
      for (int sl = 0; sl < SLOTS; ++sl)
        if (sl < nst && key[sl] == T) tm[sl / 32] |= 1u << (sl % 32);
      const int top = 31 - __clz(max(npast - 1, 1));
      for (int bit = top; bit >= 0; --bit) {
        const int c = J | (1 << bit);
        const int cs = c / kWave, cl = c % kWave;   // index c = slot cs, lane cl
        uint32_t nl = 0;
#pragma unroll
        for (int w = 0; w < kWords; ++w) {
          const int lo = cs - 32 * w;   // slots of word w above cs: bits > lo
          const uint32_t above =
              lo < 0 ? 0xffffffffu : (lo >= 31 ? 0u : ~((2u << lo) - 1u));
          nl += __popc(tm[w] & above);
          if (lo >= 0 && lo < 32 && lane >= cl) nl += (tm[w] >> lo) & 1u;
        }
        if ((int)rl_u32(wave_incl_scan_u32(nl), kWave - 1) >= need) J = c;
      }
    }
    // the picks, ascending; J = 0 (the common case) takes every key >= T
    const int nsp = fresh_uniform(nsl);
    if (J == 0) {
#pragma unroll
      for (int sl = 0; sl < SLOTS; ++sl) {
        if (sl < nsp) {
          const bool pick = key[sl] >= T;
          const uint64_t m = ballot(pick);
          if (pick) out[pos + popc64(m & lt_mask)] = sl * kWave + lane;
          pos += popc64(m);
        }
      }
    } else {
#pragma unroll
      for (int sl = 0; sl < SLOTS; ++sl) {
        if (sl < nsp) {
          const int j = sl * kWave + lane;
          const bool pick = key[sl] > T || (key[sl] == T && j >= J);
          const uint64_t m = ballot(pick);
          if (pick) out[pos + popc64(m & lt_mask)] = j;
          pos += popc64(m);
        }
      }
    }
  }
  const int dend = min((s + 1) * r, CB);
  for (int j = npast + lane; j < dend; j += kWave) out[pos + (j - npast)] = j;
  pos += dend - npast;
  for (int t = pos + lane; t < kmax; t += kWave) out[t] = -1;
  if (lane == 0) cnt[row] = pos;
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

hipError_t launch_select(const float* log_scores, const float* entropy, const SelectShape& s,
                         uint8_t* rigid, int32_t* budget_blocks, int32_t* block_idx,
                         int32_t* block_cnt, hipStream_t stream) {
  hipLaunchKernelGGL(budget_kernel, dim3((unsigned)(s.B * s.Hq)), dim3(kThreads), 0, stream,
                     entropy, s.Hq, s.CS, s.r, s.Lb, s.e_t, s.alpha, s.delta_t, s.Bh, s.mult,
                     s.mode, s.G, rigid, budget_blocks);
  hipError_t e = hipGetLastError();
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
