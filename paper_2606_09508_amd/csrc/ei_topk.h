// Top-k key-block selection of one (b, h, s) row (Section 4.2, Appendix A
// Eq. t_topk), shared by the selection kernel (scores read from HBM) and the
// fused probe -> select kernel (scores formed in LDS):
//
//   one wave per row: the row's past-block scores sit in registers as
//   order-preserving 32-bit keys (all loads issued before any is used).  The
//   k-th largest key T is found by radix selection: an 11-bit histogram (in
//   LDS, 16-bit counters) of the bits below the keys' common prefix picks T's
//   bucket (a DPP prefix sum over the lanes' 32-bucket groups, then one over
//   the chosen group's buckets); the keys of that bucket (usually few, at
//   most 128 here) are compacted to two per lane and T's remaining bits are
//   resolved there with two ballots per bit.  Ties at T keep the highest
//   block indices; the chosen blocks plus the segment's own blocks are
//   written ascending.  The routine is bound by instruction issue: the row's
//   index is wave-uniform and every slot loop tests its slot against the
//   row's length as a scalar branch, so no per-slot lane masks are formed.
#pragma once

#include "ei_internal.h"

namespace ei {
namespace topk {

constexpr int kHistBits = 11;
constexpr int kHistBins = 1 << kHistBits;
constexpr int kHistWords = kHistBins / 2;   // 16-bit counters, two per word
constexpr int kCandWords = 2 * kWave;        // compacted keys of T's bucket

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

// Order within one wave between its LDS writes and the reads of other lanes.
__device__ __forceinline__ void wave_lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// One row, by the whole wave (every argument wave-uniform but `lane`):
// `score(j)` is the binary32 score of past block j < npast = s r; kk = k_s
// blocks are kept (kk >= npast keeps all of them), then the segment's own
// blocks s r .. min((s+1) r, C_B) - 1; out receives kmax entries, ascending,
// -1 padded, and *cnt the count.  hist (kHistWords words) and cand
// (kCandWords words) are this wave's LDS scratch.
template <int SLOTS, class Score>
__device__ __forceinline__ void select_row(Score score, int s, int r, int CB, int kmax, int kk,
                                           int32_t* __restrict__ out, int32_t* __restrict__ cnt,
                                           uint32_t* hist, uint32_t* cand, int lane) {
  const int npast = s * r;
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
    for (int sl = 0; sl < SLOTS; ++sl) raw[sl] = score(min(sl * kWave + lane, npast - 1));
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
  if (lane == 0) *cnt = pos;
}

}  // namespace topk
}  // namespace ei
