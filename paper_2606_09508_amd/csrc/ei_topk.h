// Top-k key-block selection of one (b, h, s) row (Section 4.2, Appendix A
// Eq. t_topk), shared by the selection kernel (scores read from HBM) and the
// fused probe -> select kernel (scores formed in LDS):
//
//   one wave per row: the row's past-block scores sit in registers as
//   order-preserving 32-bit keys (the loads of all the row's slots issued
//   before any is used).  The k-th largest key T is found by radix
//   selection: a 2048-bucket histogram (in LDS, 16-bit counters) of the
//   keys' offsets from the row's smallest key, buckets of equal width over
//   the row's own key range, picks T's bucket (a DPP prefix sum over the
//   lanes' 32-bucket groups, then one over the chosen group's buckets); the
//   keys of that bucket (usually one or two) are compacted, one or two per
//   lane, and T is the candidate of the right rank among them (by direct
//   comparison up to 64 candidates, else by resolving the offset's low bits
//   with two ballots per bit).  Ties at T keep the highest block indices;
//   the chosen blocks plus the segment's own blocks are written ascending.
//   The row's index is wave-uniform and every slot loop tests its slot
//   against the row's length as a scalar branch, so no per-slot lane masks
//   are formed.
#pragma once

#include "ei_internal.h"

namespace ei {
namespace topk {

constexpr int kHistBits = 11;
constexpr int kHistBins = 1 << kHistBits;
constexpr int kHistWords = kHistBins / 2;   // 16-bit counters, two per word
constexpr int kCandWords = 2 * kWave;        // compacted keys of T's bucket
static_assert(kHistBins % (8 * kWave) == 0, "the histogram is cleared 16 bytes per lane at a time");

// Order-preserving key of a binary32 score, never 0 (0 marks an empty
// slot): NaN -> 1 (below -inf), -0 == +0, larger float -> larger key.
// Selects only (no branches).
__device__ __forceinline__ uint32_t score_key(float v) {
  const uint32_t u = v == 0.0f ? 0u : __float_as_uint(v);
  const uint32_t k = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return v != v ? 1u : k;   // finite / inf keys are >= 0x007fffff (-inf)
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }

// The number of set bits of the wave mask m below this lane.
__device__ __forceinline__ int rank_below(uint64_t m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

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
// `score(j)` is the binary32 score of past block j < npast = s r, and may be
// read for every j < avail (its values past npast are not used); kk = k_s
// blocks are kept (kk >= npast keeps all of them), then the segment's own
// blocks s r .. min((s+1) r, C_B) - 1; out receives kmax entries, ascending,
// -1 padded, and *cnt the count.  hist (kHistWords words) and cand
// (kCandWords words) are this wave's LDS scratch.
template <int SLOTS, class Score>
__device__ __forceinline__ void select_row(Score score, int avail, int s, int r, int CB, int kmax,
                                           int kk,
                                           int32_t* __restrict__ out, int32_t* __restrict__ cnt,
                                           uint32_t* hist, uint32_t* cand, int lane) {
  const int npast = s * r;
  const int nsl = (npast + kWave - 1) / kWave;
  int pos = 0;

  if (kk >= npast) {
    for (int j = lane; j < npast; j += kWave) out[j] = j;
    pos = npast;
  } else if (kk > 0) {
    uint32_t key[SLOTS];
    uint32_t kmx = 0, kmn1 = 0xffffffffu;   // kmn1: the smallest non-empty key - 1
    // the loads of the row's slots first, in groups of kG slots, so that
    // they are in flight together; lanes past the row read unused values
    // (past npast, or its last past block where the groups reach past avail)
    float raw[SLOTS];
    constexpr int kG = SLOTS <= 8 ? SLOTS : 8;
    const int nsr = SLOTS <= kG ? 1 : fresh_uniform(nsl);
    if ((nsl + kG - 1) / kG * kG * kWave <= avail) {
      // every slot of the groups loaded is readable: no clamp
#pragma unroll
      for (int g = 0; g < SLOTS; g += kG)
        if (g < nsr) {
#pragma unroll
          for (int sl = g; sl < g + kG; ++sl) raw[sl] = score(sl * kWave + lane);
        }
    } else {
#pragma unroll
      for (int g = 0; g < SLOTS; g += kG)
        if (g < nsr) {
#pragma unroll
          for (int sl = g; sl < g + kG; ++sl) raw[sl] = score(min(sl * kWave + lane, npast - 1));
        }
    }
    const int nsk = SLOTS <= kG ? 1 : fresh_uniform(nsl);
#pragma unroll
    for (int g = 0; g < SLOTS; g += kG) {
      if (g + kG < nsk) {
        // every slot of the group is full (only the row's last slot is not)
#pragma unroll
        for (int sl = g; sl < g + kG; ++sl) {
          key[sl] = score_key(raw[sl]);
          kmx = key[sl] > kmx ? key[sl] : kmx;
          kmn1 = min(kmn1, key[sl] - 1u);
        }
      } else if (g < nsk) {
#pragma unroll
        for (int sl = g; sl < g + kG; ++sl) {
          const uint32_t k = score_key(raw[sl]);
          key[sl] = (uint32_t)(sl * kWave + lane - npast) >> 31 ? k : 0u;   // j < npast
          kmx = key[sl] > kmx ? key[sl] : kmx;
          kmn1 = min(kmn1, key[sl] - 1u);   // an empty slot's 0 wraps to the maximum
        }
      } else {
#pragma unroll
        for (int sl = g; sl < g + kG; ++sl) key[sl] = 0u;
      }
    }
    kmx = wave_max_u32_f(kmx);
    const uint32_t kmn = wave_min_u32_f(kmn1) + 1u;
    // T = the kk-th largest key; gt / eq = keys above / equal to T.
    uint32_t T;
    int gt = -1, eq = -1;
    if (kmx == kmn) {
      T = kmx;
      gt = 0;
      eq = npast;
    } else {
      // Bucket the keys by their offset from the smallest, (key - kmn) >>
      // shift < 2^11: buckets of equal width over the row's own key range.
      const int shift = max(32 - __clz(kmx - kmn) - kHistBits, 0);
#pragma unroll
      for (int i = 0; i < kHistBins / 8 / kWave; ++i)
        ((uint4*)hist)[i * kWave + lane] = make_uint4(0, 0, 0, 0);
      wave_lds_fence();
      const int nsh = fresh_uniform(nsl);
      auto count = [&](uint32_t kv) {
        // bucket (kv - kmn) >> shift: half (bucket & 1) of word bucket >> 1
        const uint32_t d = kv - kmn;
        const uint32_t half = __builtin_amdgcn_ubfe(d, (uint32_t)shift, 1u);
        atomicAdd(&hist[d >> (shift + 1)], __umul24(half, 0xffffu) + 1u);   // 1 or 1 << 16
      };
#pragma unroll
      for (int g = 0; g < SLOTS; g += kG) {
        if (g + kG < nsh) {
#pragma unroll
          for (int sl = g; sl < g + kG; ++sl) count(key[sl]);   // full slots
        } else if (g < nsh) {
#pragma unroll
          for (int sl = g; sl < g + kG; ++sl)
            if (sl < nsh && key[sl]) count(key[sl]);
        }
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
      // T = kmn + Toff; Toff's bits below `shift` are resolved from the top
      uint32_t Toff = (uint32_t)dstar << shift;
      if (shift == 0) {
        T = kmn + Toff;
        gt = (int)above;
        eq = (int)nb;
      } else if (nb <= (uint32_t)(2 * kWave)) {
        // compact the bucket's keys, two per lane, and resolve the low bits
        // the bucket's keys are those in [blo, bhi] (an empty slot's 0 is
        // below blo >= kmn >= 1)
        const uint32_t blo = kmn + Toff, bhi = blo + ((1u << shift) - 1u);
        int cp = 0;
        const int nsc = fresh_uniform(nsl);
#pragma unroll
        for (int sl = 0; sl < SLOTS; ++sl) {
          if (sl < nsc) {
            const bool in = key[sl] >= blo && key[sl] <= bhi;
            const uint64_t m = ballot(in);
            if (m != 0) {
              if (in) cand[(uint32_t)(cp + rank_below(m))] = key[sl];
              cp += popc64(m);
            }
          }
        }
        wave_lds_fence();
        const uint32_t c0 = lane < (int)nb ? cand[lane] : 0u;
        if (nb <= (uint32_t)kWave) {
          // one candidate per lane: T is the one with fewer than `need`
          // candidates above it and at least `need` at or above it
          const int need = kk - (int)above;   // 1 .. nb
          int ngt = 0, nge = 0;
          for (int t = 0; t < (int)nb; ++t) {
            const uint32_t x = cand[t];   // the same word for every lane
            ngt += x > c0 ? 1 : 0;
            nge += x >= c0 ? 1 : 0;
          }
          const uint64_t hm = ballot(lane < (int)nb && ngt < need && need <= nge);
          T = rl_u32(c0, (int)__builtin_ctzll(hm));
          gt = (int)above + popc64(ballot(c0 > T));
          eq = popc64(ballot(c0 == T));
        } else {
        const uint32_t c1 = lane + kWave < (int)nb ? cand[lane + kWave] : 0u;
        for (int bit = shift - 1; bit >= 0; --bit) {
          const uint32_t co = Toff | (1u << bit), c = kmn + co;   // empty (0) is below c
          if ((int)above + popc64(ballot(c0 >= c)) + popc64(ballot(c1 >= c)) >= kk) Toff = co;
        }
        T = kmn + Toff;
        gt = (int)above + popc64(ballot(c0 > T)) + popc64(ballot(c1 > T));
        eq = popc64(ballot(c0 == T)) + popc64(ballot(c1 == T));
        }
      } else {
        // large bucket (many keys of nearly one value): resolve over all slots
        for (int bit = shift - 1; bit >= 0; --bit) {
          const uint32_t co = Toff | (1u << bit), c = kmn + co;
          int n = 0;
          const int nsb = fresh_uniform(nsl);
#pragma unroll
          for (int sl = 0; sl < SLOTS; ++sl)
            if (sl < nsb) n += popc64(ballot(key[sl] >= c));
          if (n >= kk) Toff = co;
        }
        T = kmn + Toff;
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
          if (pick) out[(uint32_t)(pos + rank_below(m))] = sl * kWave + lane;
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
          if (pick) out[(uint32_t)(pos + rank_below(m))] = j;
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
