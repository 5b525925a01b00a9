// Causal GQA prefill attention on bf16 MFMA (gfx950), block-sparse over the
// selected key blocks (Section 4.2, Appendix A Eq. t_spa) or dense (the
// full-attention baseline).
//
// One workgroup = one 128-row query tile of one (batch, query head); four
// waves own 32 query rows each.  Keys are visited in 64-key sub-blocks copied
// straight from global memory into a two-stage LDS ring (no register
// staging); per sub-block each wave computes
//   S^T = K Q^T        2 x 8  MFMA 32x32x16 (keys on M, queries on N)
//   online softmax     fp32, base 2, the row of one query lives in one lane
//                      pair (lanes l and l^32)
//   O^T += V^T P^T     4 x 4  MFMA 32x32x16 (head dims on M)
// With keys on the M dimension every lane owns one query's scores, so the
// softmax needs a single cross-lane exchange per sub-block, and the output
// rescale uses the lane's own running maximum.
//
// MFMA 32x32x16 bf16 operand layout (lane l, half h = l / 32):
//   A[i][k]: lane holds i = l % 32, k = 8h .. 8h+7
//   B[k][j]: lane holds j = l % 32, k = 8h .. 8h+7
//   D[i][j]: lane holds j = l % 32, i = 8 (r / 4) + 4h + r % 4, r = 0..15
// The keys of the S^T output a lane holds are therefore not contiguous; the
// V^T operand is read from the row-major V tile with the transposing LDS read
// (ds_read_b64_tr_b16) in that same key order, so P^T feeds the second
// product straight from registers.
//
// Dense workgroups are mapped so that each XCD (dispatched round-robin)
// receives a contiguous run of (batch, KV head, tile, query head) work: the G
// query heads that share a K/V head, and neighbouring tiles, run on one XCD
// and reuse K/V blocks from its L2.  Heavier (later) tiles are issued first.
//
// Sparse work per head is uneven (budgets differ per head, up to 3x).  With a
// scheduling workspace the sparse kernel is persistent: two workgroups per
// CU, each taking (tile, KV group, query head) items from a queue of its own
// XCD (the XCD's KV groups, or its share of one group's tiles in runs of
// kRun, heaviest tiles first) through an atomic counter, and from the other
// XCDs' queues once its own is empty.  Each XCD's L2 then holds the K/V of
// its own groups, whose tiles select largely the same blocks, and the
// stealing evens out the groups' different loads.  Without a workspace (or
// for KV-group counts that do not tile the XCDs) the grid is static: the KV
// groups rotate over the XCDs every 4 tiles, heaviest tiles first.
#include "ei_internal.h"

#include <math.h>

namespace ei {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int kTileQ = 128;
constexpr int kSub = 64;            // keys per staged sub-block
constexpr int kXcds = 8;
constexpr unsigned kRotRun = 4;    // tiles a KV group stays on one XCD (static sparse grid)
constexpr unsigned kRun = 16;      // tile run per XCD when XCDs share a KV group (persistent)
constexpr unsigned kHeadRun = 16;  // tiles of one query head in a row in an XCD's queue

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 w) { return __builtin_bit_cast(bf16x8, w); }

// Two fp32 values -> packed bf16 pair (round to nearest even), one instruction.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2 x = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(x, bf16x2));
}

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4_t;

// One LDS stage holds a 64-key sub-block of K and of V, each row-major with
// 256-byte rows whose 16-byte chunks are XOR-swizzled per row.  K rows are
// read 16 at a time at one logical chunk, so K uses chunk ^ (r % 16).  The
// transposing V reads take, per 16 lanes, the same 32-byte chunk pair of 4
// consecutive rows (and per 32 lanes a 64-byte chunk quad), so V uses
// chunk ^ h(r % 4) with h = {0, 6, 12, 10}: the pair index and the quad index
// then differ across any 4 consecutive rows and every read is free of bank
// conflicts.
constexpr int kRowBytes = kHeadDim * 2;
constexpr int kTileBytes = kSub * kRowBytes;       // 16 KiB
constexpr int kStageBytes = 2 * kTileBytes;        // K then V

__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ (row & 15); }
__device__ __forceinline__ int swz_v(int row, int chunk) {
  return chunk ^ ((0xAC60 >> (4 * (row & 3))) & 15);
}

// 16 bytes per lane from global memory straight into LDS at lds_base + 16 *
// lane (global_load_lds_dwordx4; M0 holds the LDS base and is restored).
// Written as asm so that the compiler does not treat the copy as a pending
// LDS write before every later LDS read: completion is enforced explicitly
// with a vmcnt wait before the barrier that publishes a stage.
__device__ __forceinline__ void copy16_to_lds(const uint16_t* src, uint32_t lds_base) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds_base), "v"(src)
      : "memory");
}

// The same copy with the global address formed as a wave-uniform base (SGPR
// pair) plus a 32-bit lane offset, so that issuing it takes no vector
// arithmetic (M0 restored as above).
__device__ __forceinline__ void copy16_to_lds_s(const unsigned char* sbase, uint32_t voff,
                                                uint32_t lds_base) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, %3\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds_base), "v"(voff), "s"(sbase)
      : "memory");
}

// Global -> LDS without registers: each wave moves 16 rows of K and 16 rows
// of V (4 + 4 instructions of 64 lanes x 16 bytes).  Lane L of instruction j
// fills row 16 w + 4 j + L / 16, swizzled chunk position L % 16; koff / voff
// hold those rows' byte offsets inside a block.  Rows at or past N are read
// from row N - 1 (finite data whose scores are masked).
__device__ __forceinline__ void issue_stage(unsigned char* stage, const uint16_t* __restrict__ kh,
                                            const uint16_t* __restrict__ vh, int k0, int N,
                                            int wave, int lane, const uint32_t* koff,
                                            const uint32_t* voff) {
  const int pos = lane & 15;
  const uint32_t base = (uint32_t)(uintptr_t)stage;
  if (k0 + kSub <= N) {   // whole block inside the sequence
    const unsigned char* kb = (const unsigned char*)kh + (size_t)k0 * kRowBytes;
    const unsigned char* vb = (const unsigned char*)vh + (size_t)k0 * kRowBytes;
    const uint32_t dst0 =
        base + (uint32_t)(16 * __builtin_amdgcn_readfirstlane(wave) * kRowBytes);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      copy16_to_lds_s(kb, koff[j], dst0 + 4 * j * kRowBytes);
      copy16_to_lds_s(vb, voff[j], dst0 + 4 * j * kRowBytes + kTileBytes);
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int row = 16 * wave + 4 * j + (lane >> 4);
    const int grow = min(k0 + row, N - 1);
    const size_t roff = (size_t)grow * kHeadDim;
    const uint32_t dst = base + (uint32_t)((16 * wave + 4 * j) * kRowBytes);
    copy16_to_lds(kh + roff + 8 * swz(row, pos), __builtin_amdgcn_readfirstlane(dst));
    copy16_to_lds(vh + roff + 8 * swz_v(row, pos),
                  __builtin_amdgcn_readfirstlane(dst + kTileBytes));
  }
}

// K operand of S^T = K Q^T: 8 bf16 of key row `row`, dims 16 s + 8 h .. +7.
__device__ __forceinline__ bf16x8 read_k(const unsigned char* stage, int row, int s, int h) {
  return as_bf16x8(*(const uint4*)(stage + row * kRowBytes + 16 * swz(row, 2 * s + h)));
}

// V^T operand of O^T += V^T P^T for head-dim tile dt and 16-key step t, read
// transposed from the row-major V tile: lane l (group g = l / 16, i = l % 16)
// receives V[key][32 dt + 16 (g % 2) + i] for the keys 16 t + 8 a + 4 (g / 2)
// + 0..3, a = 0, 1 -- the key order of the S^T output.
__device__ __forceinline__ bf16x8 read_vt(const unsigned char* stage, int dt, int t, int lane) {
  const int g = lane >> 4, i = lane & 15;
  const int d = 32 * dt + 16 * (g & 1) + 4 * (i & 3);
  const unsigned char* vt = stage + kTileBytes;
  s16x4 r[2];
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    const int row = 16 * t + 8 * a + 4 * (g >> 1) + (i >> 2);
    const unsigned char* p = vt + row * kRowBytes + 16 * swz_v(row, d >> 3) + 2 * (d & 7);
    r[a] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)p);
  }
  const uint2 lo = __builtin_bit_cast(uint2, r[0]), hi = __builtin_bit_cast(uint2, r[1]);
  return as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
}

// Wait until at most n vector-memory operations of this wave are in flight
// (gfx9 encoding: vmcnt in bits 3:0 and 15:14; expcnt, lgkmcnt left at max).
#define EI_WAIT_VMCNT(n) \
  __builtin_amdgcn_s_waitcnt(((n) & 15) | (((n) >> 4) << 14) | (7 << 4) | (15 << 8))

// The persistent sparse schedule (see the file comment).  S = 1: XCD x owns
// the KV groups x, x + 8, ... (ngx of them), its queue running over chunks of
// kHeadRun tile ranks (heaviest first) and, inside a chunk, over its (group,
// query head) pairs, each taking the chunk's tiles in a row (at the 128k
// layer: 10.5 GB fetched per launch against 13.7 GB with the heads of a
// tile next to each other, and equal or 1-2% faster).  S > 1 (8 = S x the
// number of groups): XCD x owns group x % NG and, of its tiles ranked
// heaviest first, the runs of kRun ranks with (rank / kRun) % S == x / NG.
// per_x[x] is the length of XCD x's queue.  Every item appears in exactly
// one queue.
struct XcdPlan {
  unsigned S, ngx, per_x[kXcds];
};

// Item idx of XCD x's queue -> (tile, query head in the group, KV group).
__device__ __forceinline__ void plan_item(const XcdPlan& pl, unsigned x, unsigned idx, int n_tiles,
                                          unsigned G, unsigned NG, int& tile, int& hh,
                                          unsigned& bg) {
  unsigned tr;
  if (pl.S == 1) {
    // chunks of kHeadRun tile ranks, heaviest first; inside a chunk the
    // (group, head) pairs in turn, each over the chunk's ranks
    const unsigned per_rank = G * pl.ngx;
    const unsigned c = idx / (kHeadRun * per_rank), j = idx % (kHeadRun * per_rank);
    const unsigned rr = min(kHeadRun, (unsigned)n_tiles - c * kHeadRun);   // ranks in the chunk
    const unsigned hg = j / rr;
    tr = c * kHeadRun + j % rr;
    hh = (int)(hg % G);
    bg = x + kXcds * (hg / G);
  } else {
    const unsigned kq = idx / G, part = x / NG;
    hh = (int)(idx % G);
    bg = x % NG;
    tr = (kq / kRun) * (pl.S * kRun) + part * kRun + kq % kRun;
  }
  tile = n_tiles - 1 - (int)tr;
}

// Queue counters of one call (the caller's scheduling workspace), zeroed on
// the call's stream before the kernel reads them.
__global__ void sched_reset_kernel(uint32_t* __restrict__ sched) {
  if (threadIdx.x < kXcds) sched[threadIdx.x] = 0u;
}

// Lazy rescaling: the running maximum m is only raised when a new score
// exceeds it by more than 8 (base-2 units), so O and l are rescaled rarely; O
// and l always share the same reference, so the result is the exact softmax.
// A sub-block's probabilities are first formed against the current m without
// its row maximum: if every lane's sum of them stays <= 2^32 (so each
// probability does, and O, l stay far from overflow), they are kept.
// Otherwise (the first sub-block, a score more than 32 above m, or an
// overflow) the wave takes the row maxima, raises m by the rule above and
// forms them again.
constexpr float kRescaleThreshold = 8.0f;
constexpr float kFastLimit = 0x1p32f;

// Valid prefix of a block list of c entries, 64 at a time: strictly
// ascending, inside [0, C_B), and not wholly after the tile's last query.
template <int SUB>
__device__ __forceinline__ int valid_prefix(const int32_t* lst, int c, int CB, int q_last,
                                            int lane) {
  int nv = 0;
  for (int base = 0; base < c; base += kWave) {
    const int e = base + lane;
    bool ok = false;
    if (e < c) {
      const int blk = lst[e];
      const int prv = e > 0 ? lst[e - 1] : -1;
      ok = blk > prv && blk < CB && blk * SUB * kSub <= q_last;
    }
    const uint64_t bad = ~__builtin_amdgcn_ballot_w64(ok);
    if (bad != 0) {
      nv = base + (int)__builtin_ctzll(bad);
      break;
    }
    nv = base + kWave;
  }
  return min(nv, c);
}

// One 64-key sub-block (staged at st, first key k0) for the wave's 32 query
// rows: S^T = K Q^T, the causal / length mask, the online softmax with lazy
// rescaling, and O^T += V^T P^T.
template <int MODE>
__device__ __forceinline__ void compute_step(const unsigned char* st, int k0, int qw0, int qrow,
                                             int N, int jq, int hf, int lane, const bf16x8* qf,
                                             float sc_log2, f32x16* oacc, float& m_i,
                                             float& l_i) {
  // S^T = K Q^T for the 64 keys (two 32-key tiles).
  f32x16 sacc[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
#pragma unroll
    for (int r = 0; r < 16; ++r) sacc[u][r] = 0.0f;
#pragma unroll
    for (int s = 0; s < 8; ++s)
      sacc[u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(read_k(st, 32 * u + jq, s, hf), qf[s],
                                                       sacc[u], 0, 0, 0);
  }
  // mask keys after the query (causal) or at / past N; branch-free
  const bool need_mask = (MODE != kDenseFull && k0 + kSub - 1 > qw0) || (k0 + kSub > N);
  if (need_mask) {
    const int lim = (MODE == kDenseFull ? N - 1 : min(qrow, N - 1)) - k0 - 4 * hf;
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int kk = 32 * u + 8 * (r >> 2) + (r & 3);
        sacc[u][r] = (kk <= lim) ? sacc[u][r] : -INFINITY;
      }
  }
  uint4 pw[4];   // P^T as bf16, one 16-key MFMA step each
  float lsum;
  auto probs = [&](float mneg) {
    lsum = 0.0f;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int u = s >> 1, base = 8 * (s & 1);
      float p[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        p[e] = __builtin_amdgcn_exp2f(fmaf(sacc[u][base + e], sc_log2, mneg));
        lsum += p[e];
      }
      pw[s] = make_uint4(pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]),
                         pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7]));
    }
  };
  bool kept = false;
  if (__builtin_amdgcn_ballot_w64(m_i == -INFINITY) == 0) {
    probs(-m_i);
    kept = __builtin_amdgcn_ballot_w64(!(lsum <= kFastLimit)) == 0;   // NaN fails too
  }
  if (!kept) {
    float mx = -INFINITY;
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[u][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mcand = mx * sc_log2;
    if (__builtin_amdgcn_ballot_w64(mcand > m_i + kRescaleThreshold) != 0) {
      const float m_new = fmaxf(m_i, mcand);
      const float alpha = (m_new == -INFINITY) ? 1.0f : __builtin_amdgcn_exp2f(m_i - m_new);
      l_i *= alpha;
#pragma unroll
      for (int d = 0; d < 4; ++d)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[d][r] *= alpha;
      m_i = m_new;
    }
    probs((m_i == -INFINITY) ? 0.0f : -m_i);
  }
  l_i += lsum;
  // O^T += V^T P^T
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int s = 0; s < 4; ++s)
      oacc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(read_vt(st, d, s, lane), as_bf16x8(pw[s]),
                                                       oacc[d], 0, 0, 0);
}

// O = O^T / l for the lane's query row, bf16.
__device__ __forceinline__ void store_rows(uint16_t* __restrict__ o, size_t row_base, int hf,
                                           const f32x16* oacc, float l_i) {
  const float l = l_i + __shfl_xor(l_i, 32);
  const float inv = l > 0.0f ? 1.0f / l : 0.0f;
  uint16_t* op = o + row_base * kHeadDim;
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      const int dim = 32 * d + 8 * gq + 4 * hf;
      *(uint2*)(op + dim) =
          make_uint2(pack_bf16x2(oacc[d][4 * gq] * inv, oacc[d][4 * gq + 1] * inv),
                     pack_bf16x2(oacc[d][4 * gq + 2] * inv, oacc[d][4 * gq + 3] * inv));
    }
}

template <int MODE, int SUB>
__global__ __launch_bounds__(kThreads, 2) void attn_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, uint16_t* __restrict__ o, int B, int Hq, int Hkv, int N,
    int n_tiles, int Ls, int CS, int CB, float sc_log2, const int32_t* __restrict__ bidx,
    const int32_t* __restrict__ bcnt, int kmax, uint32_t* __restrict__ sched,
    const XcdPlan plan) {
  // two LDS objects (not one array) so that the compiler can tell the copy
  // into one stage from the reads of the other
  __shared__ __attribute__((aligned(1024))) unsigned char stage0[kStageBytes];
  __shared__ __attribute__((aligned(1024))) unsigned char stage1[kStageBytes];
  __shared__ unsigned s_x, s_idx;   // the persistent workgroup's next item

  const unsigned G = (unsigned)(Hq / Hkv);
  const unsigned total = (unsigned)B * (unsigned)Hq * (unsigned)n_tiles;
  const bool pers = MODE == kSparse && sched != nullptr;
  // this workgroup's XCD (XCC_ID register): its own queue comes first
  const unsigned x0 = pers ? (__builtin_amdgcn_s_getreg((31 << 11) | 20) & (kXcds - 1)) : 0u;
  for (;;) {
    int hh, tile, g, b;
    if (pers) {
      if (threadIdx.x == 0) {
        unsigned xs = kXcds, is = 0;
        for (unsigned d = 0; d < kXcds && xs == kXcds; ++d) {
          const unsigned x = (x0 + d) & (kXcds - 1);
          if (plan.per_x[x] == 0) continue;
          const unsigned t = atomicAdd(&sched[x], 1u);
          if (t < plan.per_x[x]) {
            xs = x;
            is = t;
          }
        }
        s_x = xs;
        s_idx = is;
      }
      // (the previous item's closing barrier keeps this write after every
      // wave's read of the last item)
      __syncthreads();
      const unsigned xs = s_x;
      if (xs == kXcds) return;   // every queue is empty
      unsigned bg;
      plan_item(plan, xs, s_idx, n_tiles, G, (unsigned)(B * Hkv), tile, hh, bg);
      b = (int)(bg / (unsigned)Hkv);
      g = (int)(bg % (unsigned)Hkv);
    } else if (MODE != kSparse) {
      const unsigned per_xcd = gridDim.x / kXcds;
      unsigned t = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
      if (t >= total) return;
      hh = (int)(t % G);
      t /= G;
      tile = n_tiles - 1 - (int)(t % (unsigned)n_tiles);
      t /= (unsigned)n_tiles;
      g = (int)(t % (unsigned)Hkv);
      b = (int)(t / (unsigned)Hkv);
    } else if (((unsigned)B * (unsigned)Hkv) % kXcds == 0) {
      // Tile-major, heavier tiles first; for tile rank t, XCD x takes the KV
      // groups bg with (bg + t / kRotRun) % 8 == x (all G query heads of each):
      // a group stays on one XCD for kRotRun consecutive tiles (which select
      // mostly the same blocks, so they share its L2) and then moves on, so
      // every group's work is spread over all XCDs.
      if (blockIdx.x >= total) return;
      const unsigned x = blockIdx.x % kXcds, idx = blockIdx.x / kXcds;
      const unsigned per_tile = ((unsigned)B * (unsigned)Hq) / kXcds;
      const unsigned tr = idx / per_tile, rem = idx % per_tile;
      tile = n_tiles - 1 - (int)tr;
      hh = (int)(rem % G);
      const unsigned rot = (tr / kRotRun) % kXcds;
      const unsigned bg = (x + kXcds - rot) % kXcds + kXcds * (rem / G);
      b = (int)(bg / (unsigned)Hkv);
      g = (int)(bg % (unsigned)Hkv);
    } else {
      // Tile-major with the (batch, head) index rotated by one per tile.
      if (blockIdx.x >= total) return;
      const unsigned R = (unsigned)B * (unsigned)Hq;
      const unsigned tr = blockIdx.x / R;
      const unsigned r = (blockIdx.x % R + tr) % R;
      tile = n_tiles - 1 - (int)tr;
      b = (int)(r / (unsigned)Hq);
      hh = (int)(r % (unsigned)Hq) % (int)G;
      g = (int)(r % (unsigned)Hq) / (int)G;
    }
    const int h = g * (int)G + hh;

    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int jq = lane & 31, hf = lane >> 5;
    const int q0 = tile * kTileQ;
    const int q_last = min(q0 + kTileQ - 1, N - 1);
    const int qw0 = q0 + wave * 32;          // first query row of this wave
    const int qrow = qw0 + jq;               // this lane's query row

    const uint16_t* kh = k + (size_t)(b * Hkv + g) * N * kHeadDim;
    const uint16_t* vh = v + (size_t)(b * Hkv + g) * N * kHeadDim;

    // Q^T fragments (B operand of S^T = K Q^T), kept in registers.
    bf16x8 qf[8];
    {
      const uint16_t* qp = q + ((size_t)(b * Hq + h) * N + qrow) * kHeadDim + 8 * hf;
  #pragma unroll
      for (int s = 0; s < 8; ++s)
        qf[s] = as_bf16x8(qrow < N ? *(const uint4*)(qp + 16 * s) : make_uint4(0, 0, 0, 0));
    }

    // The sub-blocks to visit.
    const int32_t* lst = nullptr;
    int n_steps;
    if (MODE == kSparse) {
      const int seg = q0 / Ls;
      lst = bidx + ((size_t)(b * Hq + h) * CS + seg) * kmax;
      const int c = min(max(bcnt[(size_t)(b * Hq + h) * CS + seg], 0), kmax);
      n_steps = valid_prefix<SUB>(lst, c, CB, q_last, lane) * SUB;
    } else if (MODE == kDenseCausal) {
      n_steps = q_last / kSub + 1;
    } else {
      n_steps = (N + kSub - 1) / kSub;
    }
    auto step_key0 = [&](int i) -> int {
      if (MODE == kSparse) return (SUB == 1 ? lst[i] : lst[i >> 1] * SUB + (i & 1)) * kSub;
      return i * kSub;
    };

    // byte offsets of this lane's stage copies inside a 64-row block
    uint32_t koff[4], voff[4];
  #pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = 16 * wave + 4 * j + (lane >> 4);
      koff[j] = (uint32_t)(row * kRowBytes + 16 * swz(row, lane & 15));
      voff[j] = (uint32_t)(row * kRowBytes + 16 * swz_v(row, lane & 15));
    }

    f32x16 oacc[4];
  #pragma unroll
    for (int d = 0; d < 4; ++d)
  #pragma unroll
      for (int r = 0; r < 16; ++r) oacc[d][r] = 0.0f;
    float m_i = -INFINITY, l_i = 0.0f;

    // Two-stage LDS ring filled directly from global memory.  Step i waits for
    // its stage (the 8 loads of step i+1 may still be in flight), computes, and
    // after a second barrier refills the stage with step i+2.  Even steps use
    // stage0, odd steps stage1.
    auto step = [&](const int i, unsigned char* st) {
      if (i + 1 < n_steps) EI_WAIT_VMCNT(8); else EI_WAIT_VMCNT(0);
      __syncthreads();
      const int k0 = step_key0(i);
      const bool active = (MODE == kDenseFull) || (k0 <= qw0 + 31);
      if (active && qw0 < N)
        compute_step<MODE>(st, k0, qw0, qrow, N, jq, hf, lane, qf, sc_log2, oacc, m_i, l_i);
      if (i + 2 < n_steps) {
        __syncthreads();   // every wave is done reading this stage
        issue_stage(st, kh, vh, step_key0(i + 2), N, wave, lane, koff, voff);
      }
    };
    // Q fragments (and the list) have landed before any stage copy is issued,
    // so no later wait on them covers the copies in flight.
    EI_WAIT_VMCNT(0);
    if (n_steps > 0) issue_stage(stage0, kh, vh, step_key0(0), N, wave, lane, koff, voff);
    if (n_steps > 1) issue_stage(stage1, kh, vh, step_key0(1), N, wave, lane, koff, voff);
    for (int i = 0; i < n_steps; i += 2) {
      step(i, stage0);
      if (i + 1 < n_steps) step(i + 1, stage1);
    }

    if (qrow < N) store_rows(o, (size_t)(b * Hq + h) * N + qrow, hf, oacc, l_i);
    if (!pers) return;
    __syncthreads();   // every wave is done with the stages (and the item)
  }
}

// The persistent plan for a shape, if its KV groups tile the XCDs.
bool make_plan(const AttnShape& s, int n_tiles, XcdPlan& pl) {
  const unsigned NG = (unsigned)(s.B * s.Hkv), G = (unsigned)(s.Hq / s.Hkv);
  if (NG % kXcds == 0) {
    pl.S = 1;
    pl.ngx = NG / kXcds;
    for (unsigned x = 0; x < kXcds; ++x) pl.per_x[x] = (unsigned)n_tiles * G * pl.ngx;
    return true;
  }
  if (kXcds % NG != 0) return false;
  pl.S = kXcds / NG;
  pl.ngx = 1;
  const unsigned cyc = pl.S * kRun, full = (unsigned)n_tiles / cyc, rem = (unsigned)n_tiles % cyc;
  for (unsigned x = 0; x < kXcds; ++x) {
    const unsigned part = x / NG;
    const unsigned tail = rem > part * kRun ? min(rem - part * kRun, kRun) : 0u;
    pl.per_x[x] = G * (full * kRun + tail);
  }
  return true;
}

// Workgroups of the persistent grid: two per CU of the current device.
int persistent_grid() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    return 0;
  return 2 * cus;
}

template <int MODE, int SUB>
hipError_t launch_t(const uint16_t* q, const uint16_t* k, const uint16_t* v, const AttnShape& s,
                    const int32_t* bidx, const int32_t* bcnt, uint16_t* o, uint32_t* sched,
                    hipStream_t stream) {
  const int n_tiles = (s.N + kTileQ - 1) / kTileQ;
  const int64_t total = (int64_t)s.B * s.Hq * n_tiles;
  int64_t grid = (total + kXcds - 1) / kXcds * kXcds;
  XcdPlan plan{};
  int pgrid = 0;
  if (MODE == kSparse && sched != nullptr && make_plan(s, n_tiles, plan) &&
      (pgrid = persistent_grid()) > 0) {
    hipLaunchKernelGGL(sched_reset_kernel, dim3(1), dim3(kWave), 0, stream, sched);
    grid = grid < pgrid ? grid : (int64_t)pgrid;
  } else {
    sched = nullptr;
  }
  const float sc_log2 = (float)((double)s.softmax_scale * 1.4426950408889634);
  hipLaunchKernelGGL((attn_kernel<MODE, SUB>), dim3((unsigned)grid), dim3(kThreads), 0, stream,
                     q, k, v, o, s.B, s.Hq, s.Hkv, s.N, n_tiles, s.Ls, s.CS, s.CB, sc_log2, bidx,
                     bcnt, s.kmax, sched, plan);
  return hipGetLastError();
}


// ---------------------------------------------------------------------------
// GQA-union tiles.  One workgroup of 8 waves takes the same 128-row query tile
// of two query heads that share a KV head (waves 0-3 the first, 4-7 the
// second).  The heads' block lists are merged into their union (a bitmap over
// the key blocks, compacted in ascending order); each union block is copied
// into LDS once, and the waves of a head that did not select it skip its
// compute while still taking part in the barriers.  Every head visits its own
// blocks in ascending order with compute_step, so the output equals
// attn_kernel's bit for bit.
constexpr int kUnionThreads = 2 * kThreads;
constexpr int kUnionWords = kUnionMaxBlocks / 32;

// Stage copy by 8 waves: wave w moves rows 8 w .. 8 w + 7 of K and of V.
__device__ __forceinline__ void issue_stage8(unsigned char* stage, const uint16_t* __restrict__ kh,
                                             const uint16_t* __restrict__ vh, int k0, int N,
                                             int wave, int lane, const uint32_t* koff,
                                             const uint32_t* voff) {
  const int pos = lane & 15;
  const uint32_t base = (uint32_t)(uintptr_t)stage;
  if (k0 + kSub <= N) {
    const unsigned char* kb = (const unsigned char*)kh + (size_t)k0 * kRowBytes;
    const unsigned char* vb = (const unsigned char*)vh + (size_t)k0 * kRowBytes;
    const uint32_t dst0 =
        base + (uint32_t)(8 * __builtin_amdgcn_readfirstlane(wave) * kRowBytes);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      copy16_to_lds_s(kb, koff[j], dst0 + 4 * j * kRowBytes);
      copy16_to_lds_s(vb, voff[j], dst0 + 4 * j * kRowBytes + kTileBytes);
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int row = 8 * wave + 4 * j + (lane >> 4);
    const int grow = min(k0 + row, N - 1);
    const size_t roff = (size_t)grow * kHeadDim;
    const uint32_t dst = base + (uint32_t)((8 * wave + 4 * j) * kRowBytes);
    copy16_to_lds(kh + roff + 8 * swz(row, pos), __builtin_amdgcn_readfirstlane(dst));
    copy16_to_lds(vh + roff + 8 * swz_v(row, pos),
                  __builtin_amdgcn_readfirstlane(dst + kTileBytes));
  }
}

template <int SUB>
__global__ __launch_bounds__(kUnionThreads, 1) void attn_union_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, uint16_t* __restrict__ o, int B, int Hq, int Hkv, int N,
    int n_tiles, int Ls, int CS, int CB, float sc_log2, const int32_t* __restrict__ bidx,
    const int32_t* __restrict__ bcnt, int kmax) {
  __shared__ __attribute__((aligned(1024))) unsigned char stage0[kStageBytes];
  __shared__ __attribute__((aligned(1024))) unsigned char stage1[kStageBytes];
  __shared__ uint32_t sel_bits[2][kUnionWords];     // the two heads' selected blocks
  __shared__ uint32_t word_off[kUnionWords + 1];    // union entries before each word
  __shared__ uint32_t ulist[2 * kUnionMaxList];     // block | head-0 bit 30 | head-1 bit 31

  // Tile-major, heavier tiles first, the (batch, KV head, pair) index rotated
  // by one per tile.
  const int G = Hq / Hkv, npair = (G + 1) / 2;
  const unsigned R = (unsigned)B * (unsigned)Hkv * (unsigned)npair;
  if (blockIdx.x >= R * (unsigned)n_tiles) return;
  const unsigned tr = blockIdx.x / R;
  const unsigned rr = (blockIdx.x % R + tr) % R;
  const int tile = n_tiles - 1 - (int)tr;
  const int pair = (int)(rr % (unsigned)npair);
  const int bg = (int)(rr / (unsigned)npair);
  const int b = bg / Hkv, g = bg % Hkv;

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int side = wave >> 2, wq = wave & 3;
  const int jq = lane & 31, hf = lane >> 5;
  const bool has_head = 2 * pair + side < G;        // the second side of an odd G is empty
  const int h = g * G + min(2 * pair + side, G - 1);
  const int q0 = tile * kTileQ;
  const int q_last = min(q0 + kTileQ - 1, N - 1);
  const int qw0 = q0 + wq * 32;
  const int qrow = qw0 + jq;

  const uint16_t* kh = k + (size_t)(b * Hkv + g) * N * kHeadDim;
  const uint16_t* vh = v + (size_t)(b * Hkv + g) * N * kHeadDim;

  bf16x8 qf[8];
  {
    const uint16_t* qp = q + ((size_t)(b * Hq + h) * N + qrow) * kHeadDim + 8 * hf;
#pragma unroll
    for (int s = 0; s < 8; ++s)
      qf[s] = as_bf16x8(qrow < N ? *(const uint4*)(qp + 16 * s) : make_uint4(0, 0, 0, 0));
  }

  // The union of the two heads' valid list prefixes, ascending.
  const int seg = q0 / Ls;
  for (int i = tid; i < 2 * kUnionWords; i += kUnionThreads) (&sel_bits[0][0])[i] = 0u;
  __syncthreads();
  for (int sd = 0; sd < 2; ++sd) {
    if (2 * pair + sd >= G) continue;
    const int hs = g * G + 2 * pair + sd;
    const int32_t* lst = bidx + ((size_t)(b * Hq + hs) * CS + seg) * kmax;
    const int c = min(max(bcnt[(size_t)(b * Hq + hs) * CS + seg], 0), kmax);
    const int nv = valid_prefix<SUB>(lst, c, CB, q_last, lane);
    for (int e = tid; e < nv; e += kUnionThreads) {
      const int blk = lst[e];
      atomicOr(&sel_bits[sd][blk >> 5], 1u << (blk & 31));
    }
  }
  __syncthreads();
  const int nw = (CB + 31) / 32;
  if (wave == 0) {
    uint32_t cnt[4], S = 0;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int wd = 4 * lane + t;
      cnt[t] = wd < nw ? (uint32_t)__popc(sel_bits[0][wd] | sel_bits[1][wd]) : 0u;
      S += cnt[t];
    }
    const uint32_t pre = wave_incl_scan_u32(S);
    uint32_t off = pre - S;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      word_off[4 * lane + t] = off;
      off += cnt[t];
    }
    if (lane == kWave - 1) word_off[kUnionWords] = pre;
  }
  __syncthreads();
  for (int wd = tid; wd < nw; wd += kUnionThreads) {
    const uint32_t a = sel_bits[0][wd], c2 = sel_bits[1][wd];
    uint32_t u = a | c2, p = word_off[wd];
    while (u != 0u) {
      const int bit = __builtin_ctz(u);
      u &= u - 1u;
      ulist[p++] = (uint32_t)(32 * wd + bit) | (((a >> bit) & 1u) << 30) |
                   (((c2 >> bit) & 1u) << 31);
    }
  }
  __syncthreads();
  const int n_steps = (int)word_off[kUnionWords] * SUB;
  auto entry = [&](int i) -> uint32_t { return ulist[SUB == 1 ? i : i >> 1]; };
  auto key0 = [&](uint32_t e, int i) -> int {
    const int blk = (int)(e & 0x3fffffffu);
    return (SUB == 1 ? blk : blk * SUB + (i & 1)) * kSub;
  };

  uint32_t koff[2], voff[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int row = 8 * wave + 4 * j + (lane >> 4);
    koff[j] = (uint32_t)(row * kRowBytes + 16 * swz(row, lane & 15));
    voff[j] = (uint32_t)(row * kRowBytes + 16 * swz_v(row, lane & 15));
  }

  f32x16 oacc[4];
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[d][r] = 0.0f;
  float m_i = -INFINITY, l_i = 0.0f;

  // The ring of attn_kernel with four copies per wave and stage.
  auto step = [&](const int i, unsigned char* st) {
    if (i + 1 < n_steps) EI_WAIT_VMCNT(4); else EI_WAIT_VMCNT(0);
    __syncthreads();
    const uint32_t e = entry(i);
    const int k0 = key0(e, i);
    const bool mine = has_head && ((e >> (30 + side)) & 1u) != 0u;
    if (mine && k0 <= qw0 + 31 && qw0 < N)
      compute_step<kSparse>(st, k0, qw0, qrow, N, jq, hf, lane, qf, sc_log2, oacc, m_i, l_i);
    if (i + 2 < n_steps) {
      __syncthreads();   // every wave is done reading this stage
      issue_stage8(st, kh, vh, key0(entry(i + 2), i + 2), N, wave, lane, koff, voff);
    }
  };
  EI_WAIT_VMCNT(0);
  if (n_steps > 0) issue_stage8(stage0, kh, vh, key0(entry(0), 0), N, wave, lane, koff, voff);
  if (n_steps > 1) issue_stage8(stage1, kh, vh, key0(entry(1), 1), N, wave, lane, koff, voff);
  for (int i = 0; i < n_steps; i += 2) {
    step(i, stage0);
    if (i + 1 < n_steps) step(i + 1, stage1);
  }

  if (!has_head || qrow >= N) return;
  store_rows(o, (size_t)(b * Hq + h) * N + qrow, hf, oacc, l_i);
}

template <int SUB>
hipError_t launch_union_t(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                          const AttnShape& s, const int32_t* bidx, const int32_t* bcnt,
                          uint16_t* o, hipStream_t stream) {
  const int n_tiles = (s.N + kTileQ - 1) / kTileQ;
  const int npair = (s.Hq / s.Hkv + 1) / 2;
  const int64_t grid = (int64_t)s.B * s.Hkv * npair * n_tiles;
  const float sc_log2 = (float)((double)s.softmax_scale * 1.4426950408889634);
  hipLaunchKernelGGL((attn_union_kernel<SUB>), dim3((unsigned)grid), dim3(kUnionThreads), 0,
                     stream, q, k, v, o, s.B, s.Hq, s.Hkv, s.N, n_tiles, s.Ls, s.CS, s.CB,
                     sc_log2, bidx, bcnt, s.kmax);
  return hipGetLastError();
}

}  // namespace

bool attention_union_supported(const AttnShape& s) {
  return s.kmax <= kUnionMaxList && s.CB <= kUnionMaxBlocks;
}

hipError_t launch_attention_union(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                  const AttnShape& s, const int32_t* block_idx,
                                  const int32_t* block_cnt, uint16_t* o, hipStream_t stream) {
  if (!attention_union_supported(s)) return hipErrorInvalidValue;
  return s.Lb == 2 * kSub ? launch_union_t<2>(q, k, v, s, block_idx, block_cnt, o, stream)
                          : launch_union_t<1>(q, k, v, s, block_idx, block_cnt, o, stream);
}

hipError_t launch_attention(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                            const AttnShape& s, AttnMode mode, const int32_t* block_idx,
                            const int32_t* block_cnt, uint16_t* o, void* sched_ws,
                            hipStream_t stream) {
  if (s.B * (int64_t)s.Hq * ((s.N + kTileQ - 1) / kTileQ) >= (int64_t)1 << 31)
    return hipErrorInvalidValue;
  uint32_t* sched = (uint32_t*)sched_ws;
  switch (mode) {
    case kSparse:
      return s.Lb == 2 * kSub
                 ? launch_t<kSparse, 2>(q, k, v, s, block_idx, block_cnt, o, sched, stream)
                 : launch_t<kSparse, 1>(q, k, v, s, block_idx, block_cnt, o, sched, stream);
    case kDenseCausal:
      return launch_t<kDenseCausal, 1>(q, k, v, s, nullptr, nullptr, o, nullptr, stream);
    default: return launch_t<kDenseFull, 1>(q, k, v, s, nullptr, nullptr, o, nullptr, stream);
  }
}

}  // namespace ei
