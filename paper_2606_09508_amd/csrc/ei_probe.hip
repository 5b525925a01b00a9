// Entropy probe: Algorithm 1 (min/max representation vectors), Algorithm 2
// (observation attention from the four max/min logit products) and the row
// entropy of Section 4.2, for every (batch, query head, segment).
//
// Exact logits on int8 MFMA.  Every pooled element is a bf16 value.  A pooled
// vector x (128 elements) is written as x = 2^F n + x_r, with F = E - 13 for
// E the binary exponent of max |x_i| (so |n_i| < 2^14), n_i = trunc(x_i 2^-F)
// split into a low limb n_i & 127 (0..127) and a high limb n_i >> 7
// (-128..127), and x_r the part below the grid 2^F (bf16-exact: it holds the
// low bits of x_i).  Elements down to 2^-6 of the vector's maximum lie on the
// grid.  For a query vector q and a key vector k, <q_g, k_g> with
// q_g = 2^Fq n_q is an integer dot product of limbs: four int8 products of
// 128 terms, each exact in int32, combined as
//   T = P00 + 2^7 (P01 + P10) + 2^14 P11      (|T| < 2^36, exact in binary64)
// and <q, k> = 2^(Fq + Fk) T + <q_r, k> + <q_g, k_r>.  The residual part is a
// bf16 MFMA with fp32 accumulation; it runs only for tiles where its bound
// sum|q_r| max|k| + max|q| sum|k_r| can exceed 2^-30 (scaled by probe_scale),
// so a skipped residual moves a logit by less than 2^-30.  Without residuals
// the logits equal the plain binary64 definition up to its own rounding.
//
// Two kernels:
//  pool_kernel   streams K once from HBM, pools each L_B-row key block to its
//                max / min vectors and writes their limbs, residual parts and
//                scales, tiled by 16 blocks in the order the MFMA operands
//                are read.  The same code (pool_item) pools each L_S-row
//                query segment into per-vector records, run by the scores
//                kernel for its own units, so that the stream of Q (the
//                probe's largest read) overlaps the logits.
//  scores_kernel one workgroup of 4 waves per (batch, KV head, 16 query
//                units), a unit being one (query head, segment) of the KV
//                group, segment-major.  Each wave owns 4 units as one
//                16-row MFMA tile (rows: unit, max/min, limb) and streams
//                over the visible key blocks 16 at a time (columns: blocks;
//                the max and the min key vectors are two MFMAs), the key
//                limbs staged once per workgroup in LDS.  Each lane then
//                holds all 4 logits of one (unit, block).  Two passes: the
//                first keeps, per lane and logit row, the running maximum,
//                the argmax (lowest index on ties) and the sum of
//                exp(x - max) over the other entries, merged across the 16
//                lanes of a unit at the end; the second recomputes the
//                logits and writes ln A = ln max((S1+S2)/2, (S3+S4)/2) and
//                accumulates -sum A ln A.  At the entry that is the argmax of
//                both softmaxes of a pair, ln((S_a + S_b)/2) is taken as
//                log1p(-(d_a + d_b)/2) with d = 1 - S[argmax] = rest/(1+rest),
//                which keeps the tiny entropies of near one-hot rows exact.
#include "ei_internal.h"
#include "ei_topk.h"

#include <math.h>

// Both passes must form bitwise the same logits (the argmax's offset from the
// row maximum is then exactly 0): no implicit FMA contraction.
#pragma clang fp contract(off)

namespace ei {
namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kFracBits = 13;                 // F = E - 13, |n| < 2^14
constexpr int kTileBlocks = 16;               // key blocks per MFMA column tile
constexpr int kKLimbTile = 8192;              // bytes: 16 blocks x (max, min) x 2 limbs x 128
constexpr int kKMetaTile = 1024;              // bytes: 16 blocks x (max, min) x 32
constexpr int kKCorrTile = 16384;             // bytes: 16 blocks x (max, min) x (k, k_r) x 128 bf16
constexpr int kQLimb = 2 * kHeadDim;          // bytes per query vector: 2 limbs
constexpr int kQCorr = 2 * kHeadDim;          // bf16 per query vector: q_r then q_g
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.69314718055994531f;

struct QMeta {
  double scale;   // 2^Fq (NaN if the vector has a non-finite element)
  float R;        // sum |q_r|
  float A;        // max |q|
};
struct KMeta {
  double sk;      // sign(probe_scale) 2^Fk (NaN if non-finite)
  double sk14;    // 2^14 sk
  float R;        // sum |k_r|
  float A;        // max |k|
  float pad[2];
};
static_assert(sizeof(QMeta) == 16 && sizeof(KMeta) == 32, "record sizes");

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Pass 1's merged softmax statistics of one (b, h, s) unit, kept by the
// fused probe -> select path between its two kernels.
struct UnitStats {
  double m[2][2];     // maximum logit per (query vector a, key vector b)
  float lse2[2][2];   // log2 (1 + rest): rest = sum of 2^(c2 (x - m)) over the other entries
  float ltop2[2];     // log2 of the pair average at the pair's common argmax
  int jtop[2];        // that common argmax, or -1
};
static_assert(sizeof(UnitStats) == 64, "record size");

struct Layout {   // byte offsets of the probe records inside the workspace
  size_t qlimb, qcorr, qmeta, klimb, kmeta, kcorr, total;
  size_t stats, total_fused;   // fused probe -> select: UnitStats per unit after the rest
};
Layout layout(const ProbeShape& s) {
  const size_t nq = (size_t)s.B * s.Hq * s.CS * 2;   // query vectors
  const size_t nkt = (size_t)s.B * s.Hkv * ((s.CB + kTileBlocks - 1) / kTileBlocks);
  Layout L{};
  size_t o = 0;
  L.qlimb = o; o = align_up(o + nq * kQLimb);
  L.qcorr = o; o = align_up(o + nq * kQCorr * 2);
  L.qmeta = o; o = align_up(o + nq * sizeof(QMeta));
  L.klimb = o; o = align_up(o + nkt * kKLimbTile);
  L.kmeta = o; o = align_up(o + nkt * kKMetaTile);
  L.kcorr = o; o = align_up(o + nkt * kKCorrTile);
  L.total = o;
  L.stats = o; o = align_up(o + (size_t)s.B * s.Hq * s.CS * sizeof(UnitStats));
  L.total_fused = o;
  return L;
}

// ---------------------------------------------------------------------------
// Pooling and the fixed-point split
// ---------------------------------------------------------------------------

constexpr int kPoolThreads = 512;
constexpr int kPoolWaves = kPoolThreads / kWave;

// A 16-byte load marked non-temporal: Q and K are streamed once by the
// probe, and keeping them out of the caches' retained lines leaves the L2 to
// the pooled records the logits re-read (3% on the 128k probe, 15% on the
// Qwen 64k one).
__device__ __forceinline__ uint4 load_nt16(const void* p) {
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 t = __builtin_nontemporal_load((const u32x4*)p);
  return make_uint4(t.x, t.y, t.z, t.w);
}

__device__ __forceinline__ float row16_max(float v) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float row16_sum(float v) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ int row16_or(int v) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) v |= __shfl_xor(v, o);
  return v;
}

// The split of one pooled vector, for the 8 elements (dims 8c .. 8c+7) a lane
// of a 16-lane row holds; every lane of the row returns the vector's scale,
// residual sum and maximum.
struct Split {
  uint32_t lo[2], hi[2];   // int8 limbs, 4 per word
  uint32_t xr[4], xg[4];   // bf16 pairs: below-grid part, grid part
  int F;
  bool nonfinite;
  float R, A;
};

__device__ __forceinline__ uint32_t bf16_bits(float f) { return __float_as_uint(f) >> 16; }

__device__ __forceinline__ Split split_vector(const float* x) {
  Split o;
  float amax = 0.0f;
  int nf = 0;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float ax = fabsf(x[e]);
    nf |= !(ax <= 3.40282347e38f);   // inf or NaN
    amax = fmaxf(amax, ax);
  }
  amax = row16_max(amax);
  nf = row16_or(nf);
  int ex = 0;
  (void)frexpf(amax, &ex);            // amax = m 2^ex, m in [0.5, 1)
  const int F = amax > 0.0f ? ex - 1 - kFracBits : 0;
  float R = 0.0f;
#pragma unroll
  for (int w = 0; w < 2; ++w) { o.lo[w] = 0u; o.hi[w] = 0u; }
#pragma unroll
  for (int e = 0; e < 8; e += 2) {
    float g2[2], r2[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const float v = nf ? 0.0f : x[e + u];
      const int n = (int)truncf(ldexpf(v, -F));          // exact: |v 2^-F| < 2^14
      const float g = ldexpf((float)n, F);                // exact
      const float rr = v - g;                             // exact, bf16-representable
      R += fabsf(rr);
      g2[u] = g;
      r2[u] = rr;
      const int sh = 8 * ((e + u) & 3);
      o.lo[(e + u) >> 2] |= (uint32_t)(n & 127) << sh;
      o.hi[(e + u) >> 2] |= (uint32_t)((n >> 7) & 255) << sh;
    }
    o.xg[e >> 1] = bf16_bits(g2[0]) | (bf16_bits(g2[1]) << 16);
    o.xr[e >> 1] = bf16_bits(r2[0]) | (bf16_bits(r2[1]) << 16);
  }
  o.R = nf ? 0.0f : row16_sum(R);
  o.A = nf ? 0.0f : amax;
  o.F = F;
  o.nonfinite = nf != 0;
  return o;
}

// The records of query segment `item` from its pooled max (lanes 0-15) or
// min (lanes 16-31) vector: limbs, [q_r | q_g] and the scale record.
__device__ __forceinline__ void store_query(const float* x, int64_t item,
                                           unsigned char* __restrict__ ws, const Layout& lay,
                                           int lane) {
  const int c = lane & 15, m = lane >> 4;
  const Split sp = split_vector(x);
  const size_t v = (size_t)item * 2 + m;   // query vector index
  unsigned char* ql = ws + lay.qlimb + v * kQLimb;
  *(uint2*)(ql + 8 * c) = make_uint2(sp.lo[0], sp.lo[1]);
  *(uint2*)(ql + kHeadDim + 8 * c) = make_uint2(sp.hi[0], sp.hi[1]);
  uint16_t* qc = (uint16_t*)(ws + lay.qcorr) + v * kQCorr;
  *(uint4*)(qc + 8 * c) = make_uint4(sp.xr[0], sp.xr[1], sp.xr[2], sp.xr[3]);
  *(uint4*)(qc + kHeadDim + 8 * c) = make_uint4(sp.xg[0], sp.xg[1], sp.xg[2], sp.xg[3]);
  if (c == 0)
    ((QMeta*)(ws + lay.qmeta))[v] =
        QMeta{sp.nonfinite ? (double)NAN : ldexp(1.0, sp.F), sp.R, sp.A};
}

// Folds BL rows (BL chunks of 16 bytes a lane) into the lane's max / min.
template <int BL>
__device__ __forceinline__ void fold_rows(const uint4 (&w)[BL], float (&mx)[8], float (&mn)[8]) {
#pragma unroll
  for (int u = 0; u < BL; ++u) {
    const uint32_t ww[4] = {w[u].x, w[u].y, w[u].z, w[u].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = bf16_lo(ww[e]), hi = bf16_hi(ww[e]);
      mx[2 * e] = fmaxf(mx[2 * e], lo);
      mn[2 * e] = fminf(mn[2 * e], lo);
      mx[2 * e + 1] = fmaxf(mx[2 * e + 1], hi);
      mn[2 * e + 1] = fminf(mn[2 * e + 1], hi);
    }
  }
}

// Four whole query segments (items it[0..3], each L_S = 128 rows, so 32 rows
// a lane) pooled by one wave as one stream of batches of BL loads a lane, NB
// batches in flight (a batch's slot is refilled as soon as it is folded), so
// the stream runs on across segment boundaries; a segment is split and
// written as soon as its last batch is folded.  The segment bases are
// wave-uniform (scalar registers).  Against one segment at a time (two
// round trips of 16 loads each): 1-3% faster probe, same records.
constexpr int kQBatch = 4, kQRing = 4;
__device__ __forceinline__ void pool_query4(const uint16_t* __restrict__ q, int N,
                                            const int64_t (&it)[4], int CS,
                                            unsigned char* __restrict__ ws, const Layout& lay,
                                            int lane) {
  constexpr int BL = kQBatch, NB = kQRing, PER = 32 / BL, NBAT = 4 * PER;
  const int c = lane & 15, ph = lane >> 4;
  const uint32_t loff = (uint32_t)(ph * kHeadDim + 8 * c) * 2u;   // bytes
  const unsigned char* base[4];
#pragma unroll
  for (int t = 0; t < 4; ++t)
    base[t] = (const unsigned char*)(q + ((size_t)(it[t] / CS) * N + (size_t)(it[t] % CS) * 128) *
                                             kHeadDim);
  uint4 w[NB][BL];
  auto issue = [&](int b) {
#pragma unroll
    for (int i = 0; i < BL; ++i)
      w[b % NB][i] = load_nt16(base[b / PER] + loff +
                               (uint32_t)(4 * (BL * (b % PER) + i)) * (kHeadDim * 2u));
  };
  float mx[8], mn[8];
#pragma unroll
  for (int b = 0; b < NB; ++b) issue(b);
#pragma unroll
  for (int b = 0; b < NBAT; ++b) {
    if (b % PER == 0) {
#pragma unroll
      for (int e = 0; e < 8; ++e) { mx[e] = -INFINITY; mn[e] = INFINITY; }
    }
    fold_rows<BL>(w[b % NB], mx, mn);
    if (b + NB < NBAT) issue(b + NB);   // into the slot just folded
    if (b % PER == PER - 1) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        mx[e] = fmaxf(mx[e], __shfl_xor(mx[e], 16));
        mx[e] = fmaxf(mx[e], __shfl_xor(mx[e], 32));
        mn[e] = fminf(mn[e], __shfl_xor(mn[e], 16));
        mn[e] = fminf(mn[e], __shfl_xor(mn[e], 32));
      }
      if (ph < 2) store_query(ph == 0 ? mx : mn, it[b / PER], ws, lay, lane);
    }
  }
}

// One wave per item: a query segment (B*Hq*C_S items) or a key block slot
// (B*Hkv*C_Bt*16 items, C_Bt = ceil(C_B / 16); slots past C_B are written as
// zeros).  Lanes c = lane % 16 hold dims 8c .. 8c+7 of rows of phase
// lane / 16; after the reduction lanes 0-15 split the max vector and lanes
// 16-31 the min vector.
__device__ __forceinline__ void pool_item(const uint16_t* __restrict__ q,
                                          const uint16_t* __restrict__ k, int B, int Hq, int Hkv,
                                          int N, int Ls, int Lb, int CS, int CB, int CBt,
                                          double sgn, unsigned char* __restrict__ ws,
                                          const Layout& lay, int64_t item, int lane) {
  const int64_t nq = (int64_t)B * Hq * CS;
  const bool is_q = item < nq;
  const int64_t head = is_q ? item / CS : (item - nq) / ((int64_t)CBt * kTileBlocks);
  const int grp = (int)(is_q ? item % CS : (item - nq) % ((int64_t)CBt * kTileBlocks));
  const int c = lane & 15;   // 16-byte chunk: dims 8c .. 8c+7
  const int ph = lane >> 4;  // row phase 0..3

  float mx[8], mn[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) { mx[e] = -INFINITY; mn[e] = INFINITY; }
  const bool pad = !is_q && grp >= CB;
  if (!pad) {
    const int L = is_q ? Ls : Lb;
    const int64_t row0 = (int64_t)grp * L;
    const int rows = (int)min((int64_t)L, (int64_t)N - row0);
    const uint16_t* base = (is_q ? q : k) + ((size_t)head * N + row0) * kHeadDim;
    int r = ph;
    // 64 rows (16 loads of 16 bytes per lane) in flight at a time: a query
    // segment of 128 rows takes two round trips to HBM, a key block one
    for (; r + 60 < rows; r += 64) {
      uint4 w[16];
#pragma unroll
      for (int u = 0; u < 16; ++u)
        w[u] = load_nt16(base + (size_t)(r + 4 * u) * kHeadDim + 8 * c);
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const uint32_t ww[4] = {w[u].x, w[u].y, w[u].z, w[u].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float lo = bf16_lo(ww[e]), hi = bf16_hi(ww[e]);
          mx[2 * e] = fmaxf(mx[2 * e], lo);
          mn[2 * e] = fminf(mn[2 * e], lo);
          mx[2 * e + 1] = fmaxf(mx[2 * e + 1], hi);
          mn[2 * e + 1] = fminf(mn[2 * e + 1], hi);
        }
      }
    }
    for (; r < rows; r += 4) {
      const uint4 w = *(const uint4*)(base + (size_t)r * kHeadDim + 8 * c);
      const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float lo = bf16_lo(ww[e]), hi = bf16_hi(ww[e]);
        mx[2 * e] = fmaxf(mx[2 * e], lo);
        mn[2 * e] = fminf(mn[2 * e], lo);
        mx[2 * e + 1] = fmaxf(mx[2 * e + 1], hi);
        mn[2 * e + 1] = fminf(mn[2 * e + 1], hi);
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      mx[e] = fmaxf(mx[e], __shfl_xor(mx[e], 16));
      mx[e] = fmaxf(mx[e], __shfl_xor(mx[e], 32));
      mn[e] = fminf(mn[e], __shfl_xor(mn[e], 16));
      mn[e] = fminf(mn[e], __shfl_xor(mn[e], 32));
    }
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) { mx[e] = 0.0f; mn[e] = 0.0f; }
  }
  if (ph >= 2) return;
  if (is_q) {
    store_query(ph == 0 ? mx : mn, item, ws, lay, lane);
    return;
  }
  const int m = ph;   // 0: max vector, 1: min vector
  const Split sp = split_vector(m == 0 ? mx : mn);
  const uint2 lo = make_uint2(sp.lo[0], sp.lo[1]), hi = make_uint2(sp.hi[0], sp.hi[1]);
  const uint4 xr = make_uint4(sp.xr[0], sp.xr[1], sp.xr[2], sp.xr[3]);
  {
    const int t = grp / kTileBlocks, j = grp % kTileBlocks;
    const size_t tile = (size_t)head * CBt + t;
    // limb l of dims d = 8c .. 8c+7: sub-block ((m, l), d / 64), then lane
    // ((d % 64) / 16) * 16 + j, byte (d % 16)
    unsigned char* kl = ws + lay.klimb + tile * kKLimbTile;
    const int ks = c >> 3, cc = (c & 7) >> 1, e0 = 8 * (c & 1);
    *(uint2*)(kl + ((m * 2 + 0) * 2 + ks) * 1024 + (cc * 16 + j) * 16 + e0) = lo;
    *(uint2*)(kl + ((m * 2 + 1) * 2 + ks) * 1024 + (cc * 16 + j) * 16 + e0) = hi;
    // [k | k_r] as 256 bf16 of one MFMA operand column: element 128 p + d at
    // sub-block (128 p + d) / 32, lane ((d % 32) / 8) * 16 + j
    unsigned char* kc = ws + lay.kcorr + tile * kKCorrTile + m * (kKCorrTile / 2);
    uint4 korig;
    {
      const float* xv = m == 0 ? mx : mn;
      korig = make_uint4(bf16_bits(xv[0]) | (bf16_bits(xv[1]) << 16),
                         bf16_bits(xv[2]) | (bf16_bits(xv[3]) << 16),
                         bf16_bits(xv[4]) | (bf16_bits(xv[5]) << 16),
                         bf16_bits(xv[6]) | (bf16_bits(xv[7]) << 16));
      if (sp.nonfinite) korig = make_uint4(0, 0, 0, 0);
    }
    *(uint4*)(kc + (c >> 2) * 1024 + ((c & 3) * 16 + j) * 16) = korig;
    *(uint4*)(kc + (4 + (c >> 2)) * 1024 + ((c & 3) * 16 + j) * 16) = xr;
    if (c == 0) {
      const double sk = sp.nonfinite ? (double)NAN : sgn * ldexp(1.0, sp.F);
      ((KMeta*)(ws + lay.kmeta + tile * kKMetaTile))[m * kTileBlocks + j] =
          KMeta{sk, sk * 16384.0, sp.R, sp.A, {0.0f, 0.0f}};
    }
  }
}

// One wave per item: a query segment (B*Hq*C_S items, the first) or a key
// block slot (B*Hkv*C_Bt*16 items); item_offset selects where the launch
// starts (the scores kernel pools the query segments it uses itself).
__global__ __launch_bounds__(kPoolThreads) void pool_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, int B, int Hq, int Hkv,
    int N, int Ls, int Lb, int CS, int CB, int CBt, double sgn, unsigned char* __restrict__ ws,
    Layout lay, int64_t item_offset) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t item = item_offset + (int64_t)blockIdx.x * kPoolWaves + (threadIdx.x >> 6);
  const int64_t nq = (int64_t)B * Hq * CS, nk = (int64_t)B * Hkv * CBt * kTileBlocks;
  if (item >= nq + nk) return;
  pool_item(q, k, B, Hq, Hkv, N, Ls, Lb, CS, CB, CBt, sgn, ws, lay, item, lane);
}


// ---------------------------------------------------------------------------
// Logits, softmax statistics, ln A and the entropy
// ---------------------------------------------------------------------------

constexpr int kThreads = 256;                       // 4 waves
// One row tile (4 units) per wave, 16 units per workgroup.  Two row tiles
// per wave share each staged key tile over twice the rows but need ~190
// VGPRs (2 waves per SIMD against 4): 5% slower on the 128k layer.
constexpr int KT = 1;
constexpr int kWaves = kThreads / kWave;
constexpr int kUnits = kWaves * 4 * KT;
constexpr int kStageBytes = kKLimbTile + kKMetaTile;
constexpr int kTilesPerStep = 2;    // key tiles staged per barrier

// What a scores_kernel launch produces:
//  kScoresWrite    ln A and the entropy (ei_entropy_probe);
//  kScoresEntropy  the entropy and each unit's pass-1 statistics, no ln A
//                  (the first kernel of the fused probe -> select);
//  kScoresSelect   from those statistics, pass 2's ln A of the past blocks
//                  into LDS rows, then each unit's top-k selection from LDS
//                  (the second kernel of the fused path).  Same workgroups,
//                  units and per-tile arithmetic as the other two, so every
//                  ln A is bitwise the one kScoresWrite stores.
enum ScoresMode { kScoresWrite = 0, kScoresEntropy = 1, kScoresSelect = 2 };

__device__ __forceinline__ float hw_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float hw_log2(float x) { return __builtin_amdgcn_logf(x); }

// log2((2^u + 2^v) / 2) for u, v <= 0.
__device__ __forceinline__ float log2_pair_avg(float u, float v) {
  const float hi = fmaxf(u, v), lo = fminf(u, v);
  return hi + (hw_log2(1.0f + hw_exp2(lo - hi)) - 1.0f);
}

__device__ __forceinline__ double shfl_xor_f64(double v, int o) {
  const int2 w = __builtin_bit_cast(int2, v);
  return __builtin_bit_cast(double, make_int2(__shfl_xor(w.x, o), __shfl_xor(w.y, o)));
}

// Binary64 logit (in units of 2^Fq |probe_scale|, sign folded into sk) of
// query vector a of the lane's unit against key vector bk of the lane's
// block, from the limb products acc[bk][beta][2 a + alpha].
__device__ __forceinline__ double limb_logit(const i32x4 (&acc)[2][2], int a, int bk,
                                             double sk, double sk14) {
  const int p00 = acc[bk][0][2 * a], p01 = acc[bk][1][2 * a];
  const int p10 = acc[bk][0][2 * a + 1], p11 = acc[bk][1][2 * a + 1];
  const int x = p00 + (p01 + p10) * 128;   // |x| < 2^30
  return fma((double)p11, sk14, (double)x * sk);
}

template <int MODE, int TPS, int SLOTS>
__global__ __launch_bounds__(kThreads, MODE == kScoresSelect ? 1 : 4) void scores_kernel(
    const uint16_t* __restrict__ qsrc, int B, int N, int Ls, int Lb,
    unsigned char* __restrict__ ws, Layout lay, float* __restrict__ log_scores,
    float* __restrict__ entropy, int Hq, int Hkv, int CS, int CB, int CBt, int r, int n_groups,
    int n_chunks, double ps_abs, double sgn, float tau, UnitStats* __restrict__ ustats,
    const int32_t* __restrict__ kblocks, int32_t* __restrict__ idx, int32_t* __restrict__ cnt,
    int kmax, int row_cap) {
  constexpr int kTilesPerStep = TPS;
  __shared__ __attribute__((aligned(16))) unsigned char stage[2][kTilesPerStep * kStageBytes];
  // kScoresSelect: kUnits rows of row_cap scores (dynamic LDS)
  extern __shared__ __attribute__((aligned(16))) float rows_lds[];
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int gq = lane >> 4, col = lane & 15;
  const int wg = blockIdx.x;
  const int chunk = n_chunks - 1 - wg / n_groups;   // heavier chunks first
  const int gi = wg % n_groups;                      // (batch, KV head)
  const int b = gi / Hkv, g = gi % Hkv;
  const int G = Hq / Hkv;
  const int U = G * CS;
  const int u0 = chunk * kUnits;
  const int ulast = min(u0 + kUnits - 1, U - 1);
  const int nv_max = min((ulast / G + 1) * r, CB);
  // kScoresSelect visits the past blocks only (the segments' own blocks are
  // always kept): up to the last unit's s r, possibly none
  const int nt = MODE == kScoresSelect ? ((ulast / G) * r + kTileBlocks - 1) / kTileBlocks
                                       : (nv_max + kTileBlocks - 1) / kTileBlocks;

  const QMeta* qmeta = (const QMeta*)(ws + lay.qmeta);
  const unsigned char* qlimb = ws + lay.qlimb;
  const uint16_t* qcorr = (const uint16_t*)(ws + lay.qcorr);
  const unsigned char* klimb = ws + lay.klimb + (size_t)gi * CBt * kKLimbTile;
  const unsigned char* kmeta = ws + lay.kmeta + (size_t)gi * CBt * kKMetaTile;
  const unsigned char* kcorr = ws + lay.kcorr + (size_t)gi * CBt * kKCorrTile;

  auto unit_row = [&](int u) -> int64_t {   // (b, h, s) row of unit u
    const int s = u / G, hh = u % G;
    return ((int64_t)(b * Hq + g * G + hh)) * CS + s;
  };

  // The query segments of the workgroup's own units are pooled here (only
  // this workgroup reads their records, after the barrier), so that their
  // HBM reads overlap the logits of the CU's other workgroups; the key blocks
  // are pooled beforehand by pool_kernel.  kScoresSelect reads the records
  // its kScoresEntropy launch wrote.
  if constexpr (MODE != kScoresSelect) {
    const int uw = u0 + 4 * KT * __builtin_amdgcn_readfirstlane(wave);
    // whole segments: L_S = 128 and the wave's last unit's segment ends by N
    if (KT == 1 && Ls == 128 && uw + 3 < U && (int64_t)((uw + 3) / G + 1) * 128 <= N) {
      const int64_t it[4] = {unit_row(uw), unit_row(uw + 1), unit_row(uw + 2), unit_row(uw + 3)};
      pool_query4(qsrc, N, it, CS, ws, lay, lane);
    } else {
      for (int t = 0; t < 4 * KT; ++t) {
        const int u = uw + t;
        if (u < U)
          pool_item(qsrc, nullptr, B, Hq, Hkv, N, Ls, Lb, CS, CB, CBt, sgn, ws, lay, unit_row(u),
                    lane);
      }
    }
    __syncthreads();
  }

  // This lane's units (D rows 4 gq .. 4 gq + 3 of each tile): row, visible
  // blocks (0 for a unit past the group's last), per query vector a the
  // log2-unit scale c2 and the residual factor iq = sign / 2^Fq.
  int64_t urow[KT];
  int nv[KT];
  float c2[KT][2];
  double iq[KT][2];
  float Aqm[KT], Rqm[KT];
  // A operands: row i = col holds (unit i / 4, vector (i >> 1) & 1, limb i & 1)
  i32x4 aop[KT][2];
#pragma unroll
  for (int kt = 0; kt < KT; ++kt) {
    const int u = u0 + 4 * KT * wave + 4 * kt + gq;
    const bool uv = u < U;
    urow[kt] = uv ? unit_row(u) : 0;
    nv[kt] = uv ? min((u / G + 1) * r, CB) : 0;
    float am = 0.0f, rm = 0.0f;
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const QMeta qm = uv ? qmeta[urow[kt] * 2 + a] : QMeta{1.0, 0.0f, 0.0f};
      c2[kt][a] = ps_abs == 0.0 ? 1.0f : (float)(ps_abs * qm.scale * (double)kLog2e);
      iq[kt][a] = sgn / qm.scale;
      am = fmaxf(am, qm.A);
      rm = fmaxf(rm, qm.R);
    }
    am = fmaxf(am, __shfl_xor(am, 16));
    am = fmaxf(am, __shfl_xor(am, 32));
    rm = fmaxf(rm, __shfl_xor(rm, 16));
    rm = fmaxf(rm, __shfl_xor(rm, 32));
    Aqm[kt] = am;
    Rqm[kt] = rm;
    const int ui = u0 + 4 * KT * wave + 4 * kt + (col >> 2);
    const int a = (col >> 1) & 1, al = col & 1;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      aop[kt][ks] = i32x4{0, 0, 0, 0};
      if (ui < U)
        aop[kt][ks] = *(const i32x4*)(qlimb + (size_t)(unit_row(ui) * 2 + a) * kQLimb +
                                      al * kHeadDim + 64 * ks + 16 * gq);
    }
  }

  // The residual part of the 16 logits per row of tile kt and key tile t, if
  // its bound can reach tau: bf16 MFMA with rows (unit, vector, 0 / pad) and
  // the operand [q_r | q_g] . [k | k_r].  corr[bk][2 a] is the lane's value.
  // A half whose bound is zero (no residual bits in the row tile's query
  // vectors, or in the tile's key vectors) only adds exact zeros and is
  // skipped; do_q / do_k are wave-uniform.
  auto residual = [&](int kt, int t, f32x4 (&corr)[2], bool do_q, bool do_k) {
    corr[0] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    corr[1] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    const int ui = u0 + 4 * KT * wave + 4 * kt + (col >> 2);
    const int a = (col >> 1) & 1;
    const bool has = ui < U && (col & 1) == 0;
    const uint16_t* qc = qcorr + (has ? (size_t)(unit_row(ui) * 2 + a) * kQCorr : 0);
    // the tile's base is wave-uniform: only 32-bit lane offsets in vector registers
    const unsigned char* kc =
        kcorr + (size_t)__builtin_amdgcn_readfirstlane(t) * kKCorrTile;
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      if (kk < 4 ? !do_q : !do_k) continue;   // kk 0-3: <q_r, k>; 4-7: <q_g, k_r>
      const uint4 qa = has ? *(const uint4*)(qc + 32 * kk + 8 * gq) : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int bk = 0; bk < 2; ++bk) {
        const uint32_t off = (uint32_t)(bk * (kKCorrTile / 2) + kk * 1024) + (uint32_t)lane * 16u;
        const uint4 kb = *(const uint4*)(kc + off);
        corr[bk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, qa),
                                                          __builtin_bit_cast(bf16x8, kb),
                                                          corr[bk], 0, 0, 0);
      }
    }
  };

  // Per tile: the staged key limbs and records, then for each row tile the
  // eight limb MFMAs and the lane's four logits.
  auto tile_logits = [&](const unsigned char* st, int t, int kt, double (&x)[2][2]) {
    i32x4 acc[2][2];
#pragma unroll
    for (int bk = 0; bk < 2; ++bk)
#pragma unroll
      for (int be = 0; be < 2; ++be) {
        acc[bk][be] = i32x4{0, 0, 0, 0};
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const i32x4 bo = *(const i32x4*)(st + ((bk * 2 + be) * 2 + ks) * 1024 + lane * 16);
          acc[bk][be] =
              __builtin_amdgcn_mfma_i32_16x16x64_i8(aop[kt][ks], bo, acc[bk][be], 0, 0, 0);
        }
      }
    const KMeta* km = (const KMeta*)(st + kKLimbTile);
    const KMeta k0 = km[col], k1 = km[kTileBlocks + col];
    const bool need = fmaf(k0.R, Aqm[kt], k0.A * Rqm[kt]) > tau ||
                      fmaf(k1.R, Aqm[kt], k1.A * Rqm[kt]) > tau;
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      x[a][0] = limb_logit(acc, a, 0, k0.sk, k0.sk14);
      x[a][1] = limb_logit(acc, a, 1, k1.sk, k1.sk14);
    }
    if (__builtin_amdgcn_ballot_w64(need) != 0) {
      f32x4 corr[2];
      residual(kt, t, corr, __builtin_amdgcn_ballot_w64(Rqm[kt] > 0.0f) != 0,
               __builtin_amdgcn_ballot_w64(k0.R > 0.0f || k1.R > 0.0f) != 0);
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int bk = 0; bk < 2; ++bk) x[a][bk] = fma((double)corr[bk][2 * a], iq[kt][a], x[a][bk]);
    }
  };

  // Key tile staging: two LDS buffers of kTilesPerStep tiles each, the next
  // step's tiles held in registers (a slot past the last tile repeats the
  // last tile, unread).
  i32x4 p0[kTilesPerStep], p1[kTilesPerStep], pm[kTilesPerStep];
  const int n_steps = (nt + kTilesPerStep - 1) / kTilesPerStep;
  auto load_step = [&](int i) {
#pragma unroll
    for (int k = 0; k < kTilesPerStep; ++k) {
      const int t = min(kTilesPerStep * i + k, nt - 1);
      const i32x4* src = (const i32x4*)(klimb + (size_t)t * kKLimbTile);
      p0[k] = src[tid];
      p1[k] = src[kThreads + tid];
      if (tid < kKMetaTile / 16) pm[k] = ((const i32x4*)(kmeta + (size_t)t * kKMetaTile))[tid];
    }
  };
  auto store_step = [&](int buf) {
#pragma unroll
    for (int k = 0; k < kTilesPerStep; ++k) {
      i32x4* dst = (i32x4*)(stage[buf] + k * kStageBytes);
      dst[tid] = p0[k];
      dst[kThreads + tid] = p1[k];
      if (tid < kKMetaTile / 16) dst[kKLimbTile / 16 + tid] = pm[k];
    }
  };

  // pass 1 state per row tile, query vector a and key vector bk
  double m_[KT][2][2];
  float rest_[KT][2][2];
  int bj_[KT][2][2];
#pragma unroll
  for (int kt = 0; kt < KT; ++kt)
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int bk = 0; bk < 2; ++bk) {
        m_[kt][a][bk] = -1.7976931348623157e308;   // a phantom entry whose weight is 0
        rest_[kt][a][bk] = 0.0f;
        bj_[kt][a][bk] = 0x7fffffff;
      }
  // pass 1's merged statistics, as pass 2 uses them
  float lse2[KT][2][2], ltop2[KT][2];
  int jtop[KT][2];

  // tiles below nv_min are visible to every unit of the workgroup (when all
  // its units exist: a unit past the group's last has no row at all)
  const int nv_min = u0 + kUnits <= U ? min((u0 / G + 1) * r, CB) : 0;
  if constexpr (MODE != kScoresSelect) {
  load_step(0);
  store_step(0);
  if (n_steps > 1) load_step(1);
  __syncthreads();
  for (int i = 0; i < n_steps; ++i) {
#pragma unroll
  for (int k = 0; k < kTilesPerStep; ++k) {
    const int t = kTilesPerStep * i + k;
    if (t >= nt) continue;
    const unsigned char* st = stage[i & 1] + k * kStageBytes;
    const int j = kTileBlocks * t + col;
    const bool whole = kTileBlocks * (t + 1) <= nv_min;   // workgroup-uniform
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
      double x[2][2];
      tile_logits(st, t, kt, x);
      if (!whole) {
        const bool v = j < nv[kt];
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int bk = 0; bk < 2; ++bk) x[a][bk] = v ? x[a][bk] : -INFINITY;
      }
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int bk = 0; bk < 2; ++bk) {
          const double xv = x[a][bk];
          double& m = m_[kt][a][bk];
          float& rs = rest_[kt][a][bk];
          const bool gt = xv > m;
          const float e = hw_exp2(-fabsf((float)(xv - m)) * c2[kt][a]);
          rs = gt ? fmaf(rs, e, e) : rs + e;
          m = gt ? xv : m;   // a NaN logit leaves m (its weight makes rest NaN)
          bj_[kt][a][bk] = gt ? j : bj_[kt][a][bk];
        }
    }
  }
    if (i + 1 < n_steps) {
      store_step((i + 1) & 1);
      if (i + 2 < n_steps) load_step(i + 2);
    }
    __syncthreads();
  }

  // merge the 16 lanes of each unit: max, lowest argmax, and the other
  // entries' weight relative to the max
#pragma unroll
  for (int kt = 0; kt < KT; ++kt) {
    float dfc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int bk = 0; bk < 2; ++bk) {
        double m = m_[kt][a][bk];
        float rs = rest_[kt][a][bk];
        int jj = bj_[kt][a][bk];
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
          const double m2 = shfl_xor_f64(m, o);
          const float r2 = __shfl_xor(rs, o);
          const int j2 = __shfl_xor(jj, o);
          const bool w1 = m > m2 || (m == m2 && jj < j2);
          const double mw = w1 ? m : m2, ml = w1 ? m2 : m;
          const float rw = w1 ? rs : r2, rl = w1 ? r2 : rs;
          rs = fmaf(rl + 1.0f, hw_exp2(-(float)(mw - ml) * c2[kt][a]), rw);
          m = mw;
          jj = w1 ? jj : j2;
        }
        m_[kt][a][bk] = m;
        bj_[kt][a][bk] = jj;
        lse2[kt][a][bk] = log1pf(rs) * kLog2e;
        dfc[a][bk] = rs / (1.0f + rs);
      }
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      jtop[kt][a] = bj_[kt][a][0] == bj_[kt][a][1] ? bj_[kt][a][0] : -1;
      ltop2[kt][a] = log1pf(-0.5f * (dfc[a][0] + dfc[a][1])) * kLog2e;
    }
    if (MODE == kScoresEntropy && col == 0 && nv[kt] > 0) {
      UnitStats us;
#pragma unroll
      for (int a = 0; a < 2; ++a) {
#pragma unroll
        for (int bk = 0; bk < 2; ++bk) {
          us.m[a][bk] = m_[kt][a][bk];
          us.lse2[a][bk] = lse2[kt][a][bk];
        }
        us.ltop2[a] = ltop2[kt][a];
        us.jtop[a] = jtop[kt][a];
      }
      ustats[urow[kt]] = us;
    }
  }
  } else {
    // the statistics kept by the kScoresEntropy launch
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
      UnitStats us{};
      if (nv[kt] > 0) us = ustats[urow[kt]];
#pragma unroll
      for (int a = 0; a < 2; ++a) {
#pragma unroll
        for (int bk = 0; bk < 2; ++bk) {
          m_[kt][a][bk] = us.m[a][bk];
          lse2[kt][a][bk] = us.lse2[a][bk];
        }
        ltop2[kt][a] = us.ltop2[a];
        jtop[kt][a] = us.jtop[a];
      }
    }
  }

  // pass 2: ln A and the entropy (kScoresSelect: ln A of the past blocks into
  // the units' LDS rows)
  int np[KT];   // past blocks s r of the lane's unit (0 for a missing unit)
#pragma unroll
  for (int kt = 0; kt < KT; ++kt) np[kt] = nv[kt] > 0 ? (int)(urow[kt] % CS) * r : 0;
  float H2[KT];
#pragma unroll
  for (int kt = 0; kt < KT; ++kt) H2[kt] = 0.0f;
  if (n_steps > 0) {
    load_step(0);
    store_step(0);
    if (n_steps > 1) load_step(1);
    __syncthreads();
  }
  for (int i = 0; i < n_steps; ++i) {
#pragma unroll
  for (int k = 0; k < kTilesPerStep; ++k) {
    const int t = kTilesPerStep * i + k;
    if (t >= nt) continue;
    const unsigned char* st = stage[i & 1] + k * kStageBytes;
    const int j = kTileBlocks * t + col;
    const bool whole = kTileBlocks * (t + 1) <= nv_min;   // workgroup-uniform
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
      double x[2][2];
      tile_logits(st, t, kt, x);
      float l2[2];
#pragma unroll
      for (int a = 0; a < 2; ++a) {
        float ls[2];
#pragma unroll
        for (int bk = 0; bk < 2; ++bk)
          ls[bk] = fmaf((float)(x[a][bk] - m_[kt][a][bk]), c2[kt][a], -lse2[kt][a][bk]);
        float lp = log2_pair_avg(ls[0], ls[1]);
        asm volatile("" : "+v"(lp));   // formed for every lane, then selected
        l2[a] = j == jtop[kt][a] ? ltop2[kt][a] : lp;
      }
      const float L2 = l2[0] > l2[1] ? l2[0] : l2[1];
      if constexpr (MODE == kScoresSelect) {
        if (j < np[kt]) rows_lds[(4 * KT * wave + 4 * kt + gq) * row_cap + j] = L2 * kLn2;
      } else {
        const float h = hw_exp2(L2) * L2;
        float* dst = log_scores + urow[kt] * CB + j;
        if (whole || j < nv[kt]) {
          if constexpr (MODE == kScoresWrite) *dst = L2 * kLn2;
          H2[kt] += h;
        }
      }
    }
  }
    if (i + 1 < n_steps) {
      store_step((i + 1) & 1);
      if (i + 2 < n_steps) load_step(i + 2);
    }
    __syncthreads();
  }
  if constexpr (MODE != kScoresSelect) {
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
      const float h = row16_sum(H2[kt]);
      if (col == 0 && nv[kt] > 0) entropy[urow[kt]] = -h * kLn2;
    }
  } else {
    // Top-k of each of the wave's units from its LDS row (written by this
    // wave; the barrier above ordered the writes), with the stage buffers,
    // free after that barrier, as the selection's histogram and candidates.
    static_assert(kWaves * (topk::kHistWords + topk::kCandWords) * 4 <= sizeof(stage),
                  "top-k scratch must fit the stage buffers");
    const int wv = __builtin_amdgcn_readfirstlane(wave);
    uint32_t* hist = (uint32_t*)&stage[0][0] + wv * (topk::kHistWords + topk::kCandWords);
    uint32_t* cand = hist + topk::kHistWords;
    for (int ul = 4 * KT * wv; ul < 4 * KT * (wv + 1); ++ul) {
      const int u = u0 + ul;
      if (u >= U) break;
      const int64_t row = unit_row(u);
      const float* rl = rows_lds + ul * row_cap;
      topk::select_row<SLOTS>([&](int jj) { return rl[jj]; }, row_cap, u / G, r, CB, kmax,
                              kblocks[row],
                              idx + row * (int64_t)kmax, cnt + row, hist, cand, lane);
    }
  }
}

}  // namespace

size_t probe_workspace_bytes(const ProbeShape& s) { return layout(s).total; }
size_t probe_select_workspace_bytes(const ProbeShape& s) { return layout(s).total_fused; }

bool probe_supported(const ProbeShape& s) {
  (void)s;
  return true;
}

namespace {

// The fused path's LDS rows hold the past blocks of kUnits units: row_cap
// floats each, a multiple of 64 plus 16 so that the four units of a wave
// write disjoint banks.
constexpr int kFusedMaxPast = 32 * kWave;    // the 32-slot selector's longest row
int fused_row_cap(const ProbeShape& s) { return ((s.CS - 1) * s.r + 63) / 64 * 64 + 16; }
size_t fused_lds_bytes(const ProbeShape& s) { return (size_t)kUnits * fused_row_cap(s) * 4; }
constexpr size_t kLdsBytes = 160 * 1024;
constexpr size_t kFusedStaticLds = 2 * kStageBytes;   // stage buffers of the TPS = 1 instance

// The key blocks only (the scores kernels pool the query segments).
hipError_t launch_pool(const uint16_t* q, const uint16_t* k, const ProbeShape& s, double sgn,
                       unsigned char* ws, const Layout& lay, int CBt, hipStream_t stream) {
  const int64_t nq = (int64_t)s.B * s.Hq * s.CS;
  const int64_t items = (int64_t)s.B * s.Hkv * CBt * kTileBlocks;
  const int64_t grid = (items + kPoolWaves - 1) / kPoolWaves;
  hipLaunchKernelGGL(pool_kernel, dim3((unsigned)grid), dim3(kPoolThreads), 0, stream, q, k, s.B,
                     s.Hq, s.Hkv, s.N, s.Ls, s.Lb, s.CS, s.CB, CBt, sgn, ws, lay, nq);
  return hipGetLastError();
}

template <int SLOTS>
hipError_t launch_fused_select(const ProbeShape& s, const Layout& lay, unsigned char* ws,
                               int CBt, int n_groups, int n_chunks, double ps_abs, double sgn,
                               float tau, const int32_t* kblocks, int32_t* idx, int32_t* cnt,
                               int kmax, hipStream_t stream) {
  auto kern = scores_kernel<kScoresSelect, 1, SLOTS>;
  const size_t lds = fused_lds_bytes(s);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3((unsigned)((int64_t)n_groups * n_chunks)), dim3(kThreads), lds,
                     stream, nullptr, s.B, s.N, s.Ls, s.Lb, ws, lay, nullptr, nullptr, s.Hq, s.Hkv,
                     s.CS, s.CB, CBt, s.r,
                     n_groups, n_chunks, ps_abs, sgn, tau, (UnitStats*)(ws + lay.stats), kblocks,
                     idx, cnt, kmax, fused_row_cap(s));
  return hipGetLastError();
}

}  // namespace

bool probe_select_supported(const ProbeShape& s) {
  return (s.CS - 1) * s.r <= kFusedMaxPast && fused_lds_bytes(s) + kFusedStaticLds <= kLdsBytes;
}

hipError_t launch_probe(const uint16_t* q, const uint16_t* k, const ProbeShape& s,
                        double probe_scale, float* log_scores, float* entropy, void* workspace,
                        hipStream_t stream) {
  const Layout lay = layout(s);
  unsigned char* ws = (unsigned char*)workspace;
  const int CBt = (s.CB + kTileBlocks - 1) / kTileBlocks;
  const double sgn = probe_scale > 0.0 ? 1.0 : (probe_scale < 0.0 ? -1.0 : 0.0);
  hipError_t e = launch_pool(q, k, s, sgn, ws, lay, CBt, stream);
  if (e != hipSuccess) return e;
  const int G = s.Hq / s.Hkv;
  const int n_groups = s.B * s.Hkv;
  const int n_chunks = (G * s.CS + kUnits - 1) / kUnits;
  const double ps_abs = fabs(probe_scale);
  // skip the residual MFMA where it moves no logit by 2^-30 or more
  const float tau = probe_scale == 0.0 ? INFINITY : (float)(0x1p-30 / ps_abs);
  hipLaunchKernelGGL((scores_kernel<kScoresWrite, kTilesPerStep, 1>),
                     dim3((unsigned)((int64_t)n_groups * n_chunks)), dim3(kThreads), 0, stream,
                     q, s.B, s.N, s.Ls, s.Lb, ws, lay, log_scores, entropy, s.Hq, s.Hkv, s.CS,
                     s.CB, CBt, s.r, n_groups,
                     n_chunks, ps_abs, sgn, tau, nullptr, nullptr, nullptr, nullptr, 0, 0);
  return hipGetLastError();
}

hipError_t launch_probe_select(const uint16_t* q, const uint16_t* k, const ProbeShape& s,
                               double probe_scale, const SelectShape& ss, float* entropy,
                               uint8_t* rigid, int32_t* budget_blocks, int32_t* block_idx,
                               int32_t* block_cnt, void* workspace, hipStream_t stream) {
  const Layout lay = layout(s);
  unsigned char* ws = (unsigned char*)workspace;
  const int CBt = (s.CB + kTileBlocks - 1) / kTileBlocks;
  const double sgn = probe_scale > 0.0 ? 1.0 : (probe_scale < 0.0 ? -1.0 : 0.0);
  hipError_t e = launch_pool(q, k, s, sgn, ws, lay, CBt, stream);
  if (e != hipSuccess) return e;
  const int G = s.Hq / s.Hkv;
  const int n_groups = s.B * s.Hkv;
  const int n_chunks = (G * s.CS + kUnits - 1) / kUnits;
  const double ps_abs = fabs(probe_scale);
  const float tau = probe_scale == 0.0 ? INFINITY : (float)(0x1p-30 / ps_abs);
  // entropies and each unit's statistics, no ln A
  hipLaunchKernelGGL((scores_kernel<kScoresEntropy, kTilesPerStep, 1>),
                     dim3((unsigned)((int64_t)n_groups * n_chunks)), dim3(kThreads), 0, stream,
                     q, s.B, s.N, s.Ls, s.Lb, ws, lay, nullptr, entropy, s.Hq, s.Hkv, s.CS,
                     s.CB, CBt, s.r, n_groups,
                     n_chunks, ps_abs, sgn, tau, (UnitStats*)(ws + lay.stats), nullptr, nullptr,
                     nullptr, 0, 0);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // classification and budgets (Algorithm 3) from the entropies
  if ((e = launch_budget(entropy, ss, rigid, budget_blocks, stream)) != hipSuccess) return e;
  // ln A again, into LDS, and the top-k from there
  if ((s.CS - 1) * s.r <= 8 * kWave)
    return launch_fused_select<8>(s, lay, ws, CBt, n_groups, n_chunks, ps_abs, sgn, tau,
                                  budget_blocks, block_idx, block_cnt, ss.kmax, stream);
  return launch_fused_select<32>(s, lay, ws, CBt, n_groups, n_chunks, ps_abs, sgn, tau,
                                 budget_blocks, block_idx, block_cnt, ss.kmax, stream);
}

}  // namespace ei
