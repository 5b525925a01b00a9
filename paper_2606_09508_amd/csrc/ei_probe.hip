// Entropy probe: Algorithm 1 (min/max representation vectors), Algorithm 2
// (observation attention from the four max/min logit products) and the row
// entropy of Section 4.2, for every (batch, query head, segment).
//
// Two kernels:
//  pool_kernel    streams Q and K once from HBM (the bound of the probe) and
//                 writes Q_max/Q_min per segment in binary64 (so the scores
//                 kernel can read them as uniform scalar operands) and
//                 K_max/K_min per key block in fp32 (exact: pooled values are
//                 input values; one convert to binary64 per use), tiled by 64
//                 blocks: [head][j / 64][max|min][d / 4][j % 64][4], so that
//                 the scores kernel's loads (lane = block, 4 dims per load)
//                 read 1 KB contiguous per wave instruction.
//  scores_kernel  one workgroup per (b, KV head, segment, chunk of query
//                 heads).  Each lane owns one visible key block and forms the
//                 4 logits of every query head of the chunk in binary64 FMA
//                 (products of bf16 values are exact, so the logits equal the
//                 plain definition's); the query representation is staged in
//                 LDS and read with broadcast loads (in-order completion, so
//                 they pipeline, unlike scalar loads); the kernel keeps fp32
//                 offsets from a per-wave reference in LDS; then one wave per
//                 logit row finds the
//                 row's maximum, argmax and log-sum-exp, and the waves of
//                 each head evaluate A = max((S1+S2)/2, (S3+S4)/2) and
//                 H = -sum A ln A in log space (fp32 terms, fp64 sums).
#include "ei_internal.h"

#include <math.h>

namespace ei {
namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / kWave;

// K representation tile: 64 blocks x (max, min) x 128 dims in fp32.
constexpr int kKTileBlocks = 64;
constexpr int kKTileFloats = kKTileBlocks * 2 * kHeadDim;
__host__ __device__ inline int padded_blocks(int CB) {
  return (CB + kKTileBlocks - 1) / kKTileBlocks * kKTileBlocks;
}
// Offset (floats) of block j's value for dims 4 dq .. 4 dq + 3 of part m
// (0 = max, 1 = min) inside one head's K representation.
__host__ __device__ inline size_t krep_offset(int j, int m, int dq) {
  return (size_t)(j / kKTileBlocks) * kKTileFloats +
         (size_t)((m * (kHeadDim / 4) + dq) * kKTileBlocks + j % kKTileBlocks) * 4;
}

__global__ __launch_bounds__(kThreads) void pool_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, int B, int Hq, int Hkv,
    int N, int Ls, int Lb, int CS, int CB, double* __restrict__ qrep,
    float* __restrict__ krep) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t item = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
  const int64_t nq = (int64_t)B * Hq * CS, nk = (int64_t)B * Hkv * CB;
  if (item >= nq + nk) return;
  const bool is_q = item < nq;
  const int64_t head = is_q ? item / CS : (item - nq) / CB;
  const int grp = (int)(is_q ? item % CS : (item - nq) % CB);
  const int L = is_q ? Ls : Lb;
  const int64_t row0 = (int64_t)grp * L;
  const int rows = (int)min((int64_t)L, (int64_t)N - row0);
  const uint16_t* base = (is_q ? q : k) + ((size_t)head * N + row0) * kHeadDim;

  const int c = lane & 15;   // 16-byte chunk: dims 8c .. 8c+7
  const int ph = lane >> 4;  // row phase 0..3
  float mx[8], mn[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) { mx[e] = -INFINITY; mn[e] = INFINITY; }

  int r = ph;
  for (; r + 12 < rows; r += 16) {
    uint4 w[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      w[u] = *(const uint4*)(base + (size_t)(r + 4 * u) * kHeadDim + 8 * c);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
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
  if (ph != 0) return;
  if (is_q) {
    double* out = qrep + ((size_t)head * CS + grp) * 2 * kHeadDim + 8 * c;
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      *(double2*)(out + e) = make_double2((double)mx[e], (double)mx[e + 1]);
      *(double2*)(out + kHeadDim + e) = make_double2((double)mn[e], (double)mn[e + 1]);
    }
  } else {
    float* out = krep + (size_t)head * padded_blocks(CB) * 2 * kHeadDim;
    *(float4*)(out + krep_offset(grp, 0, 2 * c)) = make_float4(mx[0], mx[1], mx[2], mx[3]);
    *(float4*)(out + krep_offset(grp, 0, 2 * c + 1)) = make_float4(mx[4], mx[5], mx[6], mx[7]);
    *(float4*)(out + krep_offset(grp, 1, 2 * c)) = make_float4(mn[0], mn[1], mn[2], mn[3]);
    *(float4*)(out + krep_offset(grp, 1, 2 * c + 1)) = make_float4(mn[4], mn[5], mn[6], mn[7]);
  }
}

__device__ __forceinline__ void widen4(const float4 w, double* out) {
  out[0] = (double)w.x;
  out[1] = (double)w.y;
  out[2] = (double)w.z;
  out[3] = (double)w.w;
}

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.69314718055994531f;

// e^x and ln(1 + y) for y in [0, 1] on the hardware exp2 / log2 (relative
// error ~1e-7 for the arguments used here; the one entry per row that needs
// ln of a value near 1 is evaluated in binary64 instead).
__device__ __forceinline__ float fast_exp(float x) { return __builtin_amdgcn_exp2f(x * kLog2e); }
__device__ __forceinline__ float fast_log1p01(float y) { return __builtin_amdgcn_logf(1.0f + y) * kLn2; }

// ln((exp(a) + exp(b)) / 2) for a, b <= 0, not both near 0.
__device__ __forceinline__ float log_pair_avg(float a, float b) {
  const float hi = fmaxf(a, b), lo = fminf(a, b);
  return hi + fast_log1p01(fast_exp(lo - hi)) - kLn2;
}

// Per-row statistics of the four softmaxes, kept in LDS between phases.
struct RowStats {
  float M;       // max of the per-wave references
  float best;    // largest offset (the argmax's)
  int bj;        // argmax (lowest index among equal offsets)
  float lse;     // log1p(rest), rest = sum over j != argmax of exp(x_j - x_argmax)
  double dfc;    // 1 - S[argmax] = rest / (1 + rest)
};

// HPW query heads per workgroup of NT threads; rows of the score block: the 4
// logit products (S1..S4) of each head.
template <int HPW, int NT>
__global__ __launch_bounds__(NT) void scores_kernel(
    const double* __restrict__ qrep, const float* __restrict__ krep,
    float* __restrict__ log_scores, float* __restrict__ entropy, int Hq, int Hkv, int CS,
    int CB, int r, int s_lo, int s_hi, int n_hc, int ldy, double probe_scale) {
  constexpr int R = 4 * HPW;
  constexpr int W = NT / kWave;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
  RowStats* stats = (RowStats*)smem_raw;                        // [R]
  double* hpart = (double*)(smem_raw + sizeof(RowStats) * R);   // [W]
  double* qs = hpart + W;                                       // [HPW][128][max, min]
  float* ys = (float*)(qs + HPW * 2 * kHeadDim);                // [R][ldy] offsets x - ref
  float* refs = ys + R * ldy;                                   // [R][ldy / 64] references
  const int nref = ldy >> 6;

  int64_t id = blockIdx.x;
  const int ns = s_hi - s_lo;
  const int s = s_hi - 1 - (int)(id % ns);   // heavier segments first
  id /= ns;
  const int hc = (int)(id % n_hc);
  id /= n_hc;
  const int g = (int)(id % Hkv);
  const int b = (int)(id / Hkv);
  const int G = Hq / Hkv;
  const int h0 = g * G + hc * HPW;
  const int nh = min(HPW, G - hc * HPW);
  const int nvis = min((s + 1) * r, CB);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & (kWave - 1);

  for (int t = threadIdx.x; t < HPW * 2 * kHeadDim; t += NT) {
    const int hh = t / (2 * kHeadDim), m = (t / kHeadDim) & 1, d = t % kHeadDim;
    const double* qv = qrep + ((size_t)(b * Hq + h0 + min(hh, nh - 1)) * CS + s) * 2 * kHeadDim;
    qs[(hh * kHeadDim + d) * 2 + m] = qv[m * kHeadDim + d];
  }
  __syncthreads();
  const float* kb = krep + (size_t)(b * Hkv + g) * padded_blocks(CB) * 2 * kHeadDim;

  // Phase 1: exact logits, one key block per lane.
  for (int j0 = wave * kWave; j0 < nvis; j0 += NT) {
    const int j = j0 + lane;
    const bool valid = j < nvis;
    const float* kr = kb + krep_offset(valid ? j : nvis - 1, 0, 0);
    double acc[HPW][4];
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh)
#pragma unroll
      for (int cc = 0; cc < 4; ++cc) acc[hh][cc] = 0.0;
#pragma unroll 2
    for (int d0 = 0; d0 < kHeadDim; d0 += 8) {
      double kx[8], kn[8];
      constexpr int kDq = 4 * kKTileBlocks;             // floats between dim quads
      constexpr int kMin = (kHeadDim / 4) * kDq;        // max part -> min part
      widen4(*(const float4*)(kr + (d0 / 4) * kDq), kx);
      widen4(*(const float4*)(kr + (d0 / 4 + 1) * kDq), kx + 4);
      widen4(*(const float4*)(kr + kMin + (d0 / 4) * kDq), kn);
      widen4(*(const float4*)(kr + kMin + (d0 / 4 + 1) * kDq), kn + 4);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
#pragma unroll
        for (int hh = 0; hh < HPW; ++hh) {
          const double2 qq = *(const double2*)(qs + (hh * kHeadDim + d0 + e) * 2);
          const double qa = qq.x, qb = qq.y;
          acc[hh][0] = fma(qa, kx[e], acc[hh][0]);   // S1: Q_max . K_max
          acc[hh][1] = fma(qa, kn[e], acc[hh][1]);   // S2: Q_max . K_min
          acc[hh][2] = fma(qb, kx[e], acc[hh][2]);   // S3: Q_min . K_max
          acc[hh][3] = fma(qb, kn[e], acc[hh][3]);   // S4: Q_min . K_min
        }
      }
    }
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) {
#pragma unroll
      for (int cc = 0; cc < 4; ++cc) {
        const int row = hh * 4 + cc;
        const double x = probe_scale * acc[hh][cc];
        const float ref = wave_max_f32_dpp(valid ? (float)x : -INFINITY);
        if (valid) ys[row * ldy + j] = (float)(x - (double)ref);
        if (lane == 0) refs[row * nref + (j0 >> 6)] = ref;
      }
    }
  }
  __syncthreads();

  // Phase 2a: statistics of every logit row, one wave per row.
  const int nch = (nvis + 63) >> 6;
  for (int row = wave; row < 4 * nh; row += W) {
    const float* yr = ys + row * ldy;
    const float* rr = refs + row * nref;
    float m = -INFINITY;
    for (int c = lane; c < nch; c += kWave) m = fmaxf(m, rr[c]);
    const float M = wave_max_f32(m);
    float best = -INFINITY;
    int bj = 0x7fffffff;
    for (int j = lane; j < nvis; j += kWave) {
      const float dv = yr[j] + (rr[j >> 6] - M);
      if (dv > best) { best = dv; bj = j; }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ob = __shfl_xor(best, o);
      const int oj = __shfl_xor(bj, o);
      if (ob > best || (ob == best && oj < bj)) { best = ob; bj = oj; }
    }
    double rest = 0.0;
    for (int j = lane; j < nvis; j += kWave) {
      const float dv = yr[j] + (rr[j >> 6] - M);
      if (j != bj) rest += (double)fast_exp(dv - best);
    }
    rest = wave_sum_f64(rest);
    if (lane == 0) stats[row] = RowStats{M, best, bj, (float)log1p(rest), rest / (1.0 + rest)};
  }
  __syncthreads();

  // Phase 2b: ln A and the entropy terms; each head's row is split over
  // W / HPW waves.
  constexpr int P = W / HPW;
  const int hh = wave % HPW, part = wave / HPW;
  double H = 0.0;
  if (hh < nh) {
    const int h = h0 + hh;
    RowStats st[4];
#pragma unroll
    for (int cc = 0; cc < 4; ++cc) st[cc] = stats[hh * 4 + cc];
    const float l12_top = (st[0].bj == st[1].bj) ? (float)log1p(-0.5 * (st[0].dfc + st[1].dfc)) : 0.f;
    const float l34_top = (st[2].bj == st[3].bj) ? (float)log1p(-0.5 * (st[2].dfc + st[3].dfc)) : 0.f;
    float* Lrow = log_scores + ((size_t)(b * Hq + h) * CS + s) * CB;
    for (int j = part * kWave + lane; j < nvis; j += P * kWave) {
      float ls[4];
#pragma unroll
      for (int cc = 0; cc < 4; ++cc) {
        const int row = hh * 4 + cc;
        const float dv = ys[row * ldy + j] + (refs[row * nref + (j >> 6)] - st[cc].M);
        ls[cc] = (j == st[cc].bj) ? -st[cc].lse : (dv - st[cc].best) - st[cc].lse;
      }
      const float l12 = (j == st[0].bj && j == st[1].bj) ? l12_top : log_pair_avg(ls[0], ls[1]);
      const float l34 = (j == st[2].bj && j == st[3].bj) ? l34_top : log_pair_avg(ls[2], ls[3]);
      const float L = fmaxf(l12, l34);
      Lrow[j] = L;
      H -= (double)(fast_exp(L) * L);
    }
    H = wave_sum_f64(H);
  }
  if (lane == 0) hpart[wave] = H;
  __syncthreads();
  if ((int)threadIdx.x < nh) {
    double Ht = 0.0;
    for (int p = 0; p < P; ++p) Ht += hpart[p * HPW + threadIdx.x];
    entropy[(size_t)(b * Hq + h0 + threadIdx.x) * CS + s] = (float)Ht;
  }
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
constexpr size_t kMaxLds = 160 * 1024;

size_t scores_lds_bytes(int hpw, int nt, int ldy) {
  const size_t R = 4 * (size_t)hpw;
  return sizeof(RowStats) * R + sizeof(double) * (size_t)(nt / kWave) +
         sizeof(double) * (size_t)hpw * 2 * kHeadDim + R * (size_t)ldy * 4 +
         R * (size_t)(ldy / 64) * 4;
}

// Threads per workgroup grow with the row length so that long rows keep
// several waves per SIMD in flight.
int pick_threads(int ldy) { return ldy <= 512 ? 256 : (ldy <= 1024 ? 512 : 1024); }

// Heads per workgroup: up to 4 query heads of one KV group share each K
// representation load; fewer when the LDS tile for this row length would
// not fit.  0 if even one head does not fit.
int pick_hpw(int G, int ldy, size_t max_lds) {
  int hpw = G >= 4 ? 4 : (G >= 2 ? 2 : 1);
  while (hpw >= 1 && scores_lds_bytes(hpw, pick_threads(ldy), ldy) > max_lds) hpw /= 2;
  return hpw;
}

size_t device_max_lds() {
  int dev = 0, v = 0;
  if (hipGetDevice(&dev) != hipSuccess) return kMaxLds;
  if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess ||
      v <= 0)
    return kMaxLds;
  return (size_t)v < kMaxLds ? (size_t)v : kMaxLds;
}

template <int HPW, int NT>
hipError_t launch_scores_t(const double* qrep, const float* krep, float* log_scores,
                           float* entropy, const ProbeShape& s, int s_lo, int s_hi, int ldy,
                           double probe_scale, hipStream_t stream) {
  const int G = s.Hq / s.Hkv;
  const int n_hc = (G + HPW - 1) / HPW;
  const int64_t grid = (int64_t)s.B * s.Hkv * n_hc * (s_hi - s_lo);
  const size_t lds = scores_lds_bytes(HPW, NT, ldy);
  hipLaunchKernelGGL((scores_kernel<HPW, NT>), dim3((unsigned)grid), dim3(NT), lds, stream,
                     qrep, krep, log_scores, entropy, s.Hq, s.Hkv, s.CS, s.CB, s.r, s_lo, s_hi,
                     n_hc, ldy, probe_scale);
  return hipGetLastError();
}

template <int HPW>
hipError_t launch_scores_h(const double* qrep, const float* krep, float* log_scores,
                           float* entropy, const ProbeShape& s, int s_lo, int s_hi, int ldy,
                           double probe_scale, hipStream_t stream) {
  switch (pick_threads(ldy)) {
    case 256:
      return launch_scores_t<HPW, 256>(qrep, krep, log_scores, entropy, s, s_lo, s_hi, ldy,
                                       probe_scale, stream);
    case 512:
      return launch_scores_t<HPW, 512>(qrep, krep, log_scores, entropy, s, s_lo, s_hi, ldy,
                                       probe_scale, stream);
    default:
      return launch_scores_t<HPW, 1024>(qrep, krep, log_scores, entropy, s, s_lo, s_hi, ldy,
                                        probe_scale, stream);
  }
}

}  // namespace

size_t probe_qrep_bytes(const ProbeShape& s) {
  return align_up((size_t)s.B * s.Hq * s.CS * 2 * kHeadDim * sizeof(double));
}
size_t probe_krep_bytes(const ProbeShape& s) {
  return align_up((size_t)s.B * s.Hkv * padded_blocks(s.CB) * 2 * kHeadDim * sizeof(float));
}

bool probe_supported(const ProbeShape& s) {
  const int ldy = (s.CB + 63) / 64 * 64;
  return pick_hpw(s.Hq / s.Hkv, ldy, kMaxLds) > 0;
}

hipError_t launch_probe(const uint16_t* q, const uint16_t* k, const ProbeShape& s,
                        double probe_scale, float* log_scores, float* entropy, void* workspace,
                        hipStream_t stream) {
  double* qrep = (double*)workspace;
  float* krep = (float*)((char*)workspace + probe_qrep_bytes(s));
  {
    const int64_t items = (int64_t)s.B * s.Hq * s.CS + (int64_t)s.B * s.Hkv * s.CB;
    const int64_t grid = (items + kWavesPerBlock - 1) / kWavesPerBlock;
    hipLaunchKernelGGL(pool_kernel, dim3((unsigned)grid), dim3(kThreads), 0, stream, q, k, s.B,
                       s.Hq, s.Hkv, s.N, s.Ls, s.Lb, s.CS, s.CB, qrep, krep);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  // Segments are split into launches by visible-row length so that short
  // rows do not reserve LDS for the longest one.
  const int G = s.Hq / s.Hkv;
  const size_t max_lds = device_max_lds();
  int s_lo = 0;
  while (s_lo < s.CS) {
    const int nvis_lo = min((s_lo + 1) * s.r, s.CB);
    int cap = 512;
    while (cap < nvis_lo) cap *= 2;
    // last segment whose row fits in `cap`
    int s_hi = min(s.CS, cap / s.r);
    if (s_hi <= s_lo) s_hi = s_lo + 1;
    const int nvis_hi = min(s_hi * s.r, s.CB);
    const int ldy = (nvis_hi + 63) / 64 * 64;
    const int hpw = pick_hpw(G, ldy, max_lds);
    hipError_t e = hipErrorInvalidValue;
    if (hpw == 4)
      e = launch_scores_h<4>(qrep, krep, log_scores, entropy, s, s_lo, s_hi, ldy, probe_scale,
                             stream);
    else if (hpw == 2)
      e = launch_scores_h<2>(qrep, krep, log_scores, entropy, s, s_lo, s_hi, ldy, probe_scale,
                             stream);
    else if (hpw == 1)
      e = launch_scores_h<1>(qrep, krep, log_scores, entropy, s, s_lo, s_hi, ldy, probe_scale,
                             stream);
    if (e != hipSuccess) return e;
    s_lo = s_hi;
  }
  return hipSuccess;
}

}  // namespace ei
