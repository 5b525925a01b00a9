/*
 * oracle.c -- plain, slow, fp64 CPU reference for the entropy-guided sparse
 * prefill path of EntropyInfer ("From Rigid to Dynamic: Entropy-Guided
 * Adaptive Inference for Long-Context LLMs", Section 4.2, Algorithms 1-3,
 * Appendix A).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load this library.  It shares no code,
 * header, table or helper with the HIP library; neither side includes or links
 * the other.  Every computation is done in IEEE double precision with no FMA
 * contraction (built with -ffp-contract=off) and no fast-math.
 *
 * Notation (Section 4.1): N context length, L_S segment size, L_B block size,
 * C_S = ceil(N / L_S) segments, C_B = ceil(N / L_B) key blocks,
 * r = L_S / L_B blocks per segment, B_h base budget (tokens).
 *
 * Readings of the paper taken here (the paper is silent or garbled on them):
 *  - K_Rep is pooled over L_B-token key blocks (Algorithm 1 says K_Rep
 *    "follows a similar process"; Eq. t_obs sizes the matrix C_S x C_B).
 *  - Segment s sees the key blocks j < (s+1) r (block-causal, including its
 *    own blocks); the observation matrix is not defined elsewhere.
 *  - Algorithm 2 applies no 1/sqrt(d); a multiplicative probe_scale is
 *    exposed and 1.0 is the literal reading.
 *  - A_obs is used as it is (rows sum to between 1 and 2); the entropy is
 *    -sum a ln a with natural log and 0 ln 0 = 0 (Section 3).
 *  - A ragged tail (N not a multiple of L_S or L_B) pools the rows that
 *    exist; a segment / block never reaches past N.
 *
 * Stable evaluation.  The definitions are evaluated in log space so that
 * nothing underflows: ln S_c[j] = (x_c[j] - m_c) - log1p(rest_c) with
 * m_c = max_j x_c[j], rest_c = sum over j != argmax of exp(x_c[j] - m_c).
 * For the pair average P = (S_a + S_b) / 2, ln P[j] = logaddexp(ln S_a[j],
 * ln S_b[j]) - ln 2, except at the index that is the argmax of both softmaxes
 * where the identity 1 - S_c[argmax] = rest_c / (1 + rest_c) gives
 * ln P = log1p(-(d_a + d_b) / 2) without cancellation.  These are algebraic
 * identities of the definition, not approximations.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_OK 0
#define ORC_ERR_ARG (-1)
#define ORC_ERR_MEM (-2)

/* Classification modes of the selection (the method and two variants). */
#define ORC_CLASSIFY_HEAD 0       /* Algorithm 3 per query head */
#define ORC_CLASSIFY_GQA_GROUP 1  /* Algorithm 3 on the GQA-group mean entropy */
#define ORC_CLASSIFY_SEGMENT 2    /* rigid rule applied per segment */

static const double ORC_LN2 = 0.69314718055994530942;

/* bf16 (the upper 16 bits of an IEEE binary32) to double; exact. */
static double bf16_to_f64(uint16_t h) {
  uint32_t u = ((uint32_t)h) << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

int orc_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

void orc_set_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* ---------------------------------------------------------------------------
 * Algorithm 1: representation vectors.  Rows of one head, x[rows][D] bf16,
 * grouped into groups of L consecutive rows (the last group may be short).
 * out_max / out_min: [n_groups][D] doubles (exact copies of input values).
 * ------------------------------------------------------------------------- */
int orc_pool(const uint16_t *x, int64_t rows, int D, int L, double *out_max,
             double *out_min) {
  if (!x || !out_max || !out_min || rows < 0 || D <= 0 || L <= 0) return ORC_ERR_ARG;
  int64_t groups = ceil_div(rows, L);
  for (int64_t g = 0; g < groups; ++g) {
    int64_t r0 = g * L, r1 = r0 + L < rows ? r0 + L : rows;
    for (int d = 0; d < D; ++d) {
      double mx = -INFINITY, mn = INFINITY;
      for (int64_t r = r0; r < r1; ++r) {
        double v = bf16_to_f64(x[r * D + d]);
        if (v > mx) mx = v;
        if (v < mn) mn = v;
      }
      out_max[g * D + d] = mx;
      out_min[g * D + d] = mn;
    }
  }
  return ORC_OK;
}

/* Stable log-softmax of one row x[0..n) (n >= 1): writes ln S into lns and
 * returns argmax (lowest index among equal maxima) and the deficit
 * 1 - S[argmax] = rest / (1 + rest). */
static void log_softmax_row(const double *x, int64_t n, double *lns,
                            int64_t *argmax, double *deficit) {
  int64_t am = 0;
  double m = x[0];
  for (int64_t j = 1; j < n; ++j)
    if (x[j] > m) { m = x[j]; am = j; }
  double rest = 0.0;
  for (int64_t j = 0; j < n; ++j)
    if (j != am) rest += exp(x[j] - m);
  double off = log1p(rest);
  for (int64_t j = 0; j < n; ++j) lns[j] = (x[j] - m) - off;
  lns[am] = -off;
  *argmax = am;
  *deficit = rest / (1.0 + rest);
}

/* ln((S_a[j] + S_b[j]) / 2) for one index. */
static double log_pair_avg(double la, double lb, int both_argmax, double da,
                           double db) {
  if (both_argmax) return log1p(-0.5 * (da + db));
  double hi = la > lb ? la : lb, lo = la > lb ? lb : la;
  return hi + log1p(exp(lo - hi)) - ORC_LN2;
}

/* ---------------------------------------------------------------------------
 * Algorithm 2 + row entropy (Section 4.2): the observation matrix in log form
 * and its row entropies.
 *
 * q: [B][Hq][N][D] bf16, k: [B][Hkv][N][D] bf16.  Query head h reads key head
 * h / (Hq / Hkv).  sel: n_sel (b, h, s) triples to evaluate, or NULL for all.
 * Evaluated row t (t-th triple of sel, or t = (b Hq + h) C_S + s when sel is
 * NULL) writes log_scores[t][0 .. n_vis(s)) with L[j] = ln A_obs[s][j]
 * (log_scores has C_B doubles per row; the rest is untouched) and
 * entropy[t]; n_vis(s) = min((s+1) r, C_B).
 * ------------------------------------------------------------------------- */
int orc_probe(const uint16_t *q, const uint16_t *k, int B, int Hq, int Hkv,
              int N, int D, int Ls, int Lb, double probe_scale,
              const int32_t *sel, int64_t n_sel, double *log_scores,
              double *entropy) {
  if (!q || !k || !log_scores || !entropy) return ORC_ERR_ARG;
  if (B < 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv || N < 0 || D <= 0 || Ls <= 0 ||
      Lb <= 0 || Ls % Lb)
    return ORC_ERR_ARG;
  const int64_t CS = ceil_div(N, Ls), CB = ceil_div(N, Lb), r = Ls / Lb;
  const int G = Hq / Hkv;
  if (sel == NULL) n_sel = (int64_t)B * Hq * CS;
  if (n_sel == 0 || N == 0) return ORC_OK;

  /* K representation for every (b, g, block): [B][Hkv][C_B][D] max and min. */
  double *kmax = (double *)malloc(sizeof(double) * (size_t)B * Hkv * CB * D);
  double *kmin = (double *)malloc(sizeof(double) * (size_t)B * Hkv * CB * D);
  if (!kmax || !kmin) { free(kmax); free(kmin); return ORC_ERR_MEM; }
#pragma omp parallel for schedule(static)
  for (int64_t bg = 0; bg < (int64_t)B * Hkv; ++bg)
    orc_pool(k + bg * (int64_t)N * D, N, D, Lb, kmax + bg * CB * D, kmin + bg * CB * D);

  int err = ORC_OK;
#pragma omp parallel
  {
    double *x = (double *)malloc(sizeof(double) * (size_t)CB * 4);
    double *lns = (double *)malloc(sizeof(double) * (size_t)CB * 4);
    double *qrep = (double *)malloc(sizeof(double) * (size_t)D * 2);
    if (!x || !lns || !qrep) {
#pragma omp atomic write
      err = ORC_ERR_MEM;
    }
#pragma omp for schedule(dynamic, 4)
    for (int64_t t = 0; t < n_sel; ++t) {
      if (!x || !lns || !qrep) continue;
      int64_t b, h, s;
      if (sel) { b = sel[3 * t]; h = sel[3 * t + 1]; s = sel[3 * t + 2]; }
      else { b = t / ((int64_t)Hq * CS); h = (t / CS) % Hq; s = t % CS; }
      if (b < 0 || b >= B || h < 0 || h >= Hq || s < 0 || s >= CS) {
#pragma omp atomic write
        err = ORC_ERR_ARG;
        continue;
      }
      const int64_t g = h / G;
      const int64_t rows = (s + 1) * Ls <= N ? Ls : N - s * Ls;
      /* Algorithm 1 on this segment of query head h. */
      orc_pool(q + ((b * Hq + h) * (int64_t)N + s * Ls) * D, rows, D, (int)rows,
               qrep, qrep + D);
      const double *qa[2] = {qrep, qrep + D};
      const int64_t nvis = (s + 1) * r < CB ? (s + 1) * r : CB;
      const double *kmx = kmax + (b * Hkv + g) * CB * D;
      const double *kmn = kmin + (b * Hkv + g) * CB * D;
      /* The four products of Algorithm 2: (max,max), (max,min), (min,max),
       * (min,min); c = 0..3 stands for S1..S4. */
      for (int c = 0; c < 4; ++c) {
        const double *qv = qa[c >> 1];
        const double *kb = (c & 1) ? kmn : kmx;
        for (int64_t j = 0; j < nvis; ++j) {
          double acc = 0.0;
          for (int d = 0; d < D; ++d) acc += qv[d] * kb[j * D + d];
          x[c * CB + j] = probe_scale * acc;
        }
      }
      int64_t am[4];
      double dfc[4];
      for (int c = 0; c < 4; ++c)
        log_softmax_row(x + c * CB, nvis, lns + c * CB, &am[c], &dfc[c]);
      double H = 0.0;
      double *Lrow = log_scores + t * CB;
      for (int64_t j = 0; j < nvis; ++j) {
        /* A_obs = max((S1 + S2) / 2, (S3 + S4) / 2), in log form. */
        double l12 = log_pair_avg(lns[0 * CB + j], lns[1 * CB + j],
                                  j == am[0] && j == am[1], dfc[0], dfc[1]);
        double l34 = log_pair_avg(lns[2 * CB + j], lns[3 * CB + j],
                                  j == am[2] && j == am[3], dfc[2], dfc[3]);
        double L = l12 > l34 ? l12 : l34;
        Lrow[j] = L;
        H -= exp(L) * L;
      }
      entropy[t] = H;
    }
    free(x);
    free(lns);
    free(qrep);
  }
  free(kmax);
  free(kmin);
  return err;
}

/* ---------------------------------------------------------------------------
 * Algorithm 3 for one head: given the segment entropies e[0..cs) (binary32),
 * decide rigid / dynamic and write the budgets B[0..cs) in tokens.
 * Returns 1 for a rigid head, 0 for a dynamic one.
 *
 * Rigid iff every e_i < e_t (so max e_i < e_t; a NaN entropy makes the head
 * dynamic).  Dynamic: B_0 = B_h and for i >= 1
 *   ratio   = |e_i - e_{i-1}| / e_{i-1}       (0/0 -> 0, x/0 -> +inf)
 *   delta   = (alpha * B_h) * (ratio - Delta_t)
 *   B_i     = B_{i-1} + delta, then clamped to [B_h, mult * B_h]
 * (the printed clamp max(min(B_i, B_0), 3 B_0) always yields 3 B_0; the
 * bound B_i <= 3 B_h used in Appendix A fixes the intended clamp).  A NaN
 * budget clamps to B_h.  Evaluated in binary64 in exactly this order.
 * ------------------------------------------------------------------------- */
int orc_budget(const float *e, int64_t cs, float e_t, double alpha,
               double delta_t, int32_t base_budget, int32_t mult, double *Bout) {
  int rigid = 1;
  for (int64_t i = 0; i < cs; ++i)
    if (!(e[i] < e_t)) rigid = 0;
  const double B0 = (double)base_budget;
  const double cap = (double)mult * B0;
  if (cs <= 0) return rigid;
  Bout[0] = B0;
  if (rigid) {
    for (int64_t i = 1; i < cs; ++i) Bout[i] = B0;
    return 1;
  }
  const double a = alpha * B0;
  for (int64_t i = 1; i < cs; ++i) {
    const double ep = (double)e[i - 1], ec = (double)e[i];
    const double num = fabs(ec - ep);
    const double ratio = (num == 0.0 && ep == 0.0) ? 0.0 : num / ep;
    const double t = ratio - delta_t;
    const double delta = a * t;
    double Bn = Bout[i - 1] + delta;
    if (!(Bn >= B0)) Bn = B0;
    if (Bn > cap) Bn = cap;
    Bout[i] = Bn;
  }
  return 0;
}

/* Per-segment variant of the rigid rule (a reading of Algorithm 3 with the
 * classification moved from the head to the segment): segment i with
 * e_i < e_t takes the base budget B_0; every other segment i >= 1 follows
 * Algorithm 3's update from the previous segment's budget.  Returns 1 iff
 * every segment is rigid, in which case the result equals orc_budget's. */
int orc_budget_segment(const float *e, int64_t cs, float e_t, double alpha,
                       double delta_t, int32_t base_budget, int32_t mult,
                       double *Bout) {
  int rigid = 1;
  for (int64_t i = 0; i < cs; ++i)
    if (!(e[i] < e_t)) rigid = 0;
  const double B0 = (double)base_budget;
  const double cap = (double)mult * B0;
  if (cs <= 0) return rigid;
  Bout[0] = B0;
  const double a = alpha * B0;
  for (int64_t i = 1; i < cs; ++i) {
    if (e[i] < e_t) {
      Bout[i] = B0;
      continue;
    }
    const double ep = (double)e[i - 1], ec = (double)e[i];
    const double num = fabs(ec - ep);
    const double ratio = (num == 0.0 && ep == 0.0) ? 0.0 : num / ep;
    const double t = ratio - delta_t;
    const double delta = a * t;
    double Bn = Bout[i - 1] + delta;
    if (!(Bn >= B0)) Bn = B0;
    if (Bn > cap) Bn = cap;
    Bout[i] = Bn;
  }
  return rigid;
}

/* GQA-group entropy (the per-group aggregation the paper plots as
 * "Averaged"): the mean of the group's G query heads' entropies for each
 * segment, summed in binary64 in head order, divided by G and rounded to
 * binary32.  eg: [C_S] out; e_group: the group's first head's row of a
 * [Hq][C_S] block. */
void orc_group_entropy(const float *e_group, int64_t cs, int G, float *eg) {
  for (int64_t i = 0; i < cs; ++i) {
    double sum = 0.0;
    for (int h = 0; h < G; ++h) sum += (double)e_group[(int64_t)h * cs + i];
    eg[i] = (float)(sum / (double)G);
  }
}

/* Orderable key of a binary32 ranking score: larger float -> larger key;
 * -0 == +0; NaN below -inf. */
static uint32_t score_key(float v) {
  if (v != v) return 0u;
  if (v == 0.0f) v = 0.0f;
  uint32_t u;
  memcpy(&u, &v, sizeof u);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

typedef struct { uint32_t key; int32_t j; } orc_cand;

/* descending by score, equal scores -> higher block index first */
static int cand_cmp(const void *pa, const void *pb) {
  const orc_cand *a = (const orc_cand *)pa, *b = (const orc_cand *)pb;
  if (a->key != b->key) return a->key > b->key ? -1 : 1;
  return a->j > b->j ? -1 : (a->j < b->j ? 1 : 0);
}

/* ---------------------------------------------------------------------------
 * Head classification, budgets (Algorithm 3) and top-k block selection
 * (Section 4.2, Eq. t_topk) from binary32 log scores and entropies.
 *
 * log_scores: [B][Hq][C_S][C_B] (only j < n_past(s) = s r is read),
 * entropy: [B][Hq][C_S].  Outputs: head_is_rigid [B][Hq] (u8),
 * budget_blocks [B][Hq][C_S] = k_s = min(floor(B_s / L_B), n_past(s)),
 * block_idx [B][Hq][C_S][kmax] ascending and -1 padded: the k_s past blocks of
 * largest score plus the segment's own blocks s r .. min((s+1) r, C_B) - 1,
 * block_cnt [B][Hq][C_S] = number of valid entries.
 *
 * mode: ORC_CLASSIFY_HEAD (the method), ORC_CLASSIFY_GQA_GROUP (every head of
 * a KV group takes the budgets that Algorithm 3 gives the group's mean
 * entropy) or ORC_CLASSIFY_SEGMENT (orc_budget_segment per head).  The block
 * ranking is per query head in every mode.  A uniform budget for every head
 * (the fixed-k scheme of CritiPrefill) is ORC_CLASSIFY_HEAD with e_t = +inf.
 * ------------------------------------------------------------------------- */
int orc_select_mode(const float *log_scores, const float *entropy, int B, int Hq,
                    int Hkv, int mode, int N, int Ls, int Lb, float e_t, double alpha,
                    double delta_t, int32_t base_budget, int32_t mult, int32_t kmax,
                    uint8_t *head_is_rigid, int32_t *budget_blocks,
                    int32_t *block_idx, int32_t *block_cnt) {
  if (!log_scores || !entropy || !head_is_rigid || !budget_blocks || !block_idx ||
      !block_cnt)
    return ORC_ERR_ARG;
  if (B < 0 || Hq <= 0 || N < 0 || Ls <= 0 || Lb <= 0 || Ls % Lb || base_budget < 0 ||
      mult < 1 || Hkv <= 0 || Hq % Hkv || mode < ORC_CLASSIFY_HEAD ||
      mode > ORC_CLASSIFY_SEGMENT)
    return ORC_ERR_ARG;
  const int G = Hq / Hkv;
  const int64_t CS = ceil_div(N, Ls), CB = ceil_div(N, Lb), r = Ls / Lb;
  if ((int64_t)kmax < (int64_t)mult * base_budget / Lb + r) return ORC_ERR_ARG;
  int err = ORC_OK;
#pragma omp parallel
  {
    double *Bv = (double *)malloc(sizeof(double) * (size_t)(CS > 0 ? CS : 1));
    float *eg = (float *)malloc(sizeof(float) * (size_t)(CS > 0 ? CS : 1));
    orc_cand *cand = (orc_cand *)malloc(sizeof(orc_cand) * (size_t)(CB > 0 ? CB : 1));
    uint8_t *chosen = (uint8_t *)malloc((size_t)(CB > 0 ? CB : 1));
    if (!Bv || !eg || !cand || !chosen) {
#pragma omp atomic write
      err = ORC_ERR_MEM;
    }
#pragma omp for schedule(dynamic, 1)
    for (int64_t bh = 0; bh < (int64_t)B * Hq; ++bh) {
      if (!Bv || !eg || !cand || !chosen) continue;
      const float *e = entropy + bh * CS;
      int rigid;
      if (mode == ORC_CLASSIFY_GQA_GROUP) {
        const int64_t first = bh - (bh % Hq) % G;   /* the group's first head */
        orc_group_entropy(entropy + first * CS, CS, G, eg);
        rigid = orc_budget(eg, CS, e_t, alpha, delta_t, base_budget, mult, Bv);
      } else if (mode == ORC_CLASSIFY_SEGMENT) {
        rigid = orc_budget_segment(e, CS, e_t, alpha, delta_t, base_budget, mult, Bv);
      } else {
        rigid = orc_budget(e, CS, e_t, alpha, delta_t, base_budget, mult, Bv);
      }
      head_is_rigid[bh] = (uint8_t)rigid;
      for (int64_t s = 0; s < CS; ++s) {
        const int64_t npast = s * r;
        int64_t kb = (int64_t)floor(Bv[s] / (double)Lb);
        if (kb > npast) kb = npast;
        budget_blocks[bh * CS + s] = (int32_t)kb;
        const float *Lrow = log_scores + (bh * CS + s) * CB;
        memset(chosen, 0, (size_t)npast);
        if (kb < npast) {
          for (int64_t j = 0; j < npast; ++j) {
            cand[j].key = score_key(Lrow[j]);
            cand[j].j = (int32_t)j;
          }
          qsort(cand, (size_t)npast, sizeof(orc_cand), cand_cmp);
          for (int64_t t = 0; t < kb; ++t) chosen[cand[t].j] = 1;
        } else {
          memset(chosen, 1, (size_t)npast);
        }
        int32_t *out = block_idx + (bh * CS + s) * kmax;
        int64_t c = 0;
        for (int64_t j = 0; j < npast; ++j)
          if (chosen[j]) out[c++] = (int32_t)j;
        const int64_t dend = (s + 1) * r < CB ? (s + 1) * r : CB;
        for (int64_t j = npast; j < dend; ++j) out[c++] = (int32_t)j;
        block_cnt[bh * CS + s] = (int32_t)c;
        for (int64_t t = c; t < kmax; ++t) out[t] = -1;
      }
    }
    free(Bv);
    free(eg);
    free(cand);
    free(chosen);
  }
  return err;
}

/* The method's selection: classification per query head (Algorithm 3). */
int orc_select(const float *log_scores, const float *entropy, int B, int Hq,
               int N, int Ls, int Lb, float e_t, double alpha, double delta_t,
               int32_t base_budget, int32_t mult, int32_t kmax,
               uint8_t *head_is_rigid, int32_t *budget_blocks,
               int32_t *block_idx, int32_t *block_cnt) {
  return orc_select_mode(log_scores, entropy, B, Hq, Hq, ORC_CLASSIFY_HEAD, N, Ls, Lb,
                         e_t, alpha, delta_t, base_budget, mult, kmax, head_is_rigid,
                         budget_blocks, block_idx, block_cnt);
}

/* ---------------------------------------------------------------------------
 * Causal GQA attention (Section 2 definition of A_h, with the sparse key set
 * of Section 4.2) for selected query rows, in fp64.
 *
 * q: [B][Hq][N][D], k, v: [B][Hkv][N][D] bf16.  rows: n_rows (b, h, i)
 * triples.  If block_idx is NULL the key set of query i is {0..i} when causal
 * and {0..N-1} otherwise (dense); else it is the keys of the blocks listed in
 * block_idx[b][h][i / L_S][0 .. block_cnt) restricted to keys <= i.
 * out: [n_rows][D].
 * ------------------------------------------------------------------------- */
int orc_attention(const uint16_t *q, const uint16_t *k, const uint16_t *v, int B,
                  int Hq, int Hkv, int N, int D, int Ls, int Lb, double scale,
                  int causal, const int32_t *block_idx, const int32_t *block_cnt,
                  int32_t kmax, const int32_t *rows, int64_t n_rows, double *out) {
  if (!q || !k || !v || !rows || !out) return ORC_ERR_ARG;
  if (B < 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv || N < 0 || D <= 0) return ORC_ERR_ARG;
  if (block_idx && (!block_cnt || Ls <= 0 || Lb <= 0 || Ls % Lb)) return ORC_ERR_ARG;
  const int G = Hq / Hkv;
  const int64_t CS = block_idx ? ceil_div(N, Ls) : 0;
  int err = ORC_OK;
#pragma omp parallel
  {
    double *p = (double *)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
    uint8_t *on = (uint8_t *)malloc((size_t)(N > 0 ? N : 1));
    double *qi = (double *)malloc(sizeof(double) * (size_t)D);
    if (!p || !on || !qi) {
#pragma omp atomic write
      err = ORC_ERR_MEM;
    }
#pragma omp for schedule(dynamic, 1)
    for (int64_t t = 0; t < n_rows; ++t) {
      if (!p || !on || !qi) continue;
      const int64_t b = rows[3 * t], h = rows[3 * t + 1], i = rows[3 * t + 2];
      if (b < 0 || b >= B || h < 0 || h >= Hq || i < 0 || i >= N) {
#pragma omp atomic write
        err = ORC_ERR_ARG;
        continue;
      }
      const int64_t g = h / G;
      const uint16_t *qrow = q + ((b * Hq + h) * (int64_t)N + i) * D;
      const uint16_t *kh = k + (b * Hkv + g) * (int64_t)N * D;
      const uint16_t *vh = v + (b * Hkv + g) * (int64_t)N * D;
      for (int d = 0; d < D; ++d) qi[d] = bf16_to_f64(qrow[d]);
      const int64_t jmax = (causal || block_idx) ? i : N - 1;
      memset(on, 0, (size_t)(jmax + 1));
      if (block_idx) {
        const int64_t s = i / Ls;
        const int32_t *lst = block_idx + ((b * Hq + h) * CS + s) * kmax;
        const int32_t cnt = block_cnt[(b * Hq + h) * CS + s];
        for (int32_t c = 0; c < cnt; ++c) {
          const int64_t blk = lst[c];
          if (blk < 0) continue;
          for (int64_t j = blk * Lb; j < (blk + 1) * Lb && j <= jmax; ++j) on[j] = 1;
        }
      } else {
        memset(on, 1, (size_t)(jmax + 1));
      }
      double m = -INFINITY;
      for (int64_t j = 0; j <= jmax; ++j) {
        if (!on[j]) continue;
        double acc = 0.0;
        for (int d = 0; d < D; ++d) acc += qi[d] * bf16_to_f64(kh[j * D + d]);
        p[j] = scale * acc;
        if (p[j] > m) m = p[j];
      }
      double l = 0.0;
      for (int64_t j = 0; j <= jmax; ++j)
        if (on[j]) { p[j] = exp(p[j] - m); l += p[j]; }
      double *o = out + t * D;
      for (int d = 0; d < D; ++d) o[d] = 0.0;
      for (int64_t j = 0; j <= jmax; ++j) {
        if (!on[j]) continue;
        const double w = p[j] / l;
        for (int d = 0; d < D; ++d) o[d] += w * bf16_to_f64(vh[j * D + d]);
      }
      if (l == 0.0)
        for (int d = 0; d < D; ++d) o[d] = NAN;
    }
    free(p);
    free(on);
    free(qi);
  }
  return err;
}
