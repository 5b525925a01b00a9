/* Drives every entry point of the CPU oracle once on a small ragged problem,
 * for a build with AddressSanitizer and UndefinedBehaviorSanitizer: any
 * out-of-bounds access, leak or undefined operation aborts the run.
 * The oracle source is compiled into this program directly. */
#include "../../oracle/oracle.c"

#include <stdio.h>

static uint32_t lcg_state = 12345u;
static float uniform(void) {   /* [-1, 1) */
  lcg_state = lcg_state * 1664525u + 1013904223u;
  return (float)((lcg_state >> 8) & 0xffffff) / 8388608.0f - 1.0f;
}
static uint16_t bf16_bits(float x) {   /* round to nearest even */
  uint32_t u;
  memcpy(&u, &x, 4);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

int main(void) {
  enum { B = 1, Hq = 4, Hkv = 2, N = 300, D = 128, Ls = 128, Lb = 64 };
  const int64_t CS = (N + Ls - 1) / Ls, CB = (N + Lb - 1) / Lb;
  const int32_t kmax = 3 * 64 / Lb + Ls / Lb;   /* B_h = 64 tokens, cap 3 */
  uint16_t *q = malloc(sizeof(uint16_t) * B * Hq * N * D);
  uint16_t *k = malloc(sizeof(uint16_t) * B * Hkv * N * D);
  uint16_t *v = malloc(sizeof(uint16_t) * B * Hkv * N * D);
  for (int64_t i = 0; i < (int64_t)B * Hq * N * D; ++i) q[i] = bf16_bits(uniform());
  for (int64_t i = 0; i < (int64_t)B * Hkv * N * D; ++i) {
    k[i] = bf16_bits(uniform());
    v[i] = bf16_bits(uniform());
  }
  double *ls = malloc(sizeof(double) * B * Hq * CS * CB);
  double *en = malloc(sizeof(double) * B * Hq * CS);
  for (int64_t i = 0; i < (int64_t)B * Hq * CS * CB; ++i) ls[i] = 0.0;
  int rc = orc_probe(q, k, B, Hq, Hkv, N, D, Ls, Lb, 1.0, NULL, 0, ls, en);
  float *lsf = malloc(sizeof(float) * B * Hq * CS * CB);
  float *enf = malloc(sizeof(float) * B * Hq * CS);
  for (int64_t i = 0; i < (int64_t)B * Hq * CS * CB; ++i) lsf[i] = (float)ls[i];
  for (int64_t i = 0; i < (int64_t)B * Hq * CS; ++i) enf[i] = (float)en[i];
  uint8_t *rigid = malloc(B * Hq);
  int32_t *bud = malloc(sizeof(int32_t) * B * Hq * CS);
  int32_t *idx = malloc(sizeof(int32_t) * B * Hq * CS * kmax);
  int32_t *cnt = malloc(sizeof(int32_t) * B * Hq * CS);
  for (int mode = ORC_CLASSIFY_HEAD; mode <= ORC_CLASSIFY_SEGMENT && rc == ORC_OK; ++mode)
    rc = orc_select_mode(lsf, enf, B, Hq, Hkv, mode, N, Ls, Lb, 1e-5f, 0.5, 0.4, 64, 3, kmax,
                         rigid, bud, idx, cnt);
  double Bout[8];
  if (rc == ORC_OK) rc = orc_budget(enf, CS, 1e-5f, 0.5, 0.4, 64, 3, Bout) < 0 ? -1 : ORC_OK;
  if (rc == ORC_OK)
    rc = orc_budget_segment(enf, CS, 1e-5f, 0.5, 0.4, 64, 3, Bout) < 0 ? -1 : ORC_OK;
  int32_t rows[4 * 3] = {0, 0, 0, 0, 1, 127, 0, 2, 128, 0, 3, N - 1};
  double *out = malloc(sizeof(double) * 4 * D);
  if (rc == ORC_OK)   /* sparse, on the selection just made */
    rc = orc_attention(q, k, v, B, Hq, Hkv, N, D, Ls, Lb, 0.088, 1, idx, cnt, kmax, rows, 4,
                       out);
  if (rc == ORC_OK)   /* dense causal */
    rc = orc_attention(q, k, v, B, Hq, Hkv, N, D, Ls, Lb, 0.088, 1, NULL, NULL, 0, rows, 4,
                       out);
  free(q); free(k); free(v); free(ls); free(en); free(lsf); free(enf);
  free(rigid); free(bud); free(idx); free(cnt); free(out);
  printf("oracle sanitized run: %s\n", rc == ORC_OK ? "ok" : "error");
  return rc == ORC_OK ? 0 : 1;
}
