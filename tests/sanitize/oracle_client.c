/*
 * Runs every function of the fp64 oracle (oracle/speechkv_oracle.c, compiled
 * into this program) under AddressSanitizer and UndefinedBehaviorSanitizer
 * on small shapes that reach its edge cases: no text prefix, no speech, no
 * suffix, a window longer than the speech, a short last window, a layer below
 * l0, both mask modes, grouped heads, the zero gate, and a cache capacity
 * above every compressed length.  Checks that every output is finite (NaN
 * only where the oracle documents it: LSE of rows past a sequence) and prints
 * "ok <cases>".
 */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>

void speechkv_oracle_pool(const double*, const double*, int, int, int, int, const int*, const int*,
                          const int*, int, int, int, const double*, double*, double*, int, int*);
void speechkv_oracle_attention(const double*, const double*, const double*, int, int, int, int, int,
                               int, const int*, const int*, const int*, int, int, int, int, double,
                               double*, double*);
void speechkv_oracle_decode(const double*, const double*, const double*, const int*, int, int, int,
                            int, int, double, double*, double*);
void speechkv_oracle_attention_bwd(const double*, const double*, const double*, int, int, int, int,
                                   int, int, const int*, const int*, const int*, int, int, int, int,
                                   double, const double*, double*, double*, double*);
void speechkv_oracle_pool_bwd(const double*, const double*, int, int, int, int, const int*,
                              const int*, const int*, int, int, int, const double*, const double*,
                              const double*, int, double*, double*, double*);
int speechkv_oracle_compressed_len(int, int, int, int, int, int);

static unsigned long long rng = 88172645463325252ull;
static double draw(void) {
  rng ^= rng << 13;
  rng ^= rng >> 7;
  rng ^= rng << 17;
  return (double)(rng >> 11) / 9007199254740992.0 * 2.0 - 1.0;
}
static double* vec(size_t n) {
  double* x = malloc(sizeof(double) * (n ? n : 1));
  for (size_t i = 0; i < n; ++i) x[i] = draw();
  return x;
}
static int finite(const double* x, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (!isfinite(x[i])) return 0;
  return 1;
}

static int run(int B, const int* P, const int* T, const int* N, int w, int layer, int l0, int Hq,
               int Hkv, int D, int mode, int zero_gate) {
  int S = 1, Lc = 1;
  for (int b = 0; b < B; ++b) {
    const int r = P[b] + T[b] + N[b];
    const int c = speechkv_oracle_compressed_len(P[b], T[b], N[b], w, layer, l0);
    if (r > S) S = r;
    if (c + 2 > Lc) Lc = c + 2;
  }
  const size_t raw = (size_t)B * S * Hkv * D, hat = (size_t)B * Lc * Hkv * D;
  const size_t qn = (size_t)B * S * Hq * D;
  double *k = vec(raw), *v = vec(raw), *u = zero_gate ? NULL : vec((size_t)Hkv * D);
  double *kh = vec(hat), *vh = vec(hat), *q = vec(qn), *dout = vec(qn);
  double *out = vec(qn), *lse = vec((size_t)B * Hq * S), *dq = vec(qn);
  double *dkh = vec(hat), *dvh = vec(hat), *dk = vec(raw), *dv = vec(raw), *du = vec((size_t)Hkv * D);
  double *dq1 = vec((size_t)B * Hq * D), *do1 = vec((size_t)B * Hq * D), *dl1 = vec((size_t)B * Hq);
  int* clen = malloc(sizeof(int) * B);
  const double scale = 1.0 / sqrt((double)D);
  int ok = 1;
  speechkv_oracle_pool(k, v, B, S, Hkv, D, P, T, N, w, layer, l0, u, kh, vh, Lc, clen);
  ok &= finite(kh, hat) && finite(vh, hat);
  speechkv_oracle_attention(q, kh, vh, B, S, Hq, Hkv, D, Lc, P, T, N, w, layer, l0, mode, scale, out,
                            lse);
  ok &= finite(out, qn);
  speechkv_oracle_decode(dq1, kh, vh, clen, B, Hq, Hkv, D, Lc, scale, do1, dl1);
  ok &= finite(do1, (size_t)B * Hq * D);
  speechkv_oracle_attention_bwd(q, kh, vh, B, S, Hq, Hkv, D, Lc, P, T, N, w, layer, l0, mode, scale,
                                dout, dq, dkh, dvh);
  ok &= finite(dq, qn) && finite(dkh, hat) && finite(dvh, hat);
  speechkv_oracle_pool_bwd(k, v, B, S, Hkv, D, P, T, N, w, layer, l0, u, dkh, dvh, Lc, dk, dv, du);
  ok &= finite(dk, raw) && finite(dv, raw) && finite(du, (size_t)Hkv * D);
  free(k); free(v); free(u); free(kh); free(vh); free(q); free(dout); free(out); free(lse);
  free(dq); free(dkh); free(dvh); free(dk); free(dv); free(du); free(dq1); free(do1); free(dl1);
  free(clen);
  if (!ok) printf("FAIL B=%d w=%d layer=%d l0=%d Hq=%d Hkv=%d D=%d mode=%d\n", B, w, layer, l0, Hq, Hkv, D, mode);
  return ok;
}

int main(void) {
  int cases = 0, ok = 1;
  {
    const int P[3] = {5, 0, 9}, T[3] = {13, 7, 0}, N[3] = {3, 2, 0};
    for (int mode = 0; mode < 2; ++mode)
      for (int w = 1; w <= 9; w += 2) {
        ok &= run(3, P, T, N, w, 1, 0, 4, 2, 8, mode, 0);
        ++cases;
      }
  }
  {
    const int P[2] = {0, 4}, T[2] = {3, 30}, N[2] = {0, 5};
    ok &= run(2, P, T, N, 8, 1, 0, 8, 2, 16, 0, 1);  /* zero gate, w > T */
    ok &= run(2, P, T, N, 4, 2, 5, 4, 4, 8, 0, 0);   /* layer below l0 */
    ok &= run(2, P, T, N, 4, 3, 3, 8, 1, 8, 1, 0);   /* one KV head, G = 8 */
    cases += 3;
  }
  {
    const int P[1] = {0}, T[1] = {0}, N[1] = {4};
    ok &= run(1, P, T, N, 4, 1, 0, 2, 2, 8, 0, 0);   /* text only */
    ++cases;
  }
  printf("%s %d\n", ok ? "ok" : "failed", cases);
  return ok ? 0 : 1;
}
