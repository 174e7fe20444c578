/*
 * speechkv_oracle.c - fp64 CPU oracle of SpeechKV's pooling and attention.
 *
 * TEST INFRASTRUCTURE.  This file is the plain, slow, obviously correct
 * statement of what the SpeechKV hot path computes, used only to check the GPU
 * library: by the tests, by the package's smoke check and by the benchmark's
 * CPU-baseline leg.  Nothing in the product path may call it.  It shares no
 * source, header or helper with the GPU library and includes nothing of it.
 *
 * Source of every formula: arXiv 2607.06827, Sec. III-B (Eq. 4 for the
 * pooling, Eq. 5 and the sentence after it for attention over the compressed
 * sequence) and Sec. III-C (pool once at prefill, decode over the stored
 * compressed cache; in training the pooling runs inside the forward pass and
 * is optimised jointly with the rest of the model, so gradients flow through
 * the attention and the pooling to the queries, the raw keys and values and
 * the gate: the *_bwd functions are the chain rule of Eq. 4 and Eq. 5).  Everything is double precision; the inputs are whatever
 * the caller passes (the tests pass bf16 or fp32 values widened to double).
 *
 * Readings taken where the paper is silent (each also listed in the design
 * notes of the repository):
 *   - layers are 0-indexed and layer l is compressed iff l >= l0;
 *   - windows start at the first speech frame; a last window shorter than w
 *     (T % w != 0) is pooled over the frames it has, so nW = ceil(T / w);
 *   - the gate is g(k) = u . k per KV head; its bias cancels in the window
 *     softmax and is not taken;
 *   - a pooled key becomes visible at the last frame of its window
 *     (mask mode 0) or at its first frame (mask mode 1);
 *   - a row that sees no key returns 0 and log-sum-exp -inf;
 *   - query head h reads KV head h / (Hq / Hkv).
 *
 * Parity pins: every function here is pinned by the CPU tests (closed forms,
 * a library attention routine for w = 1, brute force on tiny shapes,
 * invariants and the paper's printed KV-memory ratios; the gradients by
 * central finite differences of the forward functions, a library autograd
 * attention for w = 1 and closed forms at the zero gate).
 *
 * Dense layouts (row-major, last index fastest):
 *   raw K/V      [B][S][Hkv][D]
 *   K^, V^       [B][Lc][Hkv][D]   (Lc >= every compressed length)
 *   prefill Q/O  [B][Sq][Hq][D],   LSE [B][Hq][Sq]
 *   decode q/o   [B][Hq][D],       LSE [B][Hq]
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Effective window of a layer: compression starts at layer l0 (Sec. III-B). */
static int window_of_layer(int w, int layer, int l0) {
  return layer >= l0 ? w : 1;
}

/* Number of windows covering T speech frames, the last one possibly short. */
static int windows_for(int T, int weff) { return (T + weff - 1) / weff; }

int speechkv_oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* P + nW + N: the length of the compressed sequence (Sec. III-B/C). */
int speechkv_oracle_compressed_len(int P, int T, int N, int w, int layer,
                                   int l0) {
  int weff = window_of_layer(w, layer, l0);
  return P + windows_for(T, weff) + N;
}

/*
 * Pooling operator P_R of Eq. 4 applied to one layer's keys and values.
 * Text rows are copied unchanged; each window of speech rows becomes one row,
 * the alpha-weighted sum of its keys (and, with the same alpha, its values),
 * alpha being the softmax over the window of the gate logits u[g] . k_j.
 * Rows of K^/V^ at or beyond a sequence's compressed length are set to 0.
 */
void speechkv_oracle_pool(const double* k_raw, const double* v_raw, int B,
                          int S, int Hkv, int D, const int* P, const int* T,
                          const int* N, int w, int layer, int l0,
                          const double* u, double* k_hat, double* v_hat,
                          int Lc, int* clen) {
  int weff = window_of_layer(w, layer, l0);
  memset(k_hat, 0, sizeof(double) * (size_t)B * Lc * Hkv * D);
  memset(v_hat, 0, sizeof(double) * (size_t)B * Lc * Hkv * D);
#pragma omp parallel for collapse(2) schedule(static)
  for (int b = 0; b < B; ++b) {
    for (int g = 0; g < Hkv; ++g) {
      int nW = windows_for(T[b], weff);
      double* logit = (double*)malloc(sizeof(double) * (size_t)weff);
      double* alpha = (double*)malloc(sizeof(double) * (size_t)weff);
#define RAW(arr, s) (arr + (((size_t)b * S + (s)) * Hkv + g) * D)
#define HAT(arr, c) (arr + (((size_t)b * Lc + (c)) * Hkv + g) * D)
      /* text before the speech: unchanged */
      for (int c = 0; c < P[b]; ++c) {
        memcpy(HAT(k_hat, c), RAW(k_raw, c), sizeof(double) * D);
        memcpy(HAT(v_hat, c), RAW(v_raw, c), sizeof(double) * D);
      }
      /* speech: one row per window */
      for (int i = 0; i < nW; ++i) {
        int first = P[b] + i * weff;
        int end = P[b] + (i + 1) * weff;
        if (end > P[b] + T[b]) end = P[b] + T[b];
        int n = end - first;
        /* gate logit of every key of the window */
        for (int j = 0; j < n; ++j) {
          const double* k = RAW(k_raw, first + j);
          double s = 0.0;
          for (int e = 0; e < D; ++e) s += (u ? u[(size_t)g * D + e] : 0.0) * k[e];
          logit[j] = s;
        }
        /* softmax over the window */
        double m = logit[0];
        for (int j = 1; j < n; ++j)
          if (logit[j] > m) m = logit[j];
        double z = 0.0;
        for (int j = 0; j < n; ++j) z += exp(logit[j] - m);
        for (int j = 0; j < n; ++j) alpha[j] = exp(logit[j] - m) / z;
        /* the same weights pool the keys and the values */
        double* kh = HAT(k_hat, P[b] + i);
        double* vh = HAT(v_hat, P[b] + i);
        for (int e = 0; e < D; ++e) {
          double ks = 0.0, vs = 0.0;
          for (int j = 0; j < n; ++j) {
            ks += alpha[j] * RAW(k_raw, first + j)[e];
            vs += alpha[j] * RAW(v_raw, first + j)[e];
          }
          kh[e] = ks;
          vh[e] = vs;
        }
      }
      /* text after the speech: unchanged, moved up to follow the windows */
      for (int m = 0; m < N[b]; ++m) {
        memcpy(HAT(k_hat, P[b] + nW + m), RAW(k_raw, P[b] + T[b] + m),
               sizeof(double) * D);
        memcpy(HAT(v_hat, P[b] + nW + m), RAW(v_raw, P[b] + T[b] + m),
               sizeof(double) * D);
      }
#undef RAW
#undef HAT
      free(logit);
      free(alpha);
    }
  }
  for (int b = 0; b < B; ++b)
    clen[b] = speechkv_oracle_compressed_len(P[b], T[b], N[b], w, layer, l0);
}

/*
 * Full-resolution position from which compressed key c may be attended
 * (the causality requirement stated after Eq. 5).  Prefix and suffix keys are
 * single positions; a pooled key stands for a whole window and is dated by the
 * window's last frame (mode 0) or first frame (mode 1).
 */
static int visible_from(int c, int P, int T, int nW, int weff, int mode) {
  if (c < P) return c;
  if (c < P + nW) {
    int i = c - P;
    if (mode == 1) return P + i * weff;
    int last = P + (i + 1) * weff - 1;
    return last < P + T - 1 ? last : P + T - 1;
  }
  return P + T + (c - P - nW);
}

/*
 * Eq. 5 for every full-resolution query row p < P+T+N of every sequence:
 * out[b,p,h] = softmax over visible c of scale * q . k^_c, times v^_c.
 * Rows at or beyond P+T+N get out = 0 and lse = NaN (undefined).
 */
void speechkv_oracle_attention(const double* q, const double* k_hat,
                               const double* v_hat, int B, int Sq, int Hq,
                               int Hkv, int D, int Lc, const int* P,
                               const int* T, const int* N, int w, int layer,
                               int l0, int mask_mode, double scale, double* out,
                               double* lse) {
  int weff = window_of_layer(w, layer, l0);
  int group = Hq / Hkv;
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int b = 0; b < B; ++b) {
    for (int h = 0; h < Hq; ++h) {
      int g = h / group;
      int nW = windows_for(T[b], weff);
      int len = P[b] + nW + N[b];
      int rows = P[b] + T[b] + N[b];
      double* z = (double*)malloc(sizeof(double) * (size_t)(len > 0 ? len : 1));
      for (int p = 0; p < Sq; ++p) {
        double* o = out + (((size_t)b * Sq + p) * Hq + h) * D;
        double* l = lse ? lse + ((size_t)b * Hq + h) * Sq + p : NULL;
        for (int e = 0; e < D; ++e) o[e] = 0.0;
        if (p >= rows) {
          if (l) *l = NAN;
          continue;
        }
        const double* qr = q + (((size_t)b * Sq + p) * Hq + h) * D;
        int seen = 0;
        double m = -INFINITY;
        for (int c = 0; c < len; ++c) {
          if (visible_from(c, P[b], T[b], nW, weff, mask_mode) > p) {
            z[c] = -INFINITY;
            continue;
          }
          const double* k = k_hat + (((size_t)b * Lc + c) * Hkv + g) * D;
          double s = 0.0;
          for (int e = 0; e < D; ++e) s += qr[e] * k[e];
          z[c] = scale * s;
          if (z[c] > m) m = z[c];
          ++seen;
        }
        if (!seen) {
          if (l) *l = -INFINITY;
          continue;
        }
        double sum = 0.0;
        for (int c = 0; c < len; ++c)
          if (z[c] != -INFINITY) sum += exp(z[c] - m);
        for (int c = 0; c < len; ++c) {
          if (z[c] == -INFINITY) continue;
          double pc = exp(z[c] - m) / sum;
          const double* v = v_hat + (((size_t)b * Lc + c) * Hkv + g) * D;
          for (int e = 0; e < D; ++e) o[e] += pc * v[e];
        }
        if (l) *l = m + log(sum);
      }
      free(z);
    }
  }
}

/*
 * One decoding step (Sec. III-C): the newest token, whose key and value are
 * already in the cache, attends to every cached key c < clen[b].
 */
void speechkv_oracle_decode(const double* q, const double* k_hat,
                            const double* v_hat, const int* clen, int B,
                            int Hq, int Hkv, int D, int Lc, double scale,
                            double* out, double* lse) {
  int group = Hq / Hkv;
#pragma omp parallel for collapse(2) schedule(static)
  for (int b = 0; b < B; ++b) {
    for (int h = 0; h < Hq; ++h) {
      int g = h / group;
      int len = clen[b];
      const double* qr = q + ((size_t)b * Hq + h) * D;
      double* o = out + ((size_t)b * Hq + h) * D;
      for (int e = 0; e < D; ++e) o[e] = 0.0;
      if (len <= 0) {
        if (lse) lse[(size_t)b * Hq + h] = -INFINITY;
        continue;
      }
      double* z = (double*)malloc(sizeof(double) * (size_t)len);
      double m = -INFINITY;
      for (int c = 0; c < len; ++c) {
        const double* k = k_hat + (((size_t)b * Lc + c) * Hkv + g) * D;
        double s = 0.0;
        for (int e = 0; e < D; ++e) s += qr[e] * k[e];
        z[c] = scale * s;
        if (z[c] > m) m = z[c];
      }
      double sum = 0.0;
      for (int c = 0; c < len; ++c) sum += exp(z[c] - m);
      for (int c = 0; c < len; ++c) {
        double pc = exp(z[c] - m) / sum;
        const double* v = v_hat + (((size_t)b * Lc + c) * Hkv + g) * D;
        for (int e = 0; e < D; ++e) o[e] += pc * v[e];
      }
      if (lse) lse[(size_t)b * Hq + h] = m + log(sum);
      free(z);
    }
  }
}

/*
 * Gradient of Eq. 5 (every full-resolution row over the compressed keys it
 * may see, the same mask as speechkv_oracle_attention) with respect to Q, K^
 * and V^, given the gradient dO of the output.  Per query row p and head h,
 * with pi = softmax_c(z), z_c = scale * q . k^_c over the visible keys and
 * o = sum_c pi_c v^_c, the chain rule gives
 *   dv^_c += pi_c dO                         (o is linear in v^)
 *   dpi_c  = dO . v^_c
 *   dz_c   = pi_c (dpi_c - sum_c' pi_c' dpi_c')   (softmax Jacobian)
 *   dq     = scale sum_c dz_c k^_c
 *   dk^_c += scale dz_c q
 * Key gradients sum over the query heads that share KV head g and over rows.
 * Rows that see no key and rows at or beyond P+T+N contribute nothing; dq is 0
 * there.  dk^/dv^ rows at or beyond a sequence's compressed length stay 0.
 */
void speechkv_oracle_attention_bwd(const double* q, const double* k_hat,
                                   const double* v_hat, int B, int Sq, int Hq,
                                   int Hkv, int D, int Lc, const int* P,
                                   const int* T, const int* N, int w, int layer,
                                   int l0, int mask_mode, double scale,
                                   const double* dout, double* dq,
                                   double* dk_hat, double* dv_hat) {
  int weff = window_of_layer(w, layer, l0);
  int group = Hq / Hkv;
  memset(dq, 0, sizeof(double) * (size_t)B * Sq * Hq * D);
  memset(dk_hat, 0, sizeof(double) * (size_t)B * Lc * Hkv * D);
  memset(dv_hat, 0, sizeof(double) * (size_t)B * Lc * Hkv * D);
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int b = 0; b < B; ++b) {
    for (int g = 0; g < Hkv; ++g) {
      int nW = windows_for(T[b], weff);
      int len = P[b] + nW + N[b];
      int rows = P[b] + T[b] + N[b];
      int n = len > 0 ? len : 1;
      double* z = (double*)malloc(sizeof(double) * (size_t)n);
      double* pi = (double*)malloc(sizeof(double) * (size_t)n);
      double* dpi = (double*)malloc(sizeof(double) * (size_t)n);
      for (int h = g * group; h < (g + 1) * group; ++h) {
        for (int p = 0; p < rows && p < Sq; ++p) {
          const double* qr = q + (((size_t)b * Sq + p) * Hq + h) * D;
          const double* go = dout + (((size_t)b * Sq + p) * Hq + h) * D;
          double* gq = dq + (((size_t)b * Sq + p) * Hq + h) * D;
          /* forward again: the probabilities of row p */
          double m = -INFINITY;
          int seen = 0;
          for (int c = 0; c < len; ++c) {
            z[c] = -INFINITY;
            if (visible_from(c, P[b], T[b], nW, weff, mask_mode) > p) continue;
            const double* k = k_hat + (((size_t)b * Lc + c) * Hkv + g) * D;
            double s = 0.0;
            for (int e = 0; e < D; ++e) s += qr[e] * k[e];
            z[c] = scale * s;
            if (z[c] > m) m = z[c];
            ++seen;
          }
          if (!seen) continue;
          double sum = 0.0;
          for (int c = 0; c < len; ++c)
            if (z[c] != -INFINITY) sum += exp(z[c] - m);
          double mean = 0.0; /* sum_c pi_c dpi_c */
          for (int c = 0; c < len; ++c) {
            pi[c] = z[c] == -INFINITY ? 0.0 : exp(z[c] - m) / sum;
            dpi[c] = 0.0;
            if (z[c] == -INFINITY) continue;
            const double* v = v_hat + (((size_t)b * Lc + c) * Hkv + g) * D;
            for (int e = 0; e < D; ++e) dpi[c] += go[e] * v[e];
            mean += pi[c] * dpi[c];
          }
          for (int c = 0; c < len; ++c) {
            if (z[c] == -INFINITY) continue;
            double dz = pi[c] * (dpi[c] - mean);
            const double* k = k_hat + (((size_t)b * Lc + c) * Hkv + g) * D;
            double* gk = dk_hat + (((size_t)b * Lc + c) * Hkv + g) * D;
            double* gv = dv_hat + (((size_t)b * Lc + c) * Hkv + g) * D;
            for (int e = 0; e < D; ++e) {
              gq[e] += scale * dz * k[e];
              gk[e] += scale * dz * qr[e];
              gv[e] += pi[c] * go[e];
            }
          }
        }
      }
      free(z);
      free(pi);
      free(dpi);
    }
  }
}

/*
 * Gradient of the pooling P_R of Eq. 4 with respect to the raw keys, the raw
 * values and the gate vectors u, given dK^ and dV^ ([B][Lc][Hkv][D]).
 * A text row was copied, so its gradient is the gradient of the row it
 * became.  For window i with frames j, logits s_j = u[g] . k_j and
 * alpha = softmax_j(s):
 *   dalpha_j = dK^_i . k_j + dV^_i . v_j      (k^ and v^ are linear in alpha)
 *   ds_j     = alpha_j (dalpha_j - sum_j' alpha_j' dalpha_j')
 *   dk_j     = alpha_j dK^_i + ds_j u[g]       (k_j enters k^ and its own logit)
 *   dv_j     = alpha_j dV^_i
 *   du[g]   += ds_j k_j                        (summed over sequences and windows)
 * u = NULL is the zero gate; du is still its gradient.  Raw rows at or beyond
 * P+T+N get 0.
 */
void speechkv_oracle_pool_bwd(const double* k_raw, const double* v_raw, int B,
                              int S, int Hkv, int D, const int* P, const int* T,
                              const int* N, int w, int layer, int l0,
                              const double* u, const double* dk_hat,
                              const double* dv_hat, int Lc, double* dk_raw,
                              double* dv_raw, double* du) {
  int weff = window_of_layer(w, layer, l0);
  memset(dk_raw, 0, sizeof(double) * (size_t)B * S * Hkv * D);
  memset(dv_raw, 0, sizeof(double) * (size_t)B * S * Hkv * D);
  memset(du, 0, sizeof(double) * (size_t)Hkv * D);
#pragma omp parallel for schedule(static)
  for (int g = 0; g < Hkv; ++g) {
    double* logit = (double*)malloc(sizeof(double) * (size_t)weff);
    double* alpha = (double*)malloc(sizeof(double) * (size_t)weff);
    double* dalpha = (double*)malloc(sizeof(double) * (size_t)weff);
    for (int b = 0; b < B; ++b) {
      int nW = windows_for(T[b], weff);
#define RAW(arr, s) (arr + (((size_t)b * S + (s)) * Hkv + g) * D)
#define HAT(arr, c) (arr + (((size_t)b * Lc + (c)) * Hkv + g) * D)
      for (int c = 0; c < P[b]; ++c) {
        memcpy(RAW(dk_raw, c), HAT(dk_hat, c), sizeof(double) * D);
        memcpy(RAW(dv_raw, c), HAT(dv_hat, c), sizeof(double) * D);
      }
      for (int i = 0; i < nW; ++i) {
        int first = P[b] + i * weff;
        int end = P[b] + (i + 1) * weff;
        if (end > P[b] + T[b]) end = P[b] + T[b];
        int n = end - first;
        const double* gk = HAT(dk_hat, P[b] + i);
        const double* gv = HAT(dv_hat, P[b] + i);
        /* forward again: the window's weights */
        for (int j = 0; j < n; ++j) {
          const double* k = RAW(k_raw, first + j);
          double s = 0.0;
          for (int e = 0; e < D; ++e) s += (u ? u[(size_t)g * D + e] : 0.0) * k[e];
          logit[j] = s;
        }
        double m = logit[0];
        for (int j = 1; j < n; ++j)
          if (logit[j] > m) m = logit[j];
        double z = 0.0;
        for (int j = 0; j < n; ++j) z += exp(logit[j] - m);
        double mean = 0.0; /* sum_j alpha_j dalpha_j */
        for (int j = 0; j < n; ++j) {
          alpha[j] = exp(logit[j] - m) / z;
          const double* k = RAW(k_raw, first + j);
          const double* v = RAW(v_raw, first + j);
          double d = 0.0;
          for (int e = 0; e < D; ++e) d += gk[e] * k[e] + gv[e] * v[e];
          dalpha[j] = d;
          mean += alpha[j] * d;
        }
        for (int j = 0; j < n; ++j) {
          double ds = alpha[j] * (dalpha[j] - mean);
          const double* k = RAW(k_raw, first + j);
          double* dk = RAW(dk_raw, first + j);
          double* dv = RAW(dv_raw, first + j);
          for (int e = 0; e < D; ++e) {
            dk[e] = alpha[j] * gk[e] + ds * (u ? u[(size_t)g * D + e] : 0.0);
            dv[e] = alpha[j] * gv[e];
            du[(size_t)g * D + e] += ds * k[e];
          }
        }
      }
      for (int m = 0; m < N[b]; ++m) {
        memcpy(RAW(dk_raw, P[b] + T[b] + m), HAT(dk_hat, P[b] + nW + m),
               sizeof(double) * D);
        memcpy(RAW(dv_raw, P[b] + T[b] + m), HAT(dv_hat, P[b] + nW + m),
               sizeof(double) * D);
      }
#undef RAW
#undef HAT
    }
    free(logit);
    free(alpha);
    free(dalpha);
  }
}
