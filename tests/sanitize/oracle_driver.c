/* Runs every function of the C oracle once or twice on small shapes, including the degenerate
 * ones (no visual keys, no tokens, one layer, rank 1, ragged sizes), with every buffer exactly
 * as large as its shape, so that a build with AddressSanitizer and UndefinedBehaviorSanitizer
 * reports any access outside a buffer or any undefined operation. Prints "ok" on success. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

double dvref_act(double x, int act);
void dvref_down(const double* X, const double* Dw, int64_t T, int d, int L, int r, int act, double* Z);
void dvref_memory(const double* E, const double* Z, const double* Uw, int64_t T, int d, int L, int r,
                  double* M);
void dvref_memory_recurrent(const double* E, const double* Dw, const double* Uw, int64_t T, int d,
                            int L, int r, int act, double* M);
void dvref_rmsnorm(const double* x, const double* gamma, int d, double eps, double* out);
void dvref_visual_kv(const double* M, const double* gamma, const double* Wk, const double* Wv,
                     int B, int Nv, int d, int L, int Hkv, int hd, double eps, double* Kv, double* Vv);
int dvref_kv_epilogue(double* Kv, double* Vv, int L, int B, int Hkv, int Nv, int hd,
                      const double* k_bias, const double* v_bias, const double* k_norm,
                      double kn_eps, const int* pos, int sec0, int sec1, int sec2, double theta);
int dvref_delta_rule(const double* k, const double* v, const double* alpha, const double* beta,
                     double* S, int B, int Hk, int Hv, int N, int dk, int dv);
int dvref_text_visual_attention(const double* Q, const double* Kv, const double* Vv,
                                const double* Kt, const double* Vt, double* O, int B, int Hq,
                                int Hkv, int hd, int Nv, int Nq, int Nkt, int q_pos0, double scale);

static uint64_t g_state = 88172645463325252ull;
static double next_value(void) { /* xorshift64, values in [-1, 1) */
  g_state ^= g_state << 13;
  g_state ^= g_state >> 7;
  g_state ^= g_state << 17;
  return (double)(g_state >> 11) / (double)(1ull << 52) - 1.0;
}
static double* buf(size_t n) {
  double* p = (double*)malloc(sizeof(double) * (n ? n : 1));
  for (size_t i = 0; i < n; ++i) p[i] = next_value();
  return p;
}
static int finite_all(const double* p, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (!isfinite(p[i])) return 0;
  return 1;
}
#define CHECK(cond, what)                      \
  do {                                         \
    if (!(cond)) {                             \
      fprintf(stderr, "failed: %s\n", what);   \
      return 1;                                \
    }                                          \
  } while (0)

static int build_case(int B, int Nv, int d, int L, int r, int Hkv, int hd, int act) {
  const int64_t T = (int64_t)B * Nv;
  const size_t kv = (size_t)Hkv * hd;
  double *E = buf(T * d), *Dw = buf((size_t)L * r * d), *Uw = buf((size_t)L * d * r);
  double *g = buf((size_t)L * d), *Wk = buf((size_t)L * kv * d), *Wv = buf((size_t)L * kv * d);
  double *Z = buf((size_t)L * T * r), *M = buf((size_t)L * T * d);
  double *Kv = buf((size_t)L * T * kv), *Vv = buf((size_t)L * T * kv), *n = buf(d);
  dvref_down(E, Dw, T, d, L, r, act, Z);
  CHECK(finite_all(Z, (size_t)L * T * r), "down");
  dvref_memory(E, Z, Uw, T, d, L, r, M);
  CHECK(finite_all(M, (size_t)L * T * d), "memory");
  dvref_rmsnorm(M, g, d, 1e-5, n);
  CHECK(finite_all(n, d), "rmsnorm");
  dvref_visual_kv(M, g, Wk, Wv, B, Nv, d, L, Hkv, hd, 1e-5, Kv, Vv);
  CHECK(finite_all(Kv, (size_t)L * T * kv), "visual_kv");
  dvref_memory_recurrent(E, Dw, Uw, T, d, L, r, act, M);
  CHECK(finite_all(M, (size_t)L * T * d), "memory_recurrent");
  double *kb = buf((size_t)L * kv), *vb = buf((size_t)L * kv), *kn = buf((size_t)L * hd);
  int* pos = (int*)malloc(sizeof(int) * (size_t)B * 3 * (Nv ? Nv : 1));
  for (int64_t i = 0; i < (int64_t)B * 3 * Nv; ++i) pos[i] = (int)(i % 97);
  CHECK(dvref_kv_epilogue(Kv, Vv, L, B, Hkv, Nv, hd, kb, vb, kn, 1e-6, pos, hd / 2, 0, 0, 1e4) == 0,
        "epilogue 1-D");
  const int s0 = hd / 8, s1 = (hd / 2 - s0) / 2, s2 = hd / 2 - s0 - s1;
  CHECK(dvref_kv_epilogue(Kv, Vv, L, B, Hkv, Nv, hd, kb, NULL, kn, 1e-6, pos, s0, s1, s2, 1e6) == 0,
        "epilogue sections");
  CHECK(dvref_kv_epilogue(Kv, Vv, L, B, Hkv, Nv, hd, NULL, NULL, NULL, 0.0, NULL, hd / 2, 0, 0, 1.0) == 0,
        "epilogue none");
  CHECK(finite_all(Kv, (size_t)L * T * kv), "epilogue output");
  free(E); free(Dw); free(Uw); free(g); free(Wk); free(Wv); free(Z); free(M); free(Kv); free(Vv);
  free(n); free(kb); free(vb); free(kn); free(pos);
  return 0;
}

static int attention_case(int B, int Hq, int Hkv, int hd, int Nv, int Nq, int Nkt, int q0) {
  double *Q = buf((size_t)B * Nq * Hq * hd), *Kv = buf((size_t)B * Hkv * Nv * hd);
  double *Vv = buf((size_t)B * Hkv * Nv * hd), *Kt = buf((size_t)B * Hkv * Nkt * hd);
  double *Vt = buf((size_t)B * Hkv * Nkt * hd), *O = buf((size_t)B * Nq * Hq * hd);
  CHECK(dvref_text_visual_attention(Q, Kv, Vv, Kt, Vt, O, B, Hq, Hkv, hd, Nv, Nq, Nkt, q0,
                                    1.0 / sqrt((double)hd)) == 0, "attention");
  CHECK(finite_all(O, (size_t)B * Nq * Hq * hd), "attention output");
  CHECK(dvref_text_visual_attention(Q, Kv, Vv, Kt, Vt, O, B, Hq, Hkv, hd, Nv, Nq, Nq + q0 - 1, q0,
                                    1.0) == -1, "attention rejects a short text cache");
  free(Q); free(Kv); free(Vv); free(Kt); free(Vt); free(O);
  return 0;
}

static int delta_case(int B, int Hk, int Hv, int N, int dk, int dv) {
  double *k = buf((size_t)B * Hk * N * dk), *v = buf((size_t)B * Hv * N * dv);
  double *a = buf((size_t)B * Hv * N), *b = buf((size_t)B * Hv * N), *S = buf((size_t)B * Hv * dk * dv);
  for (size_t i = 0; i < (size_t)B * Hv * N; ++i) a[i] = 0.5 + 0.5 * fabs(a[i]);
  CHECK(dvref_delta_rule(k, v, a, b, S, B, Hk, Hv, N, dk, dv) == 0, "delta rule");
  CHECK(finite_all(S, (size_t)B * Hv * dk * dv), "delta rule state");
  free(k); free(v); free(a); free(b); free(S);
  return 0;
}

int main(void) {
  CHECK(dvref_act(0.0, 0) == 0.0 && dvref_act(0.0, 1) == 0.0, "act");
  if (build_case(1, 5, 8, 2, 3, 2, 4, 0)) return 1;    /* ragged, rank 3 */
  if (build_case(2, 3, 16, 1, 1, 1, 8, 1)) return 1;   /* one layer, rank 1, GELU */
  if (build_case(3, 7, 12, 3, 4, 3, 2, 0)) return 1;
  if (attention_case(2, 4, 2, 8, 9, 3, 12, 4)) return 1; /* GQA, longer text cache */
  if (attention_case(1, 2, 2, 4, 0, 5, 5, 0)) return 1;  /* no visual keys */
  if (attention_case(3, 3, 1, 6, 1, 1, 7, 6)) return 1;  /* decode-like single query */
  if (delta_case(2, 1, 2, 7, 4, 3)) return 1;
  if (delta_case(1, 2, 4, 0, 8, 8)) return 1;            /* no tokens */
  if (delta_case(1, 1, 1, 1, 2, 5)) return 1;
  printf("ok\n");
  return 0;
}
