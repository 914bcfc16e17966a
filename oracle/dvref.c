/*
 * Oracle for the visual-memory path: a plain, slow, obviously correct CPU
 * implementation in fp64. TEST INFRASTRUCTURE ONLY: it is called by the tests,
 * by the smoke check and by the benchmark's CPU-baseline leg, never by the
 * product path. It shares no code, header or table with the GPU library.
 *
 * Every function is a literal transcription of a definition of the paper
 * "Just MLPs: Efficient Visual State Reconstruction for Multimodal Language
 * Models" (delta-Vision):
 *   Section 3.1, Eq. 4   adapter A_l(X) = X + phi(X D_l) U_l
 *   Section 3.1, Eq. 5   embedding adapter  M_l = A_l(E)
 *   Section 3.1, Eq. 6   recurrent adapter  M_0 = E, M_l = A_l(M_{l-1})
 *   Section 3.2, Eq. 7   visual K/V = W_{K,l} LN_l(M_l), W_{V,l} LN_l(M_l)
 *   Section 3.2, Eq. 9   text queries attend to [K^v; K^t], [V^v; V^t] with the
 *                        causal structure kept for the text part
 *   Appendix on linear attention, Eq. 15-16: gated delta-rule write of the visual
 *                        tokens into a Gated DeltaNet recurrent state
 *
 * Readings where the paper is silent (each is listed with its reason in the
 * design notes of the repository):
 *   - weights are stored out x in (the nn.Linear convention): Dw[l] = D_l^T
 *     [r,d], Uw[l] = U_l^T [d,r], Wk[l], Wv[l] [Hkv*hd, d];
 *   - LN_l is the backbone's RMSNorm: x * (mean(x^2) + eps)^-1/2 * gamma_l
 *     (Appendix K names RMSNorm as the frozen norm);
 *   - phi is SiLU (Section 3.1); the exact erf GELU is accepted as a second
 *     activation for workloads that name it;
 *   - the softmax scale is an argument (1/sqrt(hd) by default, as in the
 *     read-out of Appendix K);
 *   - query head h reads key/value head h / (Hq/Hkv);
 *   - no positional rotation is applied to visual keys by Eq. 7 itself; the
 *     backbone epilogue (bias, per-head key norm, rotary embedding at the
 *     visual tokens' unchanged positions) is a separate, optional step.
 *
 * Sums run sequentially in fp64. OpenMP only distributes independent output
 * elements over threads; it changes no arithmetic.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define DVREF_ACT_SILU 0
#define DVREF_ACT_GELU 1

/* phi of Eq. 4: SiLU(x) = x * sigmoid(x); GELU(x) = x * Phi(x) with the standard normal CDF
 * Phi(x) = erfc(-x / sqrt 2) / 2 (the erfc form avoids cancellation for negative x). */
double dvref_act(double x, int act) {
  if (act == DVREF_ACT_SILU) return x / (1.0 + exp(-x));
  return 0.5 * x * erfc(-x / sqrt(2.0));
}

/* Eq. 4 (down half) for every layer: Z[l][t][j] = phi( sum_k X[t][k] * D_l[k][j] )
 * with D_l[k][j] = Dw[l][j][k].  X [T,d], Dw [L,r,d], Z [L,T,r]. */
void dvref_down(const double* X, const double* Dw, int64_t T, int d, int L, int r, int act,
                double* Z) {
  for (int l = 0; l < L; ++l) {
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t) {
      for (int j = 0; j < r; ++j) {
        const double* x = X + t * d;
        const double* w = Dw + ((int64_t)l * r + j) * d;
        double s = 0.0;
        for (int k = 0; k < d; ++k) s += x[k] * w[k];
        Z[((int64_t)l * T + t) * r + j] = dvref_act(s, act);
      }
    }
  }
}

/* Eq. 4-5: M_l[t][n] = E[t][n] + sum_j Z_l[t][j] * U_l[j][n], U_l[j][n] = Uw[l][n][j].
 * E [T,d], Z [L,T,r], Uw [L,d,r], M [L,T,d]. */
void dvref_memory(const double* E, const double* Z, const double* Uw, int64_t T, int d, int L,
                  int r, double* M) {
  for (int l = 0; l < L; ++l) {
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t) {
      const double* z = Z + ((int64_t)l * T + t) * r;
      for (int n = 0; n < d; ++n) {
        const double* u = Uw + ((int64_t)l * d + n) * r;
        double s = 0.0;
        for (int j = 0; j < r; ++j) s += z[j] * u[j];
        M[((int64_t)l * T + t) * d + n] = E[t * d + n] + s;
      }
    }
  }
}

/* Eq. 6: M_0 = E; layer l (0-based here) applies A_l to the previous memory,
 * M_l = M_{l-1} + phi(M_{l-1} D_l) U_l, so the first layer's memory is A_0(E).
 * E [T,d], Dw [L,r,d], Uw [L,d,r], M [L,T,d]. */
void dvref_memory_recurrent(const double* E, const double* Dw, const double* Uw, int64_t T,
                            int d, int L, int r, int act, double* M) {
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < T; ++t) {
    double* z = (double*)malloc(sizeof(double) * (size_t)r);
    for (int l = 0; l < L; ++l) {
      const double* prev = (l == 0) ? E + t * d : M + ((int64_t)(l - 1) * T + t) * d;
      double* cur = M + ((int64_t)l * T + t) * d;
      for (int j = 0; j < r; ++j) {
        const double* w = Dw + ((int64_t)l * r + j) * d;
        double s = 0.0;
        for (int k = 0; k < d; ++k) s += prev[k] * w[k];
        z[j] = dvref_act(s, act);
      }
      for (int n = 0; n < d; ++n) {
        const double* u = Uw + ((int64_t)l * d + n) * r;
        double s = 0.0;
        for (int j = 0; j < r; ++j) s += z[j] * u[j];
        cur[n] = prev[n] + s;
      }
    }
    free(z);
  }
}

/* RMSNorm read of LN_l: out[n] = x[n] / sqrt( (1/d) sum_k x[k]^2 + eps ) * gamma[n]. */
void dvref_rmsnorm(const double* x, const double* gamma, int d, double eps, double* out) {
  double ss = 0.0;
  for (int k = 0; k < d; ++k) ss += x[k] * x[k];
  double rho = 1.0 / sqrt(ss / (double)d + eps);
  for (int n = 0; n < d; ++n) out[n] = x[n] * rho * gamma[n];
}

/* Eq. 7: Kv_l = LN_l(M_l) W_{K,l}^T and Vv_l = LN_l(M_l) W_{V,l}^T, stored head-major:
 * Kv[l][b][h][i][c] for token t = b*Nv + i and output channel h*hd + c.
 * M [L,B*Nv,d], gamma [L,d], Wk, Wv [L,Hkv*hd,d], Kv, Vv [L,B,Hkv,Nv,hd]. */
void dvref_visual_kv(const double* M, const double* gamma, const double* Wk, const double* Wv,
                     int B, int Nv, int d, int L, int Hkv, int hd, double eps, double* Kv,
                     double* Vv) {
  const int64_t T = (int64_t)B * Nv;
  const int kv = Hkv * hd;
  for (int l = 0; l < L; ++l) {
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t) {
      double* nrm = (double*)malloc(sizeof(double) * (size_t)d);
      dvref_rmsnorm(M + ((int64_t)l * T + t) * d, gamma + (int64_t)l * d, d, eps, nrm);
      const int64_t b = t / Nv, i = t % Nv;
      for (int o = 0; o < kv; ++o) {
        const double* wk = Wk + ((int64_t)l * kv + o) * d;
        const double* wv = Wv + ((int64_t)l * kv + o) * d;
        double sk = 0.0, sv = 0.0;
        for (int k = 0; k < d; ++k) {
          sk += nrm[k] * wk[k];
          sv += nrm[k] * wv[k];
        }
        const int h = o / hd, c = o % hd;
        const int64_t dst = ((((int64_t)l * B + b) * Hkv + h) * Nv + i) * hd + c;
        Kv[dst] = sk;
        Vv[dst] = sv;
      }
      free(nrm);
    }
  }
}

/* Backbone epilogue of the visual keys and values (outside Eq. 7). The paper keeps every
 * visual token at its original position, so a backbone whose attention adds a projection
 * bias, normalises each key head or rotates keys by position does the same to the
 * reconstructed visual K/V. In the backbone's order, per layer l, token (b, i), head h:
 *   K += k_bias[l], V += v_bias[l]                              (projection bias)
 *   K_h <- K_h * (mean_c K_h[c]^2 + kn_eps)^-1/2 * k_norm[l]    (per-head key RMSNorm)
 *   rotary embedding of K_h: channel j < hd/2 pairs with channel j + hd/2 and turns by the
 *   angle p * theta^(-2j/hd), where p = pos[b][a][i] and the position axis a is 0 for
 *   j < sec0, 1 for j < sec0 + sec1 and 2 otherwise (sections of a multimodal rotary
 *   embedding; sec0 = hd/2 is the one-dimensional case):
 *      (k_j, k_{j+hd/2}) <- (k_j cos - k_{j+hd/2} sin,  k_{j+hd/2} cos + k_j sin).
 * NULL k_bias / v_bias / k_norm / pos skips that step. In place on Kv, Vv [L,B,Hkv,Nv,hd];
 * k_bias, v_bias [L, Hkv*hd]; k_norm [L, hd]; pos [B, 3, Nv]. Returns -1 if the sections do
 * not add up to hd/2 (or hd is odd), else 0. */
int dvref_kv_epilogue(double* Kv, double* Vv, int L, int B, int Hkv, int Nv, int hd,
                      const double* k_bias, const double* v_bias, const double* k_norm,
                      double kn_eps, const int* pos, int sec0, int sec1, int sec2, double theta) {
  const int half = hd / 2;
  if (hd % 2 != 0 || sec0 < 0 || sec1 < 0 || sec2 < 0 || sec0 + sec1 + sec2 != half) return -1;
  const int64_t rows = (int64_t)L * B * Hkv * Nv;
#pragma omp parallel for schedule(static)
  for (int64_t row = 0; row < rows; ++row) {
    const int i = (int)(row % Nv);
    const int h = (int)((row / Nv) % Hkv);
    const int b = (int)((row / ((int64_t)Nv * Hkv)) % B);
    const int l = (int)(row / ((int64_t)Nv * Hkv * B));
    double* k = Kv + row * hd;
    double* v = Vv + row * hd;
    if (k_bias)
      for (int c = 0; c < hd; ++c) k[c] += k_bias[(int64_t)l * Hkv * hd + h * hd + c];
    if (v_bias)
      for (int c = 0; c < hd; ++c) v[c] += v_bias[(int64_t)l * Hkv * hd + h * hd + c];
    if (k_norm) {
      double ss = 0.0;
      for (int c = 0; c < hd; ++c) ss += k[c] * k[c];
      const double rho = 1.0 / sqrt(ss / (double)hd + kn_eps);
      for (int c = 0; c < hd; ++c) k[c] = k[c] * rho * k_norm[(int64_t)l * hd + c];
    }
    if (pos) {
      for (int j = 0; j < half; ++j) {
        const int a = j < sec0 ? 0 : (j < sec0 + sec1 ? 1 : 2);
        const double p = (double)pos[((int64_t)b * 3 + a) * Nv + i];
        const double ang = p * pow(theta, -2.0 * (double)j / (double)hd);
        const double cs = cos(ang), sn = sin(ang);
        const double x1 = k[j], x2 = k[j + half];
        k[j] = x1 * cs - x2 * sn;
        k[j + half] = x2 * cs + x1 * sn;
      }
    }
  }
  return 0;
}

/* Visual write into a linear-attention (Gated DeltaNet) state (appendix on linear attention,
 * Eq. 15-16), token by token in order, for every sequence b and value head h (key head
 * h / (Hv/Hk)):
 *     S <- alpha_t * S                                   (gated decay, Eq. 15)
 *     S <- S + beta_t * k_t (v_t - S^T k_t)^T            (delta-rule correction, Eq. 16)
 * k [B,Hk,N,dk], v [B,Hv,N,dv], alpha, beta [B,Hv,N], S [B,Hv,dk,dv] (in/out).
 * Returns -1 if Hv is not a multiple of Hk, else 0. */
int dvref_delta_rule(const double* k, const double* v, const double* alpha, const double* beta,
                     double* S, int B, int Hk, int Hv, int N, int dk, int dv) {
  if (Hk <= 0 || Hv % Hk != 0) return -1;
  const int G = Hv / Hk;
#pragma omp parallel for collapse(2) schedule(static)
  for (int b = 0; b < B; ++b) {
    for (int h = 0; h < Hv; ++h) {
      double* s = S + ((int64_t)b * Hv + h) * dk * dv;
      double* sk = (double*)malloc(sizeof(double) * (size_t)dv);
      for (int t = 0; t < N; ++t) {
        const double* kt = k + (((int64_t)b * Hk + h / G) * N + t) * dk;
        const double* vt = v + (((int64_t)b * Hv + h) * N + t) * dv;
        const double a = alpha[((int64_t)b * Hv + h) * N + t];
        const double be = beta[((int64_t)b * Hv + h) * N + t];
        for (int64_t e = 0; e < (int64_t)dk * dv; ++e) s[e] *= a;
        for (int j = 0; j < dv; ++j) {
          double acc = 0.0;
          for (int i = 0; i < dk; ++i) acc += s[(int64_t)i * dv + j] * kt[i];
          sk[j] = acc;
        }
        for (int i = 0; i < dk; ++i)
          for (int j = 0; j < dv; ++j) s[(int64_t)i * dv + j] += be * kt[i] * (vt[j] - sk[j]);
      }
      free(sk);
    }
  }
  return 0;
}

/* Eq. 9 for one layer. Query (b, i, h) reads key/value head g = h / (Hq/Hkv) and the key set
 * { visual 0..Nv-1 } U { text 0..q_pos0+i }: every visual key, and text keys up to its own
 * position (visual tokens precede the text, Eq. 2, so the causal mask never hides them).
 *   s_j = scale * <Q[b,i,h,:], K_j>,  p = softmax(s),  O[b,i,h,:] = sum_j p_j V_j.
 * Q, O [B,Nq,Hq,hd]; Kv, Vv [B,Hkv,Nv,hd]; Kt, Vt [B,Hkv,Nkt,hd].
 * Returns 0, or -1 if a query position has no text key (q_pos0 + Nq > Nkt). */
int dvref_text_visual_attention(const double* Q, const double* Kv, const double* Vv,
                                const double* Kt, const double* Vt, double* O, int B, int Hq,
                                int Hkv, int hd, int Nv, int Nq, int Nkt, int q_pos0,
                                double scale) {
  if (q_pos0 < 0 || q_pos0 + Nq > Nkt || Hq % Hkv != 0) return -1;
  const int G = Hq / Hkv;
  const int nkeys_max = Nv + Nkt;
#pragma omp parallel for collapse(3) schedule(static)
  for (int b = 0; b < B; ++b) {
    for (int i = 0; i < Nq; ++i) {
      for (int h = 0; h < Hq; ++h) {
        const int g = h / G;
        const double* q = Q + (((int64_t)b * Nq + i) * Hq + h) * hd;
        const double* kv = Kv + ((int64_t)b * Hkv + g) * (int64_t)Nv * hd;
        const double* vv = Vv + ((int64_t)b * Hkv + g) * (int64_t)Nv * hd;
        const double* kt = Kt + ((int64_t)b * Hkv + g) * (int64_t)Nkt * hd;
        const double* vt = Vt + ((int64_t)b * Hkv + g) * (int64_t)Nkt * hd;
        const int ntext = q_pos0 + i + 1;
        const int n = Nv + ntext;
        double* s = (double*)malloc(sizeof(double) * (size_t)nkeys_max);
        for (int j = 0; j < n; ++j) {
          const double* key = (j < Nv) ? kv + (int64_t)j * hd : kt + (int64_t)(j - Nv) * hd;
          double dot = 0.0;
          for (int c = 0; c < hd; ++c) dot += q[c] * key[c];
          s[j] = scale * dot;
        }
        double mx = s[0];
        for (int j = 1; j < n; ++j) mx = s[j] > mx ? s[j] : mx;
        double denom = 0.0;
        for (int j = 0; j < n; ++j) {
          s[j] = exp(s[j] - mx);
          denom += s[j];
        }
        double* o = O + (((int64_t)b * Nq + i) * Hq + h) * hd;
        for (int c = 0; c < hd; ++c) o[c] = 0.0;
        for (int j = 0; j < n; ++j) {
          const double* val = (j < Nv) ? vv + (int64_t)j * hd : vt + (int64_t)(j - Nv) * hd;
          const double p = s[j] / denom;
          for (int c = 0; c < hd; ++c) o[c] += p * val[c];
        }
        free(s);
      }
    }
  }
  return 0;
}
