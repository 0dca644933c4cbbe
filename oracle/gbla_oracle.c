/*
 * gbla_oracle.c -- plain fp64 CPU oracle of the GBLA forward pass.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  The product path
 * (the HIP library and its Python binding) never calls it, and the two share
 * no code, headers, tables or helpers.
 *
 * What it computes, for every sequence s and head h (Gated Bidirectional
 * Linear Attention, Section 2 and Section 2.1 of the paper):
 *
 *   1. Conv1D (Section 2.1, item "Conv1D"; kernel size 4 in Section 3.1).
 *      Causal, depthwise, applied to the projected q, k and v of each head:
 *          xt[i][e] = sum_{t=0}^{W-1} w[h][e][t] * x[i-W+1+t][e],
 *      with x[j] = 0 for j before the start of the sequence.  Tap W-1
 *      multiplies the current token.  No bias, no activation.
 *   2. Feature map (Section 2, "Bidirectional Linear Attention" paragraph):
 *          phi(u) = elu(u) + 1 = u + 1 for u > 0, exp(u) for u <= 0.
 *      exp(u) is evaluated directly (not as (exp(u) - 1) + 1).
 *   3. Key gates (Section 2.1, item "Key gating"): g = softmax over the
 *      tokens of the sequence of the logits a, per head:
 *          g[j] = exp(a[j] - max a) / sum_l exp(a[l] - max a).
 *   4. Global state (matrix form of the key-gating item, K^T V and K^T 1
 *      with K = g (.) phi(K)):
 *          S[c][e] = sum_j g[j] phi(kt[j][c]) vt[j][e]
 *          z[c]    = sum_j g[j] phi(kt[j][c])
 *   5. Readout (same display; Eq. (1) with the gated keys):
 *          o[i][e] = (sum_c phi(qt[i][c]) S[c][e]) / (sum_c phi(qt[i][c]) z[c])
 *   6. Gated RMSNorm (Section 2.1, item "RMSNorm with gating"), over the
 *      d channels of one token of one head:
 *          ms[i]    = (1/d) sum_e o[i][e]^2
 *          oh[i][e] = o[i][e] / sqrt(ms[i] + eps)
 *          y[i][e]  = oh[i][e] * gamma[h][e] * r[i][e] / (1 + exp(-r[i][e]))
 *
 * Every sum runs in index order in fp64.  One thread owns one (s, h) pair
 * from start to end, so results do not depend on the thread count.
 *
 * Layouts (element strides in units of elements, d fastest):
 *   dense  (offsets == NULL): x[s][h][i][e], s < nseq, i < rows  ([B,H,n,d])
 *   packed (offsets != NULL): x[h][offsets[s] + i][e], rows = T   ([H,T,d])
 *   a, g:       the same without the trailing d
 *   conv_w:     [3][H][d][W]  (q, k, v)
 *   gamma:      [H][d]
 *   S:          [nseq][H][d][d],   z: [nseq][H][d]
 * Activation inputs (q, k, v, a, r) are fp32, bf16 bit patterns or fp64
 * (dtype code 0, 1, 2); bf16 values are widened exactly.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORACLE_F32 = 0, ORACLE_BF16 = 1, ORACLE_F64 = 2 };

/* Exact widening of one stored activation element to fp64. */
static double load_act(const void* base, int dtype, size_t idx) {
  if (dtype == ORACLE_F64) return ((const double*)base)[idx];
  if (dtype == ORACLE_F32) return (double)((const float*)base)[idx];
  uint32_t bits = (uint32_t)((const uint16_t*)base)[idx] << 16;
  float f;
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

/* phi(u) = elu(u) + 1 (Section 2, BLA paragraph). */
double gbla_oracle_phi(double u) { return u > 0.0 ? u + 1.0 : exp(u); }

/* SiLU(x) = x * sigmoid(x) (Section 2.1, gated RMSNorm item). */
static double silu(double x) { return x / (1.0 + exp(-x)); }

typedef struct {
  int32_t nseq, heads, rows, d, W, dtype;
  const int32_t* offsets;
  double eps;
} problem;

/* Row index (token-major, in units of d elements) of token i of (s, h). */
static size_t row_of(const problem* P, int s, int h, int64_t i) {
  if (P->offsets == NULL)
    return ((size_t)s * (size_t)P->heads + (size_t)h) * (size_t)P->rows + (size_t)i;
  return (size_t)h * (size_t)P->rows + (size_t)P->offsets[s] + (size_t)i;
}

static int64_t length_of(const problem* P, int s) {
  if (P->offsets == NULL) return P->rows;
  return (int64_t)P->offsets[s + 1] - (int64_t)P->offsets[s];
}

/* Step 1: causal depthwise conv of one (s, h) slice of x into out[L][d]. */
static void conv_slice(const problem* P, const void* x, const double* w_h /* [d][W] */,
                       int s, int h, int64_t L, double* out) {
  const int d = P->d, W = P->W;
  for (int64_t i = 0; i < L; ++i) {
    for (int e = 0; e < d; ++e) {
      double acc = 0.0;
      for (int t = 0; t < W; ++t) {
        int64_t src = i - (W - 1) + t;
        if (src < 0) continue;
        acc += w_h[(size_t)e * W + t] * load_act(x, P->dtype, row_of(P, s, h, src) * d + e);
      }
      out[(size_t)i * d + e] = acc;
    }
  }
}

static void one_slice(const problem* P, int s, int h,
                      const void* q, const void* k, const void* v, const void* a, const void* r,
                      const double* conv_w, const double* gamma,
                      double* y, double* qt_out, double* kt_out, double* vt_out, double* g_out,
                      double* S_out, double* z_out, double* o_out, double* oh_out) {
  const int d = P->d, W = P->W, H = P->heads;
  const int64_t L = length_of(P, s);
  double* S = (double*)calloc((size_t)d * d, sizeof(double));
  double* z = (double*)calloc((size_t)d, sizeof(double));
  double* o = (double*)malloc((size_t)d * sizeof(double));
  if (L <= 0) {  /* empty sequence: nothing to produce; state stays zero */
    if (S_out) memcpy(S_out + ((size_t)s * H + h) * d * d, S, (size_t)d * d * sizeof(double));
    if (z_out) memcpy(z_out + ((size_t)s * H + h) * d, z, (size_t)d * sizeof(double));
    free(S); free(z); free(o);
    return;
  }
  double* qt = (double*)malloc((size_t)L * d * sizeof(double));
  double* kt = (double*)malloc((size_t)L * d * sizeof(double));
  double* vt = (double*)malloc((size_t)L * d * sizeof(double));
  double* g = (double*)malloc((size_t)L * sizeof(double));

  /* 1. Conv1D on q, k, v. */
  conv_slice(P, q, conv_w + ((size_t)0 * H + h) * d * W, s, h, L, qt);
  conv_slice(P, k, conv_w + ((size_t)1 * H + h) * d * W, s, h, L, kt);
  conv_slice(P, v, conv_w + ((size_t)2 * H + h) * d * W, s, h, L, vt);

  /* 3. Sequence softmax of the gate logits. */
  double amax = -INFINITY;
  for (int64_t j = 0; j < L; ++j) {
    double aj = load_act(a, P->dtype, row_of(P, s, h, j));
    if (aj > amax) amax = aj;
  }
  double denom = 0.0;
  for (int64_t j = 0; j < L; ++j) {
    g[j] = exp(load_act(a, P->dtype, row_of(P, s, h, j)) - amax);
    denom += g[j];
  }
  for (int64_t j = 0; j < L; ++j) g[j] /= denom;

  /* 2 + 4. Gated keys g[j] * phi(kt[j]) and the global state S, z. */
  for (int64_t j = 0; j < L; ++j) {
    for (int c = 0; c < d; ++c) {
      double kh = g[j] * gbla_oracle_phi(kt[(size_t)j * d + c]);
      z[c] += kh;
      for (int e = 0; e < d; ++e) S[(size_t)c * d + e] += kh * vt[(size_t)j * d + e];
    }
  }

  /* 2 + 5 + 6. Readout and gated RMSNorm, token by token. */
  const double* gam = gamma + (size_t)h * d;
  for (int64_t i = 0; i < L; ++i) {
    double den = 0.0;
    for (int e = 0; e < d; ++e) o[e] = 0.0;
    for (int c = 0; c < d; ++c) {
      double qh = gbla_oracle_phi(qt[(size_t)i * d + c]);
      den += qh * z[c];
      for (int e = 0; e < d; ++e) o[e] += qh * S[(size_t)c * d + e];
    }
    for (int e = 0; e < d; ++e) o[e] /= den;
    double ms = 0.0;
    for (int e = 0; e < d; ++e) ms += o[e] * o[e];
    ms /= (double)d;
    const double inv = 1.0 / sqrt(ms + P->eps);
    const size_t row = row_of(P, s, h, i) * d;
    for (int e = 0; e < d; ++e) {
      double oh = o[e] * inv;
      double rv = load_act(r, P->dtype, row + e);
      if (y) y[row + e] = oh * gam[e] * silu(rv);
      if (o_out) o_out[row + e] = o[e];
      if (oh_out) oh_out[row + e] = oh;
    }
  }

  for (int64_t i = 0; i < L; ++i) {
    const size_t row = row_of(P, s, h, i);
    if (g_out) g_out[row] = g[i];
    for (int e = 0; e < d; ++e) {
      if (qt_out) qt_out[row * d + e] = qt[(size_t)i * d + e];
      if (kt_out) kt_out[row * d + e] = kt[(size_t)i * d + e];
      if (vt_out) vt_out[row * d + e] = vt[(size_t)i * d + e];
    }
  }
  if (S_out) memcpy(S_out + ((size_t)s * H + h) * d * d, S, (size_t)d * d * sizeof(double));
  if (z_out) memcpy(z_out + ((size_t)s * H + h) * d, z, (size_t)d * sizeof(double));
  free(qt); free(kt); free(vt); free(g); free(S); free(z); free(o);
}

/*
 * Full forward pass.  Returns 0 on success, a negative number for invalid
 * arguments.  Every output pointer may be NULL (not produced).  nthreads <= 0
 * uses the OpenMP default.
 */
int gbla_oracle_forward(int32_t nseq, int32_t heads, int32_t rows, int32_t d, int32_t W,
                        int32_t dtype, const int32_t* offsets, double eps,
                        const void* q, const void* k, const void* v, const void* a, const void* r,
                        const double* conv_w, const double* gamma,
                        double* y, double* qt, double* kt, double* vt, double* g,
                        double* S, double* z, double* o, double* oh, int32_t nthreads) {
  if (nseq < 0 || heads <= 0 || rows < 0 || d <= 0 || W <= 0) return -1;
  if (dtype != ORACLE_F32 && dtype != ORACLE_BF16 && dtype != ORACLE_F64) return -2;
  if (!q || !k || !v || !a || !r || !conv_w || !gamma) return -3;
  if (offsets) {
    if (offsets[0] != 0 || offsets[nseq] != rows) return -4;
    for (int s = 0; s < nseq; ++s)
      if (offsets[s + 1] < offsets[s]) return -4;
  }
  problem P = {nseq, heads, rows, d, W, dtype, offsets, eps};
  const int64_t units = (int64_t)nseq * heads;
#ifdef _OPENMP
  int nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nt)
#endif
  for (int64_t u = 0; u < units; ++u) {
    int s = (int)(u / heads), h = (int)(u % heads);
    one_slice(&P, s, h, q, k, v, a, r, conv_w, gamma, y, qt, kt, vt, g, S, z, o, oh);
  }
  (void)nthreads;
  return 0;
}

/* Number of threads the OpenMP runtime would use by default. */
int32_t gbla_oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
