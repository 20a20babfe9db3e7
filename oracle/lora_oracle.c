/*
 * lora_oracle.c -- fp64 CPU oracle for the LoRA-adapted linear layer.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library
 * and its Python binding) may include, link or call this file; only the
 * tests, the smoke check and the benchmark's CPU-baseline leg use it.  It
 * shares no code, header, table or helper with the GPU implementation.
 *
 * What it computes (paper: "Background -- Parameter-Efficient Fine-Tuning"
 * describes LoRA as a frozen base weight plus a trained pair of rank-r
 * factors; the hyperparameter table fixes r and alpha; the algorithm
 * "On-the-fly Dequantization" fixes the frozen base forward y = W x and
 * backward dx = W^T dy, with no weight gradient):
 *
 *     U  = X A^T                       [T,r]      (saved LoRA activation)
 *     Y  = X W^T + s U B^T             [T,N]      s = alpha / r
 *     G  = dY B                        [T,r]
 *     dU = s G                         [T,r]
 *     dX = dY W + dU A                 [T,K]
 *     dA = dU^T X                      [r,K]
 *     dB = s dY^T U                    [N,r]
 *
 * Shapes: X [T,K], W [N,K], A [r,K], B [N,r], dY [T,N]; K = d_in, N = d_out.
 * The paper writes the base linear with column vectors (y = W x); here tokens
 * are rows, so y = x W^T and dx = dy W.  dW is never formed.
 *
 * Every value is fp64; the inputs are exact upcasts of the bf16 (or fp32)
 * values the GPU consumes.  Every sum runs over ascending index with plain
 * accumulation (no Kahan, no blocking, no BLAS).  OpenMP only splits
 * independent output rows or columns across threads; it never changes the
 * order of any single sum.
 *
 * Each function is one line of the definition above, written out.
 *
 * For a quantized frozen base the weight W is first reconstructed in fp64 by
 * oracle_dequant (below) and then used exactly as above.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>

/* U[t][j] = sum_k X[t][k] * A[j][k]  (LoRA down-projection, saved for the
 * backward pass). */
void oracle_lora_u(const double *X, const double *A, int64_t T, int64_t K,
                   int64_t r, double *U) {
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < T; ++t) {
    for (int64_t j = 0; j < r; ++j) {
      double acc = 0.0;
      for (int64_t k = 0; k < K; ++k) acc += X[t * K + k] * A[j * K + k];
      U[t * r + j] = acc;
    }
  }
}

/* Y[t][n] = sum_k X[t][k] * W[n][k] + s * sum_j U[t][j] * B[n][j]
 * (frozen base contraction plus the scaled LoRA up-projection).
 * rows == NULL computes every row t = 0..T-1 into Y[t]; otherwise row
 * rows[i] is computed into Y[i] (i = 0..nrows-1). */
void oracle_lora_y_rows(const double *X, const double *W, const double *U,
                        const double *B, int64_t T, int64_t K, int64_t N,
                        int64_t r, double s, const int64_t *rows,
                        int64_t nrows, double *Y) {
  int64_t count = rows ? nrows : T;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < count; ++i) {
    int64_t t = rows ? rows[i] : i;
    for (int64_t n = 0; n < N; ++n) {
      double base = 0.0;
      for (int64_t k = 0; k < K; ++k) base += X[t * K + k] * W[n * K + k];
      double lora = 0.0;
      for (int64_t j = 0; j < r; ++j) lora += U[t * r + j] * B[n * r + j];
      Y[i * N + n] = base + s * lora;
    }
  }
}

/* G[t][j] = sum_n dY[t][n] * B[n][j];  dU[t][j] = s * G[t][j]
 * (gradient reaching the LoRA activation U). */
void oracle_lora_grad_u(const double *dY, const double *B, int64_t T,
                        int64_t N, int64_t r, double s, double *G,
                        double *dU) {
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < T; ++t) {
    for (int64_t j = 0; j < r; ++j) {
      double acc = 0.0;
      for (int64_t n = 0; n < N; ++n) acc += dY[t * N + n] * B[n * r + j];
      G[t * r + j] = acc;
      dU[t * r + j] = s * acc;
    }
  }
}

/* dX[t][k] = sum_n dY[t][n] * W[n][k] + sum_j dU[t][j] * A[j][k]
 * (input gradient through the frozen W and through the LoRA branch).
 * Row selection as in oracle_lora_y_rows.  The sum over n is accumulated in
 * ascending n for every k (a row of dX is built up one n at a time, which
 * keeps each element's summation order ascending). */
void oracle_lora_dx_rows(const double *dY, const double *W, const double *dU,
                         const double *A, int64_t T, int64_t K, int64_t N,
                         int64_t r, const int64_t *rows, int64_t nrows,
                         double *dX) {
  int64_t count = rows ? nrows : T;
  (void)T;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < count; ++i) {
    int64_t t = rows ? rows[i] : i;
    double *out = dX + i * K;
    for (int64_t k = 0; k < K; ++k) out[k] = 0.0;
    for (int64_t n = 0; n < N; ++n) {
      double g = dY[t * N + n];
      const double *wrow = W + n * K;
      for (int64_t k = 0; k < K; ++k) out[k] += g * wrow[k];
    }
    /* The LoRA term is its own sum, added once to the base sum. */
    for (int64_t k = 0; k < K; ++k) {
      double lora = 0.0;
      for (int64_t j = 0; j < r; ++j) lora += dU[t * r + j] * A[j * K + k];
      out[k] += lora;
    }
  }
}

/* dA[j][k] = sum_t dU[t][j] * X[t][k]  (gradient of the down factor A). */
void oracle_lora_da(const double *dU, const double *X, int64_t T, int64_t K,
                    int64_t r, double *dA) {
#pragma omp parallel for schedule(static)
  for (int64_t k = 0; k < K; ++k) {
    for (int64_t j = 0; j < r; ++j) {
      double acc = 0.0;
      for (int64_t t = 0; t < T; ++t) acc += dU[t * r + j] * X[t * K + k];
      dA[j * K + k] = acc;
    }
  }
}

/* dB[n][j] = s * sum_t dY[t][n] * U[t][j]  (gradient of the up factor B). */
void oracle_lora_db(const double *dY, const double *U, int64_t T, int64_t N,
                    int64_t r, double s, double *dB) {
#pragma omp parallel for schedule(static)
  for (int64_t n = 0; n < N; ++n) {
    for (int64_t j = 0; j < r; ++j) {
      double acc = 0.0;
      for (int64_t t = 0; t < T; ++t) acc += dY[t * N + n] * U[t * r + j];
      dB[n * r + j] = s * acc;
    }
  }
}

/* W[n][k] = S[n][g] * q(n, k) + Bo[n][g],  g = k / G
 * (the dequantization step of the algorithm "On-the-fly Dequantization",
 * W = s * W_q + b, with one scale s and offset b per group of G consecutive
 * inputs of an output row).  The codes q are unsigned integers read from Wq
 * [N, K * bits / 8] bytes: bits = 8 stores one code per byte; bits = 4 two per
 * byte, the code of even k in the low nibble and of odd k in the high one.
 * S and Bo are [N, K / G]. */
void oracle_dequant(const uint8_t *Wq, const double *S, const double *Bo,
                    int64_t N, int64_t K, int bits, int64_t G, double *W) {
  const int64_t row_bytes = K * bits / 8;
  const int64_t ngroups = K / G;
#pragma omp parallel for schedule(static)
  for (int64_t n = 0; n < N; ++n) {
    for (int64_t k = 0; k < K; ++k) {
      int q;
      if (bits == 8) {
        q = Wq[n * row_bytes + k];
      } else {
        const uint8_t byte = Wq[n * row_bytes + k / 2];
        q = (k % 2 == 0) ? (byte & 0x0F) : (byte >> 4);
      }
      const int64_t g = k / G;
      W[n * K + k] = S[n * ngroups + g] * (double)q + Bo[n * ngroups + g];
    }
  }
}

/* Reduced-vocabulary cross entropy of the frozen LM head with logits masking
 * (paper: "Softmax Approximation" -- logits over the rows J of the embedding
 * matrix only; "Logits Masking" -- logits only for the trainable positions;
 * the masked causal-LM loss sums -log p_t over those positions).
 * For each listed position t = rows[i] (i < nrows):
 *   z[j]    = sum_d H[t][d] * W[J[j]][d]                 j < nJ
 *   lse     = m + log(sum_j exp(z[j] - m)),  m = max_j z[j]
 *   loss[i] = lse - z[tpos[i]]        (tpos[i]: position of the target in J)
 *   dH[t][d] = sum_j exp(z[j] - lse) * W[J[j]][d] - W[J[tpos[i]]][d]
 * (the gradient of sum_i loss[i]); rows of dH not listed are set to zero.
 * H [T, D], W [V, D] (only the rows in J are read), dH [T, D]. */
void oracle_ce_reduced(const double *H, const double *W, int64_t T, int64_t D,
                       const int64_t *rows, int64_t nrows, const int64_t *J,
                       int64_t nJ, const int64_t *tpos, double *loss, double *dH) {
  for (int64_t i = 0; i < T * D; ++i) dH[i] = 0.0;
#pragma omp parallel for schedule(dynamic)
  for (int64_t i = 0; i < nrows; ++i) {
    const int64_t t = rows[i];
    double *z = (double *)malloc(sizeof(double) * (size_t)nJ);
    double m = -INFINITY;
    for (int64_t j = 0; j < nJ; ++j) {
      double acc = 0.0;
      for (int64_t d = 0; d < D; ++d) acc += H[t * D + d] * W[J[j] * D + d];
      z[j] = acc;
      if (acc > m) m = acc;
    }
    double s = 0.0;
    for (int64_t j = 0; j < nJ; ++j) s += exp(z[j] - m);
    const double lse = m + log(s);
    loss[i] = lse - z[tpos[i]];
    double *out = dH + t * D;
    for (int64_t j = 0; j < nJ; ++j) {
      const double p = exp(z[j] - lse);
      const double *w = W + J[j] * D;
      for (int64_t d = 0; d < D; ++d) out[d] += p * w[d];
    }
    const double *wt = W + J[tpos[i]] * D;
    for (int64_t d = 0; d < D; ++d) out[d] -= wt[d];
    free(z);
  }
}

/* Order of two (similarity, token) pairs: higher similarity first, the
 * smaller token index first among equal similarities. */
typedef struct {
  double c;
  int64_t j;
} sim_pair;
static int sim_pair_cmp(const void *pa, const void *pb) {
  const sim_pair *a = (const sim_pair *)pa, *b = (const sim_pair *)pb;
  if (a->c > b->c) return -1;
  if (a->c < b->c) return 1;
  return (a->j > b->j) - (a->j < b->j);
}

/* Top-k similarity table (paper: "Softmax Approximation" -- the cosine
 * similarities C = W~^T W~ of the column-normalised embedding matrix, row i
 * sorted in descending order, the first k indices kept).  Here the
 * embeddings are the rows of W [V, D]:
 *   C[i][j] = (w_i . w_j) / (|w_i| |w_j|)
 *   A[i][0 .. k-1] = the indices j of row i sorted by C[i][j] descending
 *                    (the smaller j first among equal similarities),
 * and Cs[i][c] = C[i][A[i][c]].  A zero row has similarity 0 with all.
 * rows == NULL computes every row i into A[i]; otherwise row rows[r] goes to
 * A[r] (r < nrows). */
void oracle_topk_table(const double *W, int64_t V, int64_t D, int64_t k, const int64_t *rows,
                       int64_t nrows, int64_t *A, double *Cs) {
  double *norm = (double *)malloc(sizeof(double) * (size_t)V);
  for (int64_t v = 0; v < V; ++v) {
    double acc = 0.0;
    for (int64_t d = 0; d < D; ++d) acc += W[v * D + d] * W[v * D + d];
    norm[v] = sqrt(acc);
  }
  const int64_t count = rows ? nrows : V;
#pragma omp parallel for schedule(dynamic)
  for (int64_t r = 0; r < count; ++r) {
    const int64_t i = rows ? rows[r] : r;
    sim_pair *row = (sim_pair *)malloc(sizeof(sim_pair) * (size_t)V);
    for (int64_t j = 0; j < V; ++j) {
      double dot = 0.0;
      for (int64_t d = 0; d < D; ++d) dot += W[i * D + d] * W[j * D + d];
      const double den = norm[i] * norm[j];
      row[j].c = den > 0.0 ? dot / den : 0.0;
      row[j].j = j;
    }
    qsort(row, (size_t)V, sizeof(sim_pair), sim_pair_cmp);
    for (int64_t c = 0; c < k; ++c) {
      A[r * k + c] = row[c].j;
      Cs[r * k + c] = row[c].c;
    }
    free(row);
  }
  free(norm);
}

/* Number of OpenMP threads the oracle runs with (1 when built without
 * OpenMP); reported next to its timings. */
#ifdef _OPENMP
#include <omp.h>
int oracle_threads(void) { return omp_get_max_threads(); }
/* Thread count of the following parallel loops (timing only; the results do
 * not depend on it). */
void oracle_set_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }
#else
int oracle_threads(void) { return 1; }
void oracle_set_threads(int n) { (void)n; }
#endif
