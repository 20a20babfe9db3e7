// launch.hpp -- host-side interface between the C ABI (api.cpp) and the
// kernel translation units.  Internal to the library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lora {

enum Dtype { DT_BF16 = 0, DT_F32 = 1 };

// C[M, N] = sum_k Aop[m][k] Bop[n][k]  (+ LoRA tail), rounded to the element type.
//   Aop[m][k] = A[m*lda + k]                         m < M, k < K
//   Bop[n][k] = B[n*ldb + k]   (b_kmajor = false)    n < N
//             = B[k*ldb + n]   (b_kmajor = true)
// Tail (r > 0), an extra reduction over j < r appended to k:
//   Aop2[m][j] = s2 * A2[m*r + j]  (fp32 in memory, rounded to the element type)
//   Bop2[n][j] = B2[n*r + j]       (b_kmajor = false)
//              = B2[j*ldb2 + n]    (b_kmajor = true)
struct GemmArgs {
  const void *A;
  int64_t lda;
  const void *B;
  int64_t ldb;
  int M, N, K;
  const float *A2;
  float s2;
  const void *B2;
  int64_t ldb2;
  int r;
  void *C;
  int64_t ldc;
};

hipError_t launch_gemm(const GemmArgs &g, Dtype dt, bool b_kmajor, hipStream_t st);

// out[m][j] = scale * sum_k X[m*ldx + k] * V(j, k),  m < M, j < r, k < L,
//   V(j, k) = V[j*ldv + k] (v_kmajor = false) or V[k*ldv + j] (v_kmajor = true).
hipError_t launch_row_skinny(const void *X, int64_t ldx, int M, int L, const void *V,
                             int64_t ldv, bool v_kmajor, int r, float scale, float *out,
                             Dtype dt, hipStream_t st);

// Partial sums over token chunks:
//   part[c][l][j] = sum_{t in chunk c} X[t*ldx + l] * V[t*r + j],  l < L, j < r
// with chunk c = [c*rows_per_chunk, min(T, (c+1)*rows_per_chunk)).
hipError_t launch_col_skinny(const void *X, int64_t ldx, int T, int L, const float *V, int r,
                             int nchunks, int rows_per_chunk, float *part, Dtype dt,
                             hipStream_t st);

// out = scale * sum_c part[c]  (fixed order c = 0, 1, ...), part [nchunks][L][r];
// out layout [L][r], or [r][L] when transpose_out.
hipError_t launch_reduce_parts(const float *part, int nchunks, int L, int r, float scale,
                               float *out, bool transpose_out, hipStream_t st);

// Token chunking of the column-skinny partial sums (a pure function of the
// shapes, shared by the workspace query and the launches).
void col_chunking(int T, int L, int r, Dtype dt, int *nchunks, int *rows_per_chunk);

}  // namespace lora
