// launch.hpp -- host-side interface between the C ABI (api.cpp) and the
// kernel translation units.  Internal to the library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lora {

enum Dtype { DT_BF16 = 0, DT_F32 = 1 };

// Side work run by extra workgroups of the backward GEMM launch (they
// overlap with the dx tiles): token-reduced products
//   dA = du^T x   out [r, L] (transposed store), scale 1
//   dB = s dy^T u out [L, r],                    scale s
// out[l][j] = scale * sum_t X[t*ldx + l] * V[t*r + j], t < T.
struct ColJob {
  const void *X;
  int64_t ldx;
  int L;
  const float *V;
  float *out;
  int transpose_out;
  float scale;
};
struct SideArgs {
  ColJob job[2];
  int njobs;
  int T, r;
};

// C[M, N] = sum_k Aop[m][k] Bop[n][k]  (+ LoRA step), rounded to the element type.
//   Aop[m][k] = A[m*lda + k]                         m < M, k < K
//   Bop[n][k] = B[n*ldb + k]   (b_kmajor = false)    n < N
//             = B[k*ldb + n]   (b_kmajor = true)
// LoRA step (r > 0), extra reduction over j < r appended to k, both operands
// already in the element type:
//   Aop2[m][j] = A2[m*lda2 + j]
//   Bop2[n][j] = B2[n*ldb2 + j] (b_kmajor = false)  or  B2[j*ldb2 + n] (true)
struct GemmArgs {
  const void *A;
  int64_t lda;
  const void *B;
  int64_t ldb;
  int M, N, K;
  const void *A2;
  int64_t lda2;
  const void *B2;
  int64_t ldb2;
  int r;
  void *C;
  int64_t ldc;
};

// GEMM launch; `side` (may be NULL) adds the token-reduction workgroups.
hipError_t launch_gemm(const GemmArgs &g, Dtype dt, bool b_kmajor, const SideArgs *side,
                       hipStream_t st);

// Number of side workgroups needed for `side` (a multiple of 8).
int side_workgroups(const SideArgs &s, Dtype dt);

enum { V_ROW = 0, V_KMAJ_TR = 1, V_KMAJ_GATHER = 2 };
// Row-skinny product out[m][j] = out_mult * sum_k X[m*ldx + k] * V(j, k),
// V(j, k) = V[j*ldv + k] (V_ROW) or V[k*ldv + j] (k-major, ldv = r).
// Optional: tail[m][j] = E(tail_mult * sum) for j < r, 0 up to ldt;
// bcopy_dst[n][j] = bcopy_src[n*r + j] zero-padded to ldt, n < bcopy_rows.
struct RowArgs {
  const void *X;
  int64_t ldx;
  int M, L;
  const void *V;
  int64_t ldv;
  int vmode;
  int r;
  float out_mult;
  float *out;
  void *tail;
  int ldt;
  float tail_mult;
  const void *bcopy_src;
  void *bcopy_dst;
  int bcopy_rows;
};
hipError_t launch_row_skinny(const RowArgs &a, Dtype dt, hipStream_t st);

// Padded row length of the LoRA-step operands (a multiple of the GEMM stage).
inline int tail_ld(int r, Dtype dt) {
  const int s = dt == DT_BF16 ? 64 : 32;
  return (r + s - 1) / s * s;
}

}  // namespace lora
