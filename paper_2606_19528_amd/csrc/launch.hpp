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
// V may be given as `vparts` partial sums V_p = V + p * vstride (p < vparts),
// added in ascending p when loaded.
struct ColJob {
  const void *X;
  int64_t ldx;
  int L;
  const float *V;
  float *out;
  int transpose_out;
  float scale;
  int vparts;
  int64_t vstride;
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
// Optional (usum_out != NULL): the workgroups also write
// usum_out[m][j] = sum_{p < usum_parts} usum_src[p][m][j] (ascending p) for
// m < M, j < usum_r -- the sum of a rank-r product computed in partial sums
// (usum_parts <= MAX_SPLIT; row-major B only).
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
  const float *usum_src;
  float *usum_out;
  int usum_parts, usum_r;
  // Quantized B (launch_gemm_q): B holds unsigned codes of W ([rows][ldb]
  // weights, bits/8 bytes each, two 4-bit codes per byte with the even weight
  // in the low nibble), w = qscale * code + qoffset with one scale and offset
  // per group of 2^qlog2g consecutive weights of a W row ([rows][ldb >> qlog2g]).
  const float *qscale;
  const float *qoffset;
  int qlog2g;
};

// GEMM launch; `side` (may be NULL) adds the token-reduction workgroups.
hipError_t launch_gemm(const GemmArgs &g, Dtype dt, bool b_kmajor, const SideArgs *side,
                       hipStream_t st);
// bf16 GEMM whose B is the quantized frozen weight (bits = 4 or 8), dequantized
// into LDS; the LoRA step (r <= 64) runs first.
hipError_t launch_gemm_q(const GemmArgs &g, int bits, bool b_kmajor, const SideArgs *side,
                         hipStream_t st);

// Number of side workgroups needed for `side` (a multiple of 8).
int side_workgroups(const SideArgs &s, Dtype dt);

enum { V_ROW = 0, V_KMAJ_TR = 1, V_KMAJ_GATHER = 2 };
enum { BCOPY_NONE = 0, BCOPY_COLS = 1, BCOPY_FLAT = 2 };
// Row-skinny product, split over the reduction axis into `nsplit` segments of
// `seg` elements (seg a multiple of one 128-byte chunk of elements):
//   P_p[m][j] = sum_{k in segment p} X[m*ldx + k] * V(j, k),
//   V(j, k) = V[j*ldv + k] (V_ROW) or V[k*ldv + j] (k-major, ldv = r).
// Writes out[p * out_stride + m*r + j] = out_mult * P_p[m][j] and, if tail is
// set, tail[m][p*r + j] = E(tail_mult * P_p[m][j]), columns nsplit*r .. ldt-1
// zero.  Optional copy job:
//   BCOPY_COLS  dst[n][c] = src[n*r + c % r] for c < nsplit*r, 0 up to ldt,
//               n < bcopy_rows (B repeated once per segment, zero-padded);
//   BCOPY_FLAT  dst[i] = src[i % bcopy_period] for i < bcopy_elems.
struct RowArgs {
  const void *X;
  int64_t ldx;
  int M, L;
  const void *V;
  int64_t ldv;
  int vmode;
  int r;
  int nsplit, seg;
  float out_mult;
  float *out;
  int64_t out_stride;
  void *tail;
  int ldt;
  float tail_mult;
  int bcopy_mode;
  const void *bcopy_src;
  void *bcopy_dst;
  int bcopy_rows;
  int64_t bcopy_period, bcopy_elems;
};
hipError_t launch_row_skinny(const RowArgs &a, Dtype dt, hipStream_t st);

// Split of a row-skinny product over its reduction axis L: enough segments to
// give the T / 16 row blocks about one workgroup per CU, no more than fit in
// the padded LoRA step (nsplit * r <= ldt), each segment at least one
// 128-byte chunk per wave, and at most MAX_SPLIT segments.
constexpr int MAX_SPLIT = 8;
struct RowSplit {
  int nsplit, seg;
};
RowSplit row_split(int64_t T, int64_t L, int r, Dtype dt);

// Padded row length of the LoRA-step operands (a multiple of the GEMM stage).
inline int tail_ld(int r, Dtype dt) {
  const int s = dt == DT_BF16 ? 64 : 32;
  return (r + s - 1) / s * s;
}

}  // namespace lora
