// skinny.hip -- the rank-r products of the LoRA linear.  Each reads one big
// activation ([T, d]) once from HBM and produces a small [*, r] result, so they
// are bandwidth-bound; the arithmetic still runs on 16x16 matrix-core tiles
// because at r >= 16 vector FMAs could not keep up with HBM.
//   row-skinny  out[T, r] = X V^T      u = x A^T,  du = s dy B
//                (reduction over the long feature axis, one pass per 16 rows)
//   col-skinny  part[c][L, r] = X_c^T V_c      dB = s dy^T u,  dA = du^T x
//                (reduction over tokens, split into fixed token chunks)
//   reduce      sum of the per-chunk partials in a fixed order (deterministic).
#include "kernels.hpp"
#include "launch.hpp"

namespace lora {

// ---------------------------------------------------------------------------
// Row-skinny: a workgroup owns 16 rows; its four waves take interleaved
// 128-byte k-chunks of those rows and their partial 16 x r tiles are summed
// in LDS in a fixed order.
template <class E, bool VKMAJ, int JB>
__global__ __launch_bounds__(256) void row_skinny_kernel(const void *X, int64_t ldx, int M, int L,
                                                         const void *V, int64_t ldv, int r,
                                                         float scale, float *out) {
  typedef typename E::T T;
  constexpr int VEC = E::VEC;
  constexpr int CE = 128 / (int)sizeof(T);  // elements per 128-byte chunk
  __shared__ float red[4][16][JB * 16 + 1];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int m0 = blockIdx.x * 16;
  const int row = m0 + (lane & 15);
  const int g = lane >> 4;
  const T *Xp = (const T *)X;
  const T *Vp = (const T *)V;

  f32x4 acc[JB];
#pragma unroll
  for (int jb = 0; jb < JB; ++jb) acc[jb] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int kc = wave * CE; kc < L; kc += 4 * CE) {
    u32x4 xf[2];
    u32x4 vf[2][JB];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int k = kc + h * 4 * VEC + g * VEC;
      xf[h] = (row < M && k < L) ? ld16(Xp + (int64_t)row * ldx + k) : zero16();
#pragma unroll
      for (int jb = 0; jb < JB; ++jb) {
        const int j = jb * 16 + (lane & 15);
        if constexpr (!VKMAJ) {
          vf[h][jb] = (j < r && k < L) ? ld16(Vp + (int64_t)j * ldv + k) : zero16();
        } else {
          float f[VEC];
#pragma unroll
          for (int e = 0; e < VEC; ++e)
            f[e] = (j < r && k + e < L) ? E::to_float(Vp[(int64_t)(k + e) * ldv + j]) : 0.0f;
          vf[h][jb] = pack_vec(E(), f);
        }
      }
    }
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int jb = 0; jb < JB; ++jb) mma16(E(), acc[jb], xf[h], vf[h][jb]);
  }

  // D[m][n]: m = 4 (lane / 16) + i, n = lane % 16.
#pragma unroll
  for (int jb = 0; jb < JB; ++jb)
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave][g * 4 + i][jb * 16 + (lane & 15)] = acc[jb][i];
  __syncthreads();
  for (int idx = tid; idx < 16 * r; idx += 256) {
    const int mm = idx / r, j = idx % r;
    const float s = ((red[0][mm][j] + red[1][mm][j]) + red[2][mm][j]) + red[3][mm][j];
    if (m0 + mm < M) out[(int64_t)(m0 + mm) * r + j] = scale * s;
  }
}

template <class E, bool VKMAJ>
static hipError_t row_skinny_dispatch(const void *X, int64_t ldx, int M, int L, const void *V,
                                      int64_t ldv, int r, float scale, float *out,
                                      hipStream_t st) {
  dim3 grid((M + 15) / 16), block(256);
  const int jb = (r + 15) / 16;
#define ROWSK(J)                                                                              \
  case J:                                                                                     \
    hipLaunchKernelGGL((row_skinny_kernel<E, VKMAJ, J>), grid, block, 0, st, X, ldx, M, L, V, \
                       ldv, r, scale, out);                                                   \
    break;
  switch (jb) {
    ROWSK(1) ROWSK(2) ROWSK(3) ROWSK(4) ROWSK(5) ROWSK(6) ROWSK(7) ROWSK(8)
    default:
      return hipErrorInvalidValue;
  }
#undef ROWSK
  return hipGetLastError();
}

hipError_t launch_row_skinny(const void *X, int64_t ldx, int M, int L, const void *V,
                             int64_t ldv, bool v_kmajor, int r, float scale, float *out,
                             Dtype dt, hipStream_t st) {
  if (dt == DT_BF16)
    return v_kmajor ? row_skinny_dispatch<BF16, true>(X, ldx, M, L, V, ldv, r, scale, out, st)
                    : row_skinny_dispatch<BF16, false>(X, ldx, M, L, V, ldv, r, scale, out, st);
  return v_kmajor ? row_skinny_dispatch<F32, true>(X, ldx, M, L, V, ldv, r, scale, out, st)
                  : row_skinny_dispatch<F32, false>(X, ldx, M, L, V, ldv, r, scale, out, st);
}

// ---------------------------------------------------------------------------
// Col-skinny: a workgroup owns COLS = 16*VEC columns of X, one token chunk
// and one group of up to 32 rank indices.  Each wave reads VEC-row x
// 16-byte blocks (row-major, coalesced), transposes them in registers so that
// a lane holds VEC consecutive tokens of one column -- the matrix-core operand
// with the token axis as the reduction -- and accumulates a COLS x 32 tile.
// The four waves take interleaved row groups; their tiles are summed in LDS
// in a fixed order.
template <class E, int JB>
__global__ __launch_bounds__(256) void col_skinny_kernel(const void *X, int64_t ldx, int T_,
                                                         int L, const float *V, int r,
                                                         int rows_per_chunk, float *part) {
  typedef typename E::T T;
  constexpr int VEC = E::VEC;
  constexpr int COLS = 16 * VEC;  // columns per workgroup
  constexpr int ROWS = 4 * VEC;   // tokens per wave step
  __shared__ float red[4][COLS][JB * 16 + 1];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, cl = lane & 15;
  const int c0 = blockIdx.x * COLS;
  const int chunk = blockIdx.y;
  const int jg = blockIdx.z * (JB * 16);
  const int t_beg = chunk * rows_per_chunk;
  const int t_end = min(T_, t_beg + rows_per_chunk);
  const int col = c0 + cl * VEC;
  const T *Xp = (const T *)X;

  f32x4 acc[VEC][JB];
#pragma unroll
  for (int c = 0; c < VEC; ++c)
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) acc[c][jb] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int tb = t_beg + wave * ROWS; tb < t_end; tb += 4 * ROWS) {
    u32x4 xin[VEC], xt[VEC];
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
      const int t = tb + g * VEC + i;
      xin[i] = (t < t_end && col < L) ? ld16(Xp + (int64_t)t * ldx + col) : zero16();
    }
    transpose_block(E(), xin, xt);
    u32x4 vf[JB];
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) {
      const int j = jg + jb * 16 + cl;
      float f[VEC];
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const int t = tb + g * VEC + e;
        f[e] = (t < t_end && j < r) ? V[(int64_t)t * r + j] : 0.0f;
      }
      vf[jb] = pack_vec(E(), f);
    }
#pragma unroll
    for (int c = 0; c < VEC; ++c)
#pragma unroll
      for (int jb = 0; jb < JB; ++jb) mma16(E(), acc[c][jb], xt[c], vf[jb]);
  }

  // acc[c][jb] element i: column c0 + (4g + i) * VEC + c, rank index jg + 16 jb + cl.
#pragma unroll
  for (int c = 0; c < VEC; ++c)
#pragma unroll
    for (int jb = 0; jb < JB; ++jb)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[wave][(4 * g + i) * VEC + c][jb * 16 + cl] = acc[c][jb][i];
  __syncthreads();
  const int jn = min(JB * 16, r - jg);
  for (int idx = tid; idx < COLS * jn; idx += 256) {
    const int cc = idx / jn, j = idx % jn;
    const int l = c0 + cc;
    if (l < L) {
      const float s = ((red[0][cc][j] + red[1][cc][j]) + red[2][cc][j]) + red[3][cc][j];
      part[((int64_t)chunk * L + l) * r + jg + j] = s;
    }
  }
}

void col_chunking(int T, int L, int r, Dtype dt, int *nchunks, int *rows_per_chunk) {
  const int cols = dt == DT_BF16 ? 128 : 64;
  const int step = dt == DT_BF16 ? 128 : 64;  // 4 waves x ROWS tokens
  const int col_blocks = (L + cols - 1) / cols;
  const int jgroups = (r + 31) / 32;
  const int max_chunks = (T + step - 1) / step;
  int want = (512 + col_blocks * jgroups - 1) / (col_blocks * jgroups);
  if (want > 8) want = 8;
  if (want < 1) want = 1;
  int nch = want < max_chunks ? want : max_chunks;
  int rpc = (T + nch - 1) / nch;
  rpc = (rpc + step - 1) / step * step;
  nch = (T + rpc - 1) / rpc;
  *nchunks = nch;
  *rows_per_chunk = rpc;
}

hipError_t launch_col_skinny(const void *X, int64_t ldx, int T, int L, const float *V, int r,
                             int nchunks, int rows_per_chunk, float *part, Dtype dt,
                             hipStream_t st) {
  const int jgroups = (r + 31) / 32;
  const int jb = r >= 32 ? 2 : (r + 15) / 16;
  if (dt == DT_BF16) {
    dim3 grid((L + 127) / 128, nchunks, jgroups);
    if (jb == 1)
      hipLaunchKernelGGL((col_skinny_kernel<BF16, 1>), grid, dim3(256), 0, st, X, ldx, T, L, V, r,
                         rows_per_chunk, part);
    else
      hipLaunchKernelGGL((col_skinny_kernel<BF16, 2>), grid, dim3(256), 0, st, X, ldx, T, L, V, r,
                         rows_per_chunk, part);
  } else {
    dim3 grid((L + 63) / 64, nchunks, jgroups);
    if (jb == 1)
      hipLaunchKernelGGL((col_skinny_kernel<F32, 1>), grid, dim3(256), 0, st, X, ldx, T, L, V, r,
                         rows_per_chunk, part);
    else
      hipLaunchKernelGGL((col_skinny_kernel<F32, 2>), grid, dim3(256), 0, st, X, ldx, T, L, V, r,
                         rows_per_chunk, part);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void reduce_parts_kernel(const float *part, int nchunks, int L,
                                                           int r, float scale, float *out,
                                                           int transpose_out) {
  const int64_t n = (int64_t)L * r;
  for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < n;
       idx += (int64_t)gridDim.x * 256) {
    float s = 0.0f;
    for (int c = 0; c < nchunks; ++c) s += part[(int64_t)c * n + idx];
    s *= scale;
    if (transpose_out) {
      const int64_t l = idx / r, j = idx % r;
      out[j * L + l] = s;
    } else {
      out[idx] = s;
    }
  }
}

hipError_t launch_reduce_parts(const float *part, int nchunks, int L, int r, float scale,
                               float *out, bool transpose_out, hipStream_t st) {
  const int64_t n = (int64_t)L * r;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(reduce_parts_kernel, dim3((unsigned)blocks), dim3(256), 0, st, part, nchunks,
                     L, r, scale, out, transpose_out ? 1 : 0);
  return hipGetLastError();
}

}  // namespace lora
