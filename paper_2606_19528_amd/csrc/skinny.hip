// skinny.hip -- the rank-r "row" products of the LoRA linear: one read of a big
// activation [T, L] against a small [r, L] factor, reduced over the long axis L.
//   forward   u  = x A^T                    (A row-major [r, d_in])
//   backward  du = s dy B                   (B k-major   [d_out, r])
// Each workgroup owns 16 rows; its eight waves take interleaved 128-byte
// chunks of those rows (up to four chunks in flight per wave, enough loads
// outstanding to stream at HBM speed with only T/16 workgroups), accumulate
// 16 x r tiles on 16x16 matrix cores, and the eight partial tiles are summed
// in LDS in a fixed order.  At r >= 16 vector FMAs would not keep up with HBM.
//
// k-major B: each wave copies the B rows of its chunk into a private LDS
// region and reads them back with ds_read_b64_tr_b16, which returns four
// consecutive k of one column per lane -- exactly the matrix-core operand --
// instead of gathering 2-byte elements from global memory.
//
// Besides the fp32 result the kernel writes the operand of the big GEMM's
// LoRA step: tail = E(tail_mult * sum), zero-padded to `ldt` columns, and
// (forward) a zero-padded copy of B.
#include "kernels.hpp"
#include "launch.hpp"

namespace lora {

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int ROW_NW = 8;  // waves per workgroup

template <class E, int JB, int VMODE, int U>
__global__ __launch_bounds__(64 * ROW_NW) void row_skinny_kernel(RowArgs a) {
  constexpr int NW = ROW_NW, NT = 64 * NW;
  typedef typename E::T T;
  constexpr int VEC = E::VEC;
  constexpr int CE = 128 / (int)sizeof(T);  // elements per 128-byte chunk
  constexpr int R16 = JB * 16;
  constexpr int RSB = R16 * 2;              // LDS row of a staged B chunk (bf16)
  constexpr int REGION = U * CE * RSB;      // per-wave staging region
  constexpr int RED = NW * 16 * (R16 + 1) * 4;
  constexpr int LDS = (VMODE == V_KMAJ_TR && NW * REGION > RED) ? NW * REGION : RED;
  __shared__ __align__(16) char smem[LDS];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int m0 = blockIdx.x * 16;
  const int row = m0 + (lane & 15);
  const int g = lane >> 4;
  const int M = a.M, L = a.L, r = a.r;
  const T *Xp = (const T *)a.X;
  const T *Vp = (const T *)a.V;

  // Optional side job: copy B zero-padded (the forward LoRA-step operand).
  if (a.bcopy_src) {
    const T *src = (const T *)a.bcopy_src;
    T *dst = (T *)a.bcopy_dst;
    const int64_t total = (int64_t)a.bcopy_rows * a.ldt;
    for (int64_t i = (int64_t)blockIdx.x * NT + tid; i < total; i += (int64_t)gridDim.x * NT) {
      const int64_t n = i / a.ldt;
      const int j = (int)(i % a.ldt);
      dst[i] = j < r ? src[n * r + j] : (T)0;
    }
  }

  f32x4 acc[JB];
#pragma unroll
  for (int jb = 0; jb < JB; ++jb) acc[jb] = f32x4{0.f, 0.f, 0.f, 0.f};
  char *region = smem + wave * REGION;

  for (int kc0 = wave * CE; kc0 < L; kc0 += NW * CE * U) {
    u32x4 xf[U][2];
    u32x4 vf[U][2][JB];
    // issue every global load of the U chunks first
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kc = kc0 + u * NW * CE;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int k = kc + h * 4 * VEC + g * VEC;
        xf[u][h] = (row < M && k < L) ? ld16(Xp + (int64_t)row * a.ldx + k) : zero16();
        if constexpr (VMODE == V_ROW) {
#pragma unroll
          for (int jb = 0; jb < JB; ++jb) {
            const int j = jb * 16 + (lane & 15);
            vf[u][h][jb] = (j < r && k < L) ? ld16(Vp + (int64_t)j * a.ldv + k) : zero16();
          }
        } else if constexpr (VMODE == V_KMAJ_GATHER) {
#pragma unroll
          for (int jb = 0; jb < JB; ++jb) {
            const int j = jb * 16 + (lane & 15);
            float f[VEC];
#pragma unroll
            for (int e = 0; e < VEC; ++e)
              f[e] = (j < r && k + e < L) ? E::to_float(Vp[(int64_t)(k + e) * a.ldv + j]) : 0.0f;
            vf[u][h][jb] = pack_vec(E(), f);
          }
        }
      }
    }
    if constexpr (VMODE == V_KMAJ_TR) {
      // Stage B rows [kc, kc + 64) x r of each chunk into this wave's region
      // (r is a multiple of 8, so a row is whole 16-byte pieces).
      const int cpr = r / 8;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int kc = kc0 + u * NW * CE;
        for (int c = lane; c < CE * cpr; c += 64) {
          const int br = c / cpr, bc = c % cpr;
          const int n = kc + br;
          const u32x4 v = n < L ? ld16(Vp + (int64_t)n * r + bc * 8) : zero16();
          st16(region + (u * CE + br) * RSB + bc * 16, v);
        }
      }
      // Read back transposed: lane (group gq, index iq) gets 4 consecutive k of
      // column 4*(iq%4) + iq/4... of its 16-column block (see kernels.hpp).
      const int iq = lane & 15;
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int jb = 0; jb < JB; ++jb) {
            const char *p = region + (u * CE + h * 32 + 8 * g + (iq >> 2)) * RSB +
                            (jb * 16 + 4 * (iq & 3)) * 2;
            i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)p);
            i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(p + 4 * RSB));
            vf[u][h][jb] = u32x4{__builtin_bit_cast(uint2, lo).x, __builtin_bit_cast(uint2, lo).y,
                                 __builtin_bit_cast(uint2, hi).x, __builtin_bit_cast(uint2, hi).y};
          }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int jb = 0; jb < JB; ++jb) mma16(E(), acc[jb], xf[u][h], vf[u][h][jb]);
  }

  // D[m][n]: m = 4 (lane / 16) + i, n = lane % 16.  Sum the waves' tiles.
  __syncthreads();
  float *red = (float *)smem;
#pragma unroll
  for (int jb = 0; jb < JB; ++jb)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      red[(wave * 16 + g * 4 + i) * (R16 + 1) + jb * 16 + (lane & 15)] = acc[jb][i];
  __syncthreads();
  T *tail = (T *)a.tail;
  const int ncol = a.tail ? a.ldt : r;
  for (int idx = tid; idx < 16 * ncol; idx += NT) {
    const int mm = idx / ncol, j = idx % ncol;
    if (m0 + mm >= M) continue;
    float s = 0.0f;
    if (j < r) {
      s = red[(0 * 16 + mm) * (R16 + 1) + j];
#pragma unroll
      for (int w = 1; w < NW; ++w) s += red[(w * 16 + mm) * (R16 + 1) + j];
      a.out[(int64_t)(m0 + mm) * r + j] = a.out_mult * s;
    }
    if (tail) tail[(int64_t)(m0 + mm) * a.ldt + j] = E::from_float(a.tail_mult * s);
  }
}

template <class E, int VMODE>
static hipError_t row_dispatch(const RowArgs &a, hipStream_t st) {
  dim3 grid((a.M + 15) / 16), block(64 * ROW_NW);
  const int jb = (a.r + 15) / 16;
#define ROWSK(J)                                                                                  \
  case J:                                                                                         \
    hipLaunchKernelGGL((row_skinny_kernel<E, J, VMODE, (J <= 2 ? 4 : 1)>), grid, block, 0, st, a); \
    break;
  switch (jb) {
    ROWSK(1) ROWSK(2) ROWSK(3) ROWSK(4) ROWSK(5) ROWSK(6) ROWSK(7) ROWSK(8)
    default:
      return hipErrorInvalidValue;
  }
#undef ROWSK
  return hipGetLastError();
}

hipError_t launch_row_skinny(const RowArgs &a, Dtype dt, hipStream_t st) {
  if (a.r < 1 || a.r > 128) return hipErrorInvalidValue;
  if (dt == DT_BF16) {
    if (a.vmode == V_ROW) return row_dispatch<BF16, V_ROW>(a, st);
    if (a.r % 8 == 0) return row_dispatch<BF16, V_KMAJ_TR>(a, st);
    return row_dispatch<BF16, V_KMAJ_GATHER>(a, st);
  }
  if (a.vmode == V_ROW) return row_dispatch<F32, V_ROW>(a, st);
  return row_dispatch<F32, V_KMAJ_GATHER>(a, st);
}

}  // namespace lora
