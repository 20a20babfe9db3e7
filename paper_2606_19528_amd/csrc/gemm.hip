// gemm.hip -- LDS-tiled matrix-core GEMM for the two big contractions of the
// LoRA linear, each with the rank-r LoRA term folded in as extra reduction
// steps:
//   forward   y  = [x | s*u] [W | B]^T          (NT: both operands k-contiguous)
//   backward  dx = [dy | du] [W ; A]            (NN: W and A are k-major, i.e.
//                                                 the reduction index is the row)
//   frozen    dx = dy W                          (NN, no tail)
// One workgroup computes a BM x BN output tile.  The reduction runs over
// 128-byte k-stages staged through double-buffered LDS (one barrier per
// stage); the next stage's global loads are issued before the current
// stage's MFMAs.  k-major operands are transposed in registers (VEC x VEC
// blocks) on their way into LDS, so the LDS layout -- rows of 128 bytes of k
// plus 16 bytes of padding -- is the same for every operand.
#include "kernels.hpp"
#include "launch.hpp"

namespace lora {

template <class E, int BM, int BN, int WM, int WN, bool KMAJ>
__global__ __launch_bounds__(WM * WN * 64) void gemm_kernel(GemmArgs g) {
  typedef typename E::T T;
  constexpr int NT = WM * WN * 64;
  constexpr int VEC = E::VEC;
  constexpr int BKB = 128;                  // k bytes per stage and row
  constexpr int BKE = BKB / (int)sizeof(T); // k elements per stage
  constexpr int ROWB = BKB + 16;            // padded LDS row
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int FM = WTM / 32, FN = WTN / 32;
  constexpr int CPR = BKB / 16;             // 16-byte chunks per row and stage
  constexpr int A_CH = BM * CPR, A_PER = (A_CH + NT - 1) / NT;
  constexpr int B_CH = BN * CPR, B_PER = (B_CH + NT - 1) / NT;
  constexpr int NBV = BN / VEC;             // k-major: VEC x VEC blocks per k-row band
  constexpr int KB_BLK = (BKE / VEC) * NBV, KB_PER = (KB_BLK + NT - 1) / NT;
  constexpr int RB = KMAJ ? KB_PER * VEC : B_PER;
  static_assert(BM % (WM * 32) == 0 && BN % (WN * 32) == 0, "tile shape");

  __shared__ __align__(16) char smem[2 * (BM + BN) * ROWB];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  const int tiles_m = (g.M + BM - 1) / BM;
  const int mt = blockIdx.x % tiles_m;
  const int nt = blockIdx.x / tiles_m;
  const int m0 = mt * BM, n0 = nt * BN;

  const char *Ab = (const char *)g.A;
  const char *Bb = (const char *)g.B;
  const int nk_main = (g.K + BKE - 1) / BKE;
  const int nk_tail = g.r > 0 ? (g.r + BKE - 1) / BKE : 0;
  const int nk = nk_main + nk_tail;

  u32x4 ra[A_PER];
  u32x4 rb[RB];

  auto load_stage = [&](int kt) {
    if (kt < nk_main) {
      const int k0 = kt * BKE;
#pragma unroll
      for (int i = 0; i < A_PER; ++i) {
        const int c = tid + i * NT;
        const int row = c / CPR, kc = c % CPR;
        const int m = m0 + row, k = k0 + kc * VEC;
        ra[i] = (c < A_CH && m < g.M && k < g.K)
                    ? ld16(Ab + ((int64_t)m * g.lda + k) * (int64_t)sizeof(T))
                    : zero16();
      }
      if constexpr (!KMAJ) {
#pragma unroll
        for (int i = 0; i < B_PER; ++i) {
          const int c = tid + i * NT;
          const int row = c / CPR, kc = c % CPR;
          const int n = n0 + row, k = k0 + kc * VEC;
          rb[i] = (c < B_CH && n < g.N && k < g.K)
                      ? ld16(Bb + ((int64_t)n * g.ldb + k) * (int64_t)sizeof(T))
                      : zero16();
        }
      } else {
#pragma unroll
        for (int i = 0; i < KB_PER; ++i) {
          const int b = tid + i * NT;
          const int kb = b / NBV, nb = b % NBV;
          const int n = n0 + nb * VEC;
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            const int k = k0 + kb * VEC + e;
            rb[i * VEC + e] = (b < KB_BLK && n < g.N && k < g.K)
                                  ? ld16(Bb + ((int64_t)k * g.ldb + n) * (int64_t)sizeof(T))
                                  : zero16();
          }
        }
      }
    } else {
      // LoRA tail stage: reduction index j in [j0, j0 + BKE), valid below r.
      const int j0 = (kt - nk_main) * BKE;
#pragma unroll
      for (int i = 0; i < A_PER; ++i) {
        const int c = tid + i * NT;
        const int row = c / CPR, kc = c % CPR;
        const int m = m0 + row;
        float f[VEC];
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const int j = j0 + kc * VEC + e;
          f[e] = (c < A_CH && m < g.M && j < g.r) ? g.s2 * g.A2[(int64_t)m * g.r + j] : 0.0f;
        }
        ra[i] = pack_vec(E(), f);
      }
      const T *B2 = (const T *)g.B2;
      if constexpr (!KMAJ) {
#pragma unroll
        for (int i = 0; i < B_PER; ++i) {
          const int c = tid + i * NT;
          const int row = c / CPR, kc = c % CPR;
          const int n = n0 + row;
          float f[VEC];
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            const int j = j0 + kc * VEC + e;
            f[e] = (c < B_CH && n < g.N && j < g.r) ? E::to_float(B2[(int64_t)n * g.r + j]) : 0.0f;
          }
          rb[i] = pack_vec(E(), f);
        }
      } else {
#pragma unroll
        for (int i = 0; i < KB_PER; ++i) {
          const int b = tid + i * NT;
          const int kb = b / NBV, nb = b % NBV;
          const int n = n0 + nb * VEC;
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            const int j = j0 + kb * VEC + e;
            rb[i * VEC + e] = (b < KB_BLK && n < g.N && j < g.r)
                                  ? ld16(B2 + (int64_t)j * g.ldb2 + n)
                                  : zero16();
          }
        }
      }
    }
  };

  auto store_stage = [&](int buf) {
    char *sA = smem + buf * (BM + BN) * ROWB;
    char *sB = sA + BM * ROWB;
#pragma unroll
    for (int i = 0; i < A_PER; ++i) {
      const int c = tid + i * NT;
      if (c < A_CH) st16(sA + (c / CPR) * ROWB + (c % CPR) * 16, ra[i]);
    }
    if constexpr (!KMAJ) {
#pragma unroll
      for (int i = 0; i < B_PER; ++i) {
        const int c = tid + i * NT;
        if (c < B_CH) st16(sB + (c / CPR) * ROWB + (c % CPR) * 16, rb[i]);
      }
    } else {
#pragma unroll
      for (int i = 0; i < KB_PER; ++i) {
        const int b = tid + i * NT;
        if (b < KB_BLK) {
          const int kb = b / NBV, nb = b % NBV;
          u32x4 t[VEC];
          transpose_block(E(), &rb[i * VEC], t);
#pragma unroll
          for (int c = 0; c < VEC; ++c) st16(sB + (nb * VEC + c) * ROWB + kb * 16, t[c]);
        }
      }
    }
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.0f;

  load_stage(0);
  store_stage(0);
  __syncthreads();

  const int lrow = lane & 31;
  const int lko = (lane >> 5) * 16;
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) load_stage(kt + 1);
    const char *sA = smem + (kt & 1) * (BM + BN) * ROWB;
    const char *sB = sA + BM * ROWB;
#pragma unroll
    for (int s = 0; s < BKB / 32; ++s) {
      u32x4 af[FM], bf[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) af[i] = ld16(sA + (wm * WTM + i * 32 + lrow) * ROWB + s * 32 + lko);
#pragma unroll
      for (int j = 0; j < FN; ++j) bf[j] = ld16(sB + (wn * WTN + j * 32 + lrow) * ROWB + s * 32 + lko);
      // D = Bop * Aop^T: D rows are output columns n, D columns are rows m, so
      // each lane ends up holding runs of 4 consecutive n of one output row.
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) mma32(E(), acc[i][j], bf[j], af[i]);
    }
    if (kt + 1 < nk) store_stage((kt + 1) & 1);
    __syncthreads();
  }

  // Epilogue: lane holds D[n][m] at m = lane % 32, n = 8q + 4(lane / 32) + e
  // for accumulator element 4q + e.
  T *C = (T *)g.C;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int m = m0 + wm * WTM + i * 32 + lrow;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = n0 + wn * WTN + j * 32 + 8 * q + 4 * (lane >> 5);
        if (m < g.M && n < g.N) {
          T *dst = C + (int64_t)m * g.ldc + n;
          if constexpr (sizeof(T) == 2) {
            uint32_t lo = (uint32_t)E::from_float(acc[i][j][4 * q + 0]) |
                          ((uint32_t)E::from_float(acc[i][j][4 * q + 1]) << 16);
            uint32_t hi = (uint32_t)E::from_float(acc[i][j][4 * q + 2]) |
                          ((uint32_t)E::from_float(acc[i][j][4 * q + 3]) << 16);
            *(uint2 *)dst = make_uint2(lo, hi);
          } else {
            *(f32x4 *)dst = f32x4{acc[i][j][4 * q + 0], acc[i][j][4 * q + 1],
                                  acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
          }
        }
      }
    }
  }
}

template <class E, int BM, int BN, int WM, int WN, bool KMAJ>
static hipError_t launch_tile(const GemmArgs &g, hipStream_t st) {
  const int tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  hipLaunchKernelGGL((gemm_kernel<E, BM, BN, WM, WN, KMAJ>), dim3(tiles), dim3(WM * WN * 64), 0,
                     st, g);
  return hipGetLastError();
}

hipError_t launch_gemm(const GemmArgs &g, Dtype dt, bool b_kmajor, hipStream_t st) {
  if (dt == DT_BF16)
    return b_kmajor ? launch_tile<BF16, 128, 128, 2, 2, true>(g, st)
                    : launch_tile<BF16, 128, 128, 2, 2, false>(g, st);
  return b_kmajor ? launch_tile<F32, 128, 128, 2, 2, true>(g, st)
                  : launch_tile<F32, 128, 128, 2, 2, false>(g, st);
}

}  // namespace lora
