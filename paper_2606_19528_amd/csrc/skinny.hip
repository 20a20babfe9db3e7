// skinny.hip -- the rank-r "row" products of the LoRA linear as a kernel of
// their own: one read of a big activation [T, L] against a small [r, L]
// factor, reduced over the long axis L (the work item is in rowprod.hpp).
//   forward   u  = x A^T                    (A row-major [r, d_in])
//   backward  du = s dy B                   (B k-major   [d_out, r])
// Each workgroup owns 16 * mb rows and one segment of the reduction axis (the
// axis is split so that the row blocks times the segments give about one
// workgroup per CU).  Each segment's sum is written separately: the GEMM that
// consumes the LoRA-step operand adds the segments as extra reduction
// columns, and the other consumers add them in ascending order when they load
// them.
#include <algorithm>

#include "rowprod.hpp"

namespace lora {

template <class E, int JB, int VMODE, int U, int MB>
__global__ __launch_bounds__(64 * ROW_NW) void row_skinny_kernel(RowArgs a) {
  __shared__ __align__(16) char smem[row_lds_bytes<E, JB, VMODE, U, MB>()];
  row_item<E, JB, VMODE, U, MB>(a, blockIdx.x, blockIdx.y, gridDim.x, gridDim.y, smem);
  // After the row work, so that nothing delays its first loads.
  if (blockIdx.x == 0 && blockIdx.y == 0)
    for (int i = threadIdx.x; i < a.nzero; i += blockDim.x) a.zero[i] = 0;
}

template <class E, int VMODE, int MB>
static hipError_t row_dispatch(const RowArgs &a, hipStream_t st) {
  dim3 grid((a.M + 16 * MB - 1) / (16 * MB), a.nsplit), block(64 * ROW_NW);
  const int jb = (a.r + 15) / 16;
#define ROWSK(J)                                                                                      \
  case J:                                                                                             \
    hipLaunchKernelGGL((row_skinny_kernel<E, J, VMODE, (J <= 2 ? 4 : 1), MB>), grid, block, 0, st, a); \
    break;
  if constexpr (MB == 1) {
    switch (jb) {
      ROWSK(1) ROWSK(2) ROWSK(3) ROWSK(4) ROWSK(5) ROWSK(6) ROWSK(7) ROWSK(8)
      default:
        return hipErrorInvalidValue;
    }
  } else {
    switch (jb) {  // several row tiles: ranks up to 32
      ROWSK(1) ROWSK(2)
      default:
        return hipErrorInvalidValue;
    }
  }
#undef ROWSK
  return hipGetLastError();
}

template <class E, int VMODE>
static hipError_t row_dispatch_mb(const RowArgs &a, hipStream_t st) {
  switch (a.mb) {
    case 0:
    case 1:
      return row_dispatch<E, VMODE, 1>(a, st);
    case 2:
      return row_dispatch<E, VMODE, 2>(a, st);
    case 4:
      return row_dispatch<E, VMODE, 4>(a, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_row_skinny(const RowArgs &a, Dtype dt, hipStream_t st) {
  if (a.r < 1 || a.r > 128 || a.nsplit < 1 || a.nsplit > MAX_SPLIT || a.seg < 1) return hipErrorInvalidValue;
  if ((int64_t)(a.nsplit - 1) * a.seg >= a.L || (int64_t)a.nsplit * a.seg < a.L) return hipErrorInvalidValue;
  if (a.tail && a.nsplit * a.r > a.ldt) return hipErrorInvalidValue;
  if (a.mb > 1 && (a.r > 32 || dt != DT_BF16)) return hipErrorInvalidValue;
  if (a.nzero < 0 || (a.nzero > 0 && !a.zero)) return hipErrorInvalidValue;
  if (dt == DT_BF16) {
    if (a.vmode == V_ROW) return row_dispatch_mb<BF16, V_ROW>(a, st);
    if (a.r % 8 == 0) return row_dispatch_mb<BF16, V_KMAJ_TR>(a, st);
    return row_dispatch_mb<BF16, V_KMAJ_GATHER>(a, st);
  }
  if (a.vmode == V_ROW) return row_dispatch<F32, V_ROW, 1>(a, st);
  return row_dispatch<F32, V_KMAJ_GATHER, 1>(a, st);
}

RowSplit row_split(int64_t T, int64_t L, int r, Dtype dt) {
  const int ce = dt == DT_BF16 ? 64 : 32;  // elements per 128-byte chunk
  const int64_t max_by_l = std::max<int64_t>(1, (L + (int64_t)ROW_NW * ce - 1) / ((int64_t)ROW_NW * ce));
  auto make = [&](int64_t s, int mb) {
    s = std::max<int64_t>(1, std::min<int64_t>(s, max_by_l));
    const int64_t seg = ((L + s - 1) / s + ce - 1) / ce * ce;
    return RowSplit{(int)((L + seg - 1) / seg), (int)seg, mb};
  };
  if (dt == DT_BF16 && r <= 32 && r % 8 == 0 && T >= 16 * 256 && L <= 4096) {
    // 16-row blocks fill the machine on their own: whole rows, no partial
    // sums (measured at T = 4096, r = 32 against 32 rows x 2 segments: 5.5
    // against 6.2 us at L = 3072, 3.9 against 4.0 us at L = 1024; at L = 8192
    // the two segments win, 13.6 against 17.2 us).
    return make(1, 1);
  }
  if (dt == DT_BF16 && r <= 32 && r % 8 == 0 && T >= 2048 && T < 16 * 256) {
    // Two segments of 16-row blocks: the dA / dB side items, which read every
    // partial sum, then read two instead of four (measured at T = 2048:
    // Qwen layer 1.017 -> 1.003 ms per step, Llama MLP unchanged).
    return make(2, 1);
  }
  if (dt == DT_BF16 && r <= 32 && r % 8 == 0 && T >= 2048) {
    // (at most 4 partial sums: every dA / dB side item reads all of them)
    const int64_t smax = std::min<int64_t>({(int64_t)4, std::max(1, tail_ld(r, dt) / r), max_by_l});
    for (int mb : {4, 2}) {
      const int64_t blocks = (T + 16 * mb - 1) / (16 * mb);
      if (blocks * smax >= 256) return make((256 + blocks - 1) / blocks, mb);
    }
    const int64_t blocks = (T + 15) / 16;
    return make(std::min<int64_t>(smax, (256 + blocks - 1) / blocks), 1);
  }
  const int64_t blocks = (T + 15) / 16;
  int64_t s = (256 + blocks - 1) / blocks;
  s = std::min<int64_t>(s, std::max(1, tail_ld(r, dt) / r));
  s = std::min<int64_t>(s, MAX_SPLIT);
  return make(s, 1);
}

}  // namespace lora
