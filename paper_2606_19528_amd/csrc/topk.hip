// topk.hip -- the top-k cosine-similarity table of the embedding matrix
// (each token's k nearest tokens, the lookup table of the reduced-vocabulary
// softmax), built without ever storing the V x V similarities:
//   * the similarity GEMM runs over a batch of rows and one chunk of columns
//     at a time; its epilogue (gemm.hip, EPI_TOPK) appends to each row's
//     candidate list every cosine above the row's current threshold;
//   * after each chunk, topk_select_kernel keeps each row's k best
//     candidates (exact radix select on 64-bit keys: similarity, then the
//     smaller token index) and raises its threshold to the k-th best;
//   * after the last chunk, the same kernel sorts the k best and writes the
//     table row.
// The candidate set after a chunk does not depend on the order of the
// appends, so the table is deterministic.
#include <algorithm>

#include "kernels.hpp"
#include "launch.hpp"

namespace lora {

// rn[v] = 1 / |W[v]| (0 for a zero row); one wave per row.
__global__ void row_rnorm_kernel(const uint16_t *W, int V, int D, float *rn) {
  const int v = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (v >= V) return;
  float s = 0.0f;
  for (int d = lane * 8; d < D; d += 64 * 8) {
    const u32x4 q = ld16(W + (int64_t)v * D + d);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = __builtin_bit_cast(float, q[e] << 16), hi = __builtin_bit_cast(float, q[e] & 0xFFFF0000u);
      s += lo * lo + hi * hi;
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off);
  if (lane == 0) rn[v] = s > 0.0f ? 1.0f / sqrtf(s) : 0.0f;
}

__device__ __forceinline__ uint32_t ordered(float f) {
  const uint32_t u = __builtin_bit_cast(uint32_t, f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float unordered(uint32_t o) {
  return __builtin_bit_cast(float, (o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}
// larger key = higher similarity, then smaller token index
__device__ __forceinline__ uint64_t make_key(float v, int32_t j) {
  return ((uint64_t)ordered(v) << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)j);
}

constexpr int SEL_NT = 512;
constexpr int SEL_MAX = 8192;  // candidates per row (k + chunk)

// Per row (one workgroup): the k best of the row's candidates.  final = 0:
// keep them (in the list's first k slots) and set the threshold to the k-th
// best similarity; final = 1: sort them (best first) into the table row.
__global__ __launch_bounds__(SEL_NT) void topk_select_kernel(float *cval, int32_t *cidx, int *cnt,
                                                             float *thr, int cap, int k, int final,
                                                             int32_t *table, float *tvals,
                                                             int64_t row0) {
  __shared__ uint64_t key[SEL_MAX];
  __shared__ int hist[256];
  __shared__ int part[SEL_NT];
  __shared__ uint64_t s_prefix;
  __shared__ int s_rank;
  const int row = blockIdx.x, t = threadIdx.x;
  const int n = min(cnt[row], cap);
  float *rv = cval + (int64_t)row * cap;
  int32_t *ri = cidx + (int64_t)row * cap;
  if (!final && n <= k) return;
  for (int i = t; i < n; i += SEL_NT) key[i] = make_key(rv[i], ri[i]);
  __syncthreads();
  uint64_t kth = 0;  // every key >= kth is among the k best (all when n <= k)
  if (n > k) {
    // MSB-first radix select of the k-th largest key, 8 bits per pass
    if (t == 0) {
      s_prefix = 0;
      s_rank = k;
    }
    for (int shift = 56; shift >= 0; shift -= 8) {
      for (int b = t; b < 256; b += SEL_NT) hist[b] = 0;
      __syncthreads();
      const uint64_t prefix = s_prefix;
      const uint64_t hmask = shift == 56 ? 0 : ~0ull << (shift + 8);
      for (int i = t; i < n; i += SEL_NT)
        if ((key[i] & hmask) == prefix) atomicAdd(&hist[(key[i] >> shift) & 0xFF], 1);
      __syncthreads();
      if (t == 0) {
        int rank = s_rank, b = 255;
        while (hist[b] < rank) rank -= hist[b--];
        s_prefix = prefix | ((uint64_t)b << shift);
        s_rank = rank;
      }
      __syncthreads();
    }
    kth = s_prefix;
  }
  // compact the keys >= kth into the first slots, in list order (block scan)
  const int per = (n + SEL_NT - 1) / SEL_NT;
  const int lo = min(n, t * per), hi = min(n, lo + per);
  int c = 0;
  for (int i = lo; i < hi; ++i) c += key[i] >= kth;
  part[t] = c;
  __syncthreads();
  for (int off = 1; off < SEL_NT; off <<= 1) {
    const int add = t >= off ? part[t - off] : 0;
    __syncthreads();
    part[t] += add;
    __syncthreads();
  }
  int pos = part[t] - c;
  uint64_t mine[SEL_MAX / SEL_NT];
  int nm = 0;
  for (int i = lo; i < hi; ++i)
    if (key[i] >= kth) mine[nm++] = key[i];
  __syncthreads();
  for (int q = 0; q < nm; ++q) key[pos + q] = mine[q];
  const int kept = min(n, k);
  if (!final) {
    __syncthreads();
    for (int i = t; i < kept; i += SEL_NT) {
      rv[i] = unordered((uint32_t)(key[i] >> 32));
      ri[i] = (int32_t)(0xFFFFFFFFu - (uint32_t)key[i]);
    }
    if (t == 0) {
      cnt[row] = kept;
      thr[row] = unordered((uint32_t)(kth >> 32));
    }
    return;
  }
  // final: bitonic sort of the kept keys, descending (pad with 0 = smallest)
  int p2 = 1;
  while (p2 < kept) p2 <<= 1;
  for (int i = kept + t; i < p2; i += SEL_NT) key[i] = 0;
  __syncthreads();
  for (int size = 2; size <= p2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = t; i < p2 / 2; i += SEL_NT) {
        const int a = 2 * i - (i & (stride - 1)), b = a + stride;
        const bool desc = (a & size) == 0;
        const uint64_t ka = key[a], kb = key[b];
        if ((ka < kb) == desc) {
          key[a] = kb;
          key[b] = ka;
        }
      }
      __syncthreads();
    }
  }
  for (int i = t; i < k; i += SEL_NT) {
    const uint64_t kk = i < kept ? key[i] : 0;
    table[(row0 + row) * k + i] = i < kept ? (int32_t)(0xFFFFFFFFu - (uint32_t)kk) : -1;
    if (tvals) tvals[(row0 + row) * k + i] = i < kept ? unordered((uint32_t)(kk >> 32)) : 0.0f;
  }
}

__global__ void topk_reset_kernel(float *thr, int *cnt, int R) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < R) {
    thr[i] = -INFINITY;
    cnt[i] = 0;
  }
}

hipError_t launch_row_rnorm(const void *W, int V, int D, float *rn, hipStream_t st) {
  hipLaunchKernelGGL(row_rnorm_kernel, dim3((V + 3) / 4), dim3(256), 0, st, (const uint16_t *)W, V,
                     D, rn);
  return hipGetLastError();
}

hipError_t launch_topk_reset(float *thr, int *cnt, int R, hipStream_t st) {
  hipLaunchKernelGGL(topk_reset_kernel, dim3((R + 255) / 256), dim3(256), 0, st, thr, cnt, R);
  return hipGetLastError();
}

hipError_t launch_topk_select(const TopkArgs &a, int R, int final, hipStream_t st) {
  if (a.cap > SEL_MAX || a.k > 2048 || a.k < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(topk_select_kernel, dim3(R), dim3(SEL_NT), 0, st, a.val, a.idx, a.cnt, a.thr,
                     a.cap, a.k, final, a.table, a.tvals, a.row0);
  return hipGetLastError();
}

}  // namespace lora
