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

constexpr int SEL_NT = 256, SEL_NW = SEL_NT / 64;  // the histogram has one bucket per thread
constexpr int SEL_MAX = 8192;  // candidate slots plus sort slots per row

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, off);
    const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), off);
    const uint64_t o = ((uint64_t)hi << 32) | lo;
    v = o < v ? o : v;
  }
  return v;
}

// Per row (one workgroup): the k best of the row's candidates.  final = 0:
// keep them (in the list's first k slots, in list order) and set the
// threshold to the k-th best similarity; final = 1: sort them (best first)
// into the table row.
//
// The k-th largest key is found by an MSB-first radix select, 8 bits a pass:
// a histogram of the keys that share the prefix chosen so far, then one wave
// locates the bucket holding the rank-th largest key with a suffix scan over
// its 256 counts.  The select stops as soon as that bucket holds exactly the
// keys still needed (usually after three or four passes, once the prefix
// isolates one similarity value); every key at or above the prefix is then
// among the k best.
static_assert(SEL_NT == 256, "one histogram bucket per thread");
__global__ __launch_bounds__(SEL_NT) void topk_select_kernel(float *cval, int32_t *cidx, int *cnt,
                                                             float *thr, int cap, int k, int final,
                                                             int32_t *table, float *tvals,
                                                             int64_t row0) {
  extern __shared__ uint64_t key[];  // [cap] candidates, then (final) [p2] kept keys
  __shared__ int hist[2][256];
  __shared__ int wcount[SEL_NW];
  __shared__ uint64_t wmin[SEL_NW];
  __shared__ uint64_t s_prefix;
  __shared__ int s_rank, s_done;
  const int row = blockIdx.x, t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int n = min(cnt[row], cap);
  float *rv = cval + (int64_t)row * cap;
  int32_t *ri = cidx + (int64_t)row * cap;
  if (!final && n <= k) return;
  for (int i = t; i < n; i += SEL_NT) key[i] = make_key(rv[i], ri[i]);
  uint64_t kth = 0;  // every key >= kth is among the k best (all when n <= k)
  if (n > k) {
    hist[0][t] = 0;
    hist[1][t] = 0;
    if (t == 0) {
      s_prefix = 0;
      s_rank = k;
      s_done = 0;
    }
    __syncthreads();
    for (int shift = 56, pb = 0;; shift -= 8, pb ^= 1) {
      const uint64_t prefix = s_prefix;
      const uint64_t hmask = shift == 56 ? 0 : ~0ull << (shift + 8);
      for (int i = t; i < n; i += SEL_NT) {
        const uint64_t kk = key[i];
        if ((kk & hmask) == prefix) atomicAdd(&hist[pb][(kk >> shift) & 0xFF], 1);
      }
      __syncthreads();
      if (wave == 0) {
        // lane l holds buckets 4l .. 4l+3; above = keys in higher buckets
        const int rank = s_rank;
        int h[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) h[j] = hist[pb][4 * lane + j];
        const int sl = h[0] + h[1] + h[2] + h[3];
        int x = sl;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
          const int y = __shfl_down(x, off);
          if (lane + off < 64) x += y;
        }
        int above = x - sl;
#pragma unroll
        for (int j = 3; j >= 0; --j) {
          if (above < rank && above + h[j] >= rank) {
            s_prefix = prefix | ((uint64_t)(4 * lane + j) << shift);
            s_rank = rank - above;
            s_done = h[j] == rank - above;
          }
          above += h[j];
        }
      } else {
        for (int b = t - 64; b < 256; b += SEL_NT - 64) hist[pb ^ 1][b] = 0;
      }
      __syncthreads();
      if (s_done || shift == 0) break;
    }
    kth = s_prefix;
  }
  // Compact the keys >= kth in list order: each wave takes a contiguous
  // range, counts its keys by ballot, then writes them after the lower waves'.
  const int per = ((n + SEL_NW - 1) / SEL_NW + 63) / 64 * 64;
  const int lo = min(n, wave * per), hi = min(n, lo + per);
  int c = 0;
  uint64_t mn = ~0ull;
  for (int i0 = lo; i0 < hi; i0 += 64) {
    const int i = i0 + lane;
    const bool keep = i < hi && key[i] >= kth;
    c += __popcll(__ballot(keep));
    if (keep) mn = key[i] < mn ? key[i] : mn;
  }
  mn = wave_min_u64(mn);
  if (lane == 0) {
    wcount[wave] = c;
    wmin[wave] = mn;
  }
  __syncthreads();
  int pos = 0;
  uint64_t kmin = ~0ull;
  for (int w = 0; w < SEL_NW; ++w) {
    if (w < wave) pos += wcount[w];
    kmin = wmin[w] < kmin ? wmin[w] : kmin;
  }
  const int kept = min(n, k);
  uint64_t *out = key + cap;
  for (int i0 = lo; i0 < hi; i0 += 64) {
    const int i = i0 + lane;
    const bool keep = i < hi && key[i] >= kth;
    const uint64_t bal = __ballot(keep);
    if (keep) {
      const int q = pos + __popcll(bal & ((1ull << lane) - 1));
      const uint64_t kk = key[i];
      if (final) {
        out[q] = kk;
      } else {
        rv[q] = unordered((uint32_t)(kk >> 32));
        ri[q] = (int32_t)(0xFFFFFFFFu - (uint32_t)kk);
      }
    }
    pos += __popcll(bal);
  }
  if (!final) {
    // the k-th best similarity: the smallest kept key's value
    if (t == 0) {
      cnt[row] = kept;
      thr[row] = unordered((uint32_t)(kmin >> 32));
    }
    return;
  }
  // final: bitonic sort of the kept keys, descending (pad with 0 = smallest)
  int p2 = 1;
  while (p2 < kept) p2 <<= 1;
  for (int i = kept + t; i < p2; i += SEL_NT) out[i] = 0;
  __syncthreads();
  for (int size = 2; size <= p2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = t; i < p2 / 2; i += SEL_NT) {
        const int a = 2 * i - (i & (stride - 1)), b = a + stride;
        const bool desc = (a & size) == 0;
        const uint64_t ka = out[a], kb = out[b];
        if ((ka < kb) == desc) {
          out[a] = kb;
          out[b] = ka;
        }
      }
      __syncthreads();
    }
  }
  for (int i = t; i < k; i += SEL_NT) {
    const uint64_t kk = i < kept ? out[i] : 0;
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
  if (a.k > 2048 || a.k < 1 || a.cap < a.k) return hipErrorInvalidValue;
  int p2 = 1;
  while (p2 < a.k) p2 <<= 1;
  const int slots = a.cap + (final ? p2 : 0);
  if (slots > SEL_MAX) return hipErrorInvalidValue;
  // up to 64 KB of dynamic LDS besides the static part (gfx950: 160 KB per CU)
  static const hipError_t attr = hipFuncSetAttribute(
      (const void *)topk_select_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, SEL_MAX * 8);
  if (attr != hipSuccess) return attr;
  const size_t lds = (size_t)slots * 8;
  hipLaunchKernelGGL(topk_select_kernel, dim3(R), dim3(SEL_NT), lds, st, a.val, a.idx, a.cnt, a.thr,
                     a.cap, a.k, final, a.table, a.tvals, a.row0);
  return hipGetLastError();
}

}  // namespace lora
