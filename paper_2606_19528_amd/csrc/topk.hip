// topk.hip -- the top-k cosine-similarity table of the embedding matrix
// (each token's k nearest tokens, the lookup table of the reduced-vocabulary
// softmax), built without ever storing the V x V similarities:
//   * the similarity GEMM runs over a batch of rows and one chunk of columns
//     at a time; its epilogue (gemm.hip, EPI_TOPK) appends to each row's
//     candidate list every cosine above the row's current threshold;
//   * after each chunk, topk_select_kernel keeps the k best candidates of
//     each row whose list might not hold another chunk (exact radix select on
//     64-bit keys: similarity, then the smaller token index) and raises its
//     threshold to the k-th best; with lists much longer than k + one chunk
//     a row is selected a handful of times instead of after every chunk;
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
constexpr int SEL_MAX = TOPK_SLOTS;

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
// rows with at most `lazy` candidates are left alone (their list still has
// room for the next chunk; the threshold stays where it was, which only lets
// more candidates in); the others keep their k best (in the list's first k
// slots) and set the threshold to the k-th best similarity.  final = 1: sort
// the k best (best first) into the table row.
//
// Each thread holds its candidates in registers: slots 4 (t + 256 q) + e,
// read four at a time (the list length is a multiple of 4, so a vector
// never leaves the list).  Key 0 marks an empty slot (every real key is
// larger).  The k-th largest key is found by an MSB-first radix select over
// the keys minus the row's smallest, up to 8 bits a pass starting at the top
// bit of their span: a histogram in LDS of the keys that share the prefix
// chosen so far, then one wave locates the bucket holding the rank-th largest
// key with a suffix scan over the 256 counts.  The select stops as soon as
// that bucket holds exactly the keys still needed (usually after two
// passes); every key at or above the prefix is then among the k best.  The
// kept keys are written out wave by wave in a fixed order.
constexpr int SEL_Q = SEL_MAX / (4 * SEL_NT);  // vectors of 4 slots per thread
static_assert(SEL_NT == 256, "one histogram bucket per thread");
__global__ __launch_bounds__(SEL_NT) void topk_select_kernel(float *cval, int32_t *cidx, int *cnt,
                                                             float *thr, int cap, int k, int lazy,
                                                             int final, int32_t *table, float *tvals,
                                                             int64_t row0) {
  __shared__ uint64_t out[2048];  // final: the kept keys, sorted in place
  __shared__ int hist[2][256];
  __shared__ int wcount[SEL_NW];
  __shared__ uint64_t wmin[SEL_NW], wmax[SEL_NW];
  __shared__ uint64_t s_prefix;
  __shared__ int s_rank, s_done;
  const int row = blockIdx.x, t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int n = min(cnt[row], cap);
  float *rv = cval + (int64_t)row * cap;
  int32_t *ri = cidx + (int64_t)row * cap;
  if (!final && n <= (lazy > k ? lazy : k)) return;  // room left for the next chunk
  uint64_t key[SEL_Q][4];
#pragma unroll
  for (int q = 0; q < SEL_Q; ++q) {
    const int b = 4 * (t + SEL_NT * q);
    if (b < n) {
      const float4 v = *(const float4 *)(rv + b);
      const int4 x = *(const int4 *)(ri + b);
      key[q][0] = make_key(v.x, x.x);
      key[q][1] = b + 1 < n ? make_key(v.y, x.y) : 0;
      key[q][2] = b + 2 < n ? make_key(v.z, x.z) : 0;
      key[q][3] = b + 3 < n ? make_key(v.w, x.w) : 0;
    } else {
      key[q][0] = key[q][1] = key[q][2] = key[q][3] = 0;
    }
  }
  uint64_t kth = 1;  // every key >= kth is among the k best (all real keys when n <= k)
  if (n > k) {
    // The digits are taken from the key minus the row's smallest key, the
    // first one from the top bit of the span, so the first histogram spreads
    // over the keys' actual range (similarities share their sign and most of
    // their exponent bits, which would put nearly every key in one bucket).
    uint64_t lo = ~0ull, hi = 0;
#pragma unroll
    for (int q = 0; q < SEL_Q; ++q)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint64_t kk = key[q][e];
        lo = (kk != 0 && kk < lo) ? kk : lo;
        hi = kk > hi ? kk : hi;
      }
    lo = wave_min_u64(lo);
    hi = ~wave_min_u64(~hi);
    if (lane == 0) {
      wmin[wave] = lo;
      wmax[wave] = hi;
    }
    hist[0][t] = 0;
    hist[1][t] = 0;
    if (t == 0) {
      s_prefix = 0;
      s_rank = k;
      s_done = 0;
    }
    __syncthreads();
#pragma unroll
    for (int w = 0; w < SEL_NW; ++w) {
      lo = wmin[w] < lo ? wmin[w] : lo;
      hi = wmax[w] > hi ? wmax[w] : hi;
    }
    const int top = 63 - __clzll(hi - lo);  // keys are distinct and n >= 2, so hi > lo
    // Pass: digit = bits [shift, shift + width) of key - lo among the keys
    // whose bits above them equal the prefix chosen so far.
    int width = top < 8 ? top + 1 : 8;
    int shift = top + 1 - width;
    for (int pb = 0;; pb ^= 1) {
      const uint64_t prefix = s_prefix;  // chosen bits above shift + width, in place
      const uint64_t hmask = shift + width >= 64 ? 0 : ~0ull << (shift + width);
      const uint32_t dmask = (1u << width) - 1;
#pragma unroll
      for (int q = 0; q < SEL_Q; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint64_t r = key[q][e] - lo;
          if (key[q][e] != 0 && (r & hmask) == prefix) atomicAdd(&hist[pb][(r >> shift) & dmask], 1);
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
      width = shift < 8 ? shift : 8;
      shift -= width;
    }
    kth = lo + s_prefix;
  }
  // Write the keys >= kth: each wave counts its kept keys, then writes them
  // after the lower waves' (per vector slot q, element e, lane order).
  int c = 0;
  uint64_t mn = ~0ull;
#pragma unroll
  for (int q = 0; q < SEL_Q; ++q)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool keep = key[q][e] >= kth;
      c += __popcll(__ballot(keep));
      mn = keep && key[q][e] < mn ? key[q][e] : mn;
    }
  mn = wave_min_u64(mn);
  if (lane == 0) {
    wcount[wave] = c;
    wmin[wave] = mn;
  }
  __syncthreads();
  int pos = 0;
  uint64_t kmin = ~0ull;
#pragma unroll
  for (int w = 0; w < SEL_NW; ++w) {
    if (w < wave) pos += wcount[w];
    kmin = wmin[w] < kmin ? wmin[w] : kmin;
  }
  const int kept = min(n, k);
#pragma unroll
  for (int q = 0; q < SEL_Q; ++q)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint64_t kk = key[q][e];
      const bool keep = kk >= kth;
      const uint64_t bal = __ballot(keep);
      if (keep) {
        const int o = pos + __popcll(bal & ((1ull << lane) - 1));
        if (final) {
          out[o] = kk;
        } else {
          rv[o] = unordered((uint32_t)(kk >> 32));
          ri[o] = (int32_t)(0xFFFFFFFFu - (uint32_t)kk);
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
  if (a.k > 2048 || a.k < 1 || a.cap < a.k || a.lazy > a.cap || a.cap > SEL_MAX || a.cap % 4)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(topk_select_kernel, dim3(R), dim3(SEL_NT), 0, st, a.val, a.idx, a.cnt, a.thr,
                     a.cap, a.k, a.lazy, final, a.table, a.tvals, a.row0);
  return hipGetLastError();
}

}  // namespace lora
