// colred.hpp -- token-reduced rank-r products run as extra workgroups of the
// backward GEMM launch (they overlap with the dx tiles):
//   dA = du^T x   and   dB = s dy^T u,
// both of the form out[l][j] = scale * sum_t X[t][l] V[t][j] with X a bf16 (or
// fp32) activation [T, L] and V an fp32 [T, r] matrix, possibly given as
// partial sums over a split reduction (added in ascending order on load).
//
// One work item = (column block of 16*VEC columns, group of 32 rank indices)
// over all T tokens, so no partial sums leave the workgroup (cross-workgroup
// reductions would need device-scope fences, which write back and invalidate
// the per-XCD L2s).  Each wave reads VEC rows x 16 bytes of X (row-major,
// coalesced), transposes the VEC x VEC block in registers so a lane holds VEC
// consecutive tokens of one column -- the matrix-core operand whose reduction
// axis is the token axis -- and accumulates a (16*VEC) x 32 tile, two token
// steps in flight.  The waves take interleaved token steps; their tiles are
// summed in LDS by a fixed pairwise tree, so the result is deterministic.
#pragma once

#include "kernels.hpp"
#include "launch.hpp"

namespace lora {

constexpr int SIDE_JB = 2;  // rank indices per item: 32

template <class E>
struct SideShape {
  static constexpr int VEC = E::VEC;
  static constexpr int COLS = 16 * VEC;  // columns per item
  static constexpr int ROWS = 4 * VEC;   // tokens per wave step
};

// LDS bytes the side items need with NW waves.
template <class E, int NW>
constexpr int side_lds_bytes() {
  return (NW / 2) * SideShape<E>::COLS * (SIDE_JB * 16 + 1) * 4;
}

template <class E>
__device__ __forceinline__ int side_items_of(const ColJob &job, const SideArgs &s) {
  const int ncb = (job.L + SideShape<E>::COLS - 1) / SideShape<E>::COLS;
  return ncb * ((s.r + 31) / 32);
}

template <class E>
__device__ __forceinline__ int side_items_total(const SideArgs &s) {
  int n = 0;
  for (int i = 0; i < s.njobs; ++i) n += side_items_of<E>(s.job[i], s);
  return n;
}

template <class E, int NW>
__device__ void side_item(const SideArgs &s, int item, char *smem) {
  typedef typename E::T T;
  constexpr int VEC = E::VEC;
  constexpr int COLS = SideShape<E>::COLS;
  constexpr int ROWS = SideShape<E>::ROWS;
  constexpr int JB = SIDE_JB;
  constexpr int RS = JB * 16 + 1;  // padded LDS row (floats)

  int ji = 0;
  {
    const int n0 = side_items_of<E>(s.job[0], s);
    if (item >= n0) {
      ji = 1;
      item -= n0;
    }
  }
  const ColJob &job = s.job[ji];
  const int r = s.r;
  const int ngz = (r + 31) / 32;
  const int z = item % ngz;
  const int cb = item / ngz;
  const int jg = z * 32;
  const int c0 = cb * COLS;
  const int t_end = s.T;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, cl = lane & 15;
  const int col = c0 + cl * VEC;
  const T *Xp = (const T *)job.X;

  f32x4 acc[VEC][JB];
#pragma unroll
  for (int q = 0; q < VEC; ++q)
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) acc[q][jb] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto step = [&](int tb) {
    u32x4 xin[VEC], xt[VEC];
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
      const int t = tb + g * VEC + i;
      xin[i] = (t < t_end && col < job.L) ? ld16(Xp + (int64_t)t * job.ldx + col) : zero16();
    }
    u32x4 vf[JB];
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) {
      const int j = jg + jb * 16 + cl;
      float f[VEC];
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const int t = tb + g * VEC + e;
        float part[MAX_SPLIT];  // all loads issued before the first add
        const bool ok = t < t_end && j < r;
        const float *src = job.V + (int64_t)t * r + j;
#pragma unroll
        for (int q = 0; q < MAX_SPLIT; ++q) part[q] = (ok && q < job.vparts) ? src[q * job.vstride] : 0.0f;
        float v = part[0];
#pragma unroll
        for (int q = 1; q < MAX_SPLIT; ++q)
          if (q < job.vparts) v += part[q];
        f[e] = v;
      }
      vf[jb] = pack_vec(E(), f);
    }
    transpose_block(E(), xin, xt);
#pragma unroll
    for (int q = 0; q < VEC; ++q)
#pragma unroll
      for (int jb = 0; jb < JB; ++jb) mma16(E(), acc[q][jb], xt[q], vf[jb]);
  };
  for (int tb = wave * ROWS; tb < t_end; tb += 2 * NW * ROWS) {
    step(tb);
    if (tb + NW * ROWS < t_end) step(tb + NW * ROWS);
  }

  // Pairwise tree over waves: in round h the upper half of the active waves
  // writes, the lower half adds (wave w receives wave w + h).
  // acc[q][jb] element i: local column (4g + i) * VEC + q, rank index 16 jb + cl.
  float *red = (float *)smem;
#pragma unroll
  for (int h = NW / 2; h >= 1; h /= 2) {
    __syncthreads();
    if (wave >= h && wave < 2 * h) {
      float *slot = red + (wave - h) * COLS * RS;
#pragma unroll
      for (int q = 0; q < VEC; ++q)
#pragma unroll
        for (int jb = 0; jb < JB; ++jb)
#pragma unroll
          for (int i = 0; i < 4; ++i) slot[((4 * g + i) * VEC + q) * RS + jb * 16 + cl] = acc[q][jb][i];
    }
    __syncthreads();
    if (wave < h) {
      const float *slot = red + wave * COLS * RS;
#pragma unroll
      for (int q = 0; q < VEC; ++q)
#pragma unroll
        for (int jb = 0; jb < JB; ++jb)
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[q][jb][i] += slot[((4 * g + i) * VEC + q) * RS + jb * 16 + cl];
    }
  }
  // Wave 0 holds the item's tile: scale and store it.
  const int jn = min(32, r - jg);
  if (wave == 0) {
#pragma unroll
    for (int q = 0; q < VEC; ++q)
#pragma unroll
      for (int jb = 0; jb < JB; ++jb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int l = c0 + (4 * g + i) * VEC + q;
          const int j = jb * 16 + cl;
          if (l < job.L && j < jn) {
            const float v = job.scale * acc[q][jb][i];
            if (job.transpose_out)
              job.out[(int64_t)(jg + j) * job.L + l] = v;
            else
              job.out[(int64_t)l * r + jg + j] = v;
          }
        }
  }
}

}  // namespace lora
