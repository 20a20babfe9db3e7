// colred.hpp -- token-reduced rank-r products run as extra workgroups of the
// backward GEMM launch (they overlap with the dx tiles):
//   dA = du^T x   and   dB = s dy^T u,
// both of the form out[l][j] = scale * sum_t X[t][l] V[t][j] with X a bf16 (or
// fp32) activation [T, L] and V an fp32 [T, r] matrix, possibly given as
// partial sums over a split reduction (added in ascending order on load).
//
// One work item = (column block of 16*VEC columns, group of 32 rank indices)
// over all T tokens -- or, in an unfused launch whose tiles leave CUs idle,
// over one of `tparts` consecutive token ranges, the last part to finish
// adding the parts' tiles in ascending part order (SideArgs), so the result
// does not depend on the order the parts finish in.  Each wave reads VEC rows x 16 bytes of X (row-major,
// coalesced), transposes the VEC x VEC block in registers so a lane holds VEC
// consecutive tokens of one column -- the matrix-core operand whose reduction
// axis is the token axis -- and accumulates a (16*VEC) x 32 tile, two token
// steps in flight.  Eight (virtual) waves take interleaved token steps; their
// tiles are summed by a fixed pairwise tree, so the result is deterministic
// and the same whether the launch has eight waves per workgroup or four (a
// wave then runs virtual waves w and w + 4 and adds the two tiles first, the
// tree's first round).
#pragma once

#include "kernels.hpp"
#include "launch.hpp"

namespace lora {

constexpr int SIDE_JB = 2;  // rank indices per item: 32

template <int V>
struct SideIC {
  static constexpr int value = V;
};
template <int B, int E, class F>
__device__ __forceinline__ void static_for_side(F &&f) {
  if constexpr (B < E) {
    f(SideIC<B>());
    static_for_side<B + 1, E>(f);
  }
}

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

// Work items: job 0's, then job 1's (counted on the host: side_count).
template <class E>
__device__ __forceinline__ int side_items_total(const SideArgs &s) {
  return s.ntot;
}

// Always inlined: called as a function, it takes the launch's arguments by
// address, so every wave of the launch first copies them to scratch memory.
// PARTS: the launch may run its items as token parts (s.tparts > 1); the
// fused launches (no registers to spare) run every item over all T.
template <class E, int NW, bool PARTS>
__device__ __forceinline__ void side_item(const SideArgs &s, int item, char *smem) {
  typedef typename E::T T;
  constexpr int VEC = E::VEC;
  constexpr int COLS = SideShape<E>::COLS;
  constexpr int ROWS = SideShape<E>::ROWS;
  constexpr int JB = SIDE_JB;
  constexpr int RS = JB * 16 + 1;  // padded LDS row (floats)

  // Work unit -> (item, token part).
  const int unit = item;
  const int tparts = PARTS ? s.tparts : 1;
  int part = 0;
  if (tparts > 1) {
    item = unit / tparts;
    part = unit - item * tparts;
  }
  const int gitem = item;
  int ji = 0;
  if (item >= s.n0) {
    ji = 1;
    item -= s.n0;
  }
  // The job's fields, each a select between the two jobs' (indexing the job
  // array with the run-time ji would copy the arguments to scratch memory).
  const void *jX = ji ? s.job[1].X : s.job[0].X;
  const float *jV = ji ? s.job[1].V : s.job[0].V;
  float *jout = ji ? s.job[1].out : s.job[0].out;
  const int jL = ji ? s.job[1].L : s.job[0].L;
  const int jvparts = ji ? s.job[1].vparts : s.job[0].vparts;
  const float jscale = ji ? s.scale1 : 1.0f;
  const int r = s.r;
  const int ngz = (r + 31) / 32;
  const int z = item % ngz;
  const int cb = item / ngz;
  const int jg = z * 32;
  const int c0 = cb * COLS;
  const int t_begin = part * s.tchunk;
  const int t_end = tparts > 1 ? min(s.T, t_begin + s.tchunk) : s.T;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, cl = lane & 15;
  const int col = c0 + cl * VEC;
  const T *Xp = (const T *)jX;

  constexpr int VW = 8, PER = VW / NW;  // virtual waves, per real wave
  static_assert(NW * PER == VW, "four or eight waves");
  f32x4 acc[PER][VEC][JB];
#pragma unroll
  for (int p = 0; p < PER; ++p)
#pragma unroll
    for (int q = 0; q < VEC; ++q)
#pragma unroll
      for (int jb = 0; jb < JB; ++jb) acc[p][q][jb] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Loads go through buffer resources based at the step's first token row
  // (so every offset stays small whatever T is): rows past T and columns past
  // L (or rank indices past r) read zeros without branches.  The loads of a
  // token step are issued one step ahead of its MFMAs.
  constexpr uint32_t OOB = 0x80000000u;
  constexpr int ES = (int)sizeof(T);
  struct Step {
    u32x4 x[VEC];
    float v[JB][VEC];
  };
  auto load = [&](int tb, Step &st) {
    const int rows = min(ROWS, t_end - tb);  // <= 0 past the end: nothing is read
    const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(Xp + (int64_t)tb * jL), (short)0, rows > 0 ? rows * jL * ES : 0, 0x00020000);
#pragma unroll
    for (int i = 0; i < VEC; ++i)
      st.x[i] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                     rx, col < jL ? (uint32_t)(((g * VEC + i) * jL + col) * ES) : OOB, 0, 0));
    // V and its further partial sums, added in ascending order (uniform loop)
    for (int q = 0; q < jvparts; ++q) {
      const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
          (void *)(jV + (int64_t)q * s.vstride + (int64_t)tb * r), (short)0, rows > 0 ? rows * r * 4 : 0,
          0x00020000);
#pragma unroll
      for (int jb = 0; jb < JB; ++jb) {
        const int j = jg + jb * 16 + cl;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const uint32_t off = j < r ? (uint32_t)(((g * VEC + e) * r + j) * 4) : OOB;
          const float v = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rv, off, 0, 0));
          st.v[jb][e] = q == 0 ? v : st.v[jb][e] + v;
        }
      }
    }
  };
  auto compute = [&](const Step &st, f32x4(&a)[VEC][JB]) {
    u32x4 xt[VEC], vf[JB];
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) vf[jb] = pack_vec(E(), st.v[jb]);
    transpose_block(E(), st.x, xt);
#pragma unroll
    for (int q = 0; q < VEC; ++q)
#pragma unroll
      for (int jb = 0; jb < JB; ++jb) mma16(E(), a[q][jb], xt[q], vf[jb]);
  };
  {
    // Step n of this wave: virtual wave w + NW (n % PER), its (n / PER)-th
    // token step.  Each virtual wave runs its own steps in ascending order,
    // exactly as a wave of an eight-wave workgroup would.
    const int w0 = __builtin_amdgcn_readfirstlane(wave);
    auto tb_of = [&](int n) { return t_begin + (w0 + NW * (n % PER) + VW * (n / PER)) * ROWS; };
    Step cur, nxt;
    load(tb_of(0), cur);
    for (int n = 0; tb_of(n) < t_end; n += PER) {
      static_for_side<0, PER>([&](auto P) {
        constexpr int p = decltype(P)::value;
        load(tb_of(n + p + 1), nxt);  // past the end: zeros, no memory traffic
        if (tb_of(n + p) < t_end) compute(cur, acc[p]);
        cur = nxt;
      });
    }
#pragma unroll
    for (int p = 1; p < PER; ++p)
#pragma unroll
      for (int q = 0; q < VEC; ++q)
#pragma unroll
        for (int jb = 0; jb < JB; ++jb) acc[0][q][jb] += acc[p][q][jb];
  }

  // Pairwise tree over waves: in round h the upper half of the active waves
  // writes, the lower half adds (wave w receives wave w + h).
  // acc[0][q][jb] element i: local column (4g + i) * VEC + q, rank index 16 jb + cl.
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
          for (int i = 0; i < 4; ++i) slot[((4 * g + i) * VEC + q) * RS + jb * 16 + cl] = acc[0][q][jb][i];
    }
    __syncthreads();
    if (wave < h) {
      const float *slot = red + wave * COLS * RS;
#pragma unroll
      for (int q = 0; q < VEC; ++q)
#pragma unroll
        for (int jb = 0; jb < JB; ++jb)
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[0][q][jb][i] += slot[((4 * g + i) * VEC + q) * RS + jb * 16 + cl];
    }
  }
  // Wave 0 holds the tile (of the item, or of this part).
  const int jn = min(32, r - jg);
  if (wave == 0) {
    if (tparts > 1) {
      // A part: its tile to its slot, one 16-byte quad per accumulator
      // (quad (q, jb) of lane l at ((q * JB + jb) * 64 + l) * 4), by
      // device-scope stores (relaxed atomic stores carry the sc1 policy on
      // gfx950: written through to the point of coherence, no L2 write-back),
      // complete before the count.
      static_assert(VEC * JB * 4 * 64 <= SIDE_SLOT_FLOATS, "slot size");
      float *slot = s.part + (int64_t)unit * SIDE_SLOT_FLOATS;
#pragma unroll
      for (int q = 0; q < VEC; ++q)
#pragma unroll
        for (int jb = 0; jb < JB; ++jb)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            __hip_atomic_store(slot + ((q * JB + jb) * 64 + lane) * 4 + i, acc[0][q][jb][i], __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
      __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
      unsigned before = 0;
      if (lane == 0) before = __hip_atomic_fetch_add(s.cnt + gitem, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      before = __builtin_amdgcn_readfirstlane(before);
      if (before != (unsigned)(tparts - 1)) return;
      // The last part: every slot of the item is complete.  Its lines are in
      // no cache (see SideArgs), so ordinary loads, issued after the count
      // (the compiler barrier keeps them there), fetch the stored values.
      // A slot's sixteen 16-byte loads are all issued before its sums.
      asm volatile("" ::: "memory");
      const float *first = s.part + (int64_t)(unit - part) * SIDE_SLOT_FLOATS;
      for (int pp = 0; pp < tparts; ++pp) {
        const f32x4 *sl = (const f32x4 *)(first + (int64_t)pp * SIDE_SLOT_FLOATS);
        f32x4 v[VEC][JB];
#pragma unroll
        for (int q = 0; q < VEC; ++q)
#pragma unroll
          for (int jb = 0; jb < JB; ++jb) v[q][jb] = sl[(q * JB + jb) * 64 + lane];
#pragma unroll
        for (int q = 0; q < VEC; ++q)
#pragma unroll
          for (int jb = 0; jb < JB; ++jb) acc[0][q][jb] = pp == 0 ? v[q][jb] : acc[0][q][jb] + v[q][jb];
      }
    }
#pragma unroll
    for (int q = 0; q < VEC; ++q)
#pragma unroll
      for (int jb = 0; jb < JB; ++jb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int l = c0 + (4 * g + i) * VEC + q;
          const int j = jb * 16 + cl;
          if (l < jL && j < jn) {
            const float v = jscale * acc[0][q][jb][i];
            if (ji == 0)
              jout[(int64_t)(jg + j) * jL + l] = v;
            else
              jout[(int64_t)l * r + jg + j] = v;
          }
        }
  }
}

}  // namespace lora
