// rowprod.hpp -- one work item of the rank-r "row" product, shared by the
// standalone row-skinny kernel (skinny.hip) and the producer workgroups of a
// fused GEMM launch (gemm_kernel.hpp):
//   P_p[m][j] = sum_{k in segment p} X[m][k] V(j, k)
// for the 16 * MB rows of row block `bx` and reduction segment `by` (see
// RowArgs in launch.hpp).  The eight waves accumulate 16 x r tiles on 16x16
// matrix cores over their share of the segment, and the eight partial tiles
// are summed in LDS in a fixed order.  At r >= 16 vector FMAs would not keep
// up with HBM.
//
// bf16 with r <= 32 (row-major V, or k-major V with r a multiple of 8): both
// operands stream through LDS.  A stage is 256 k of the item's rows and of V;
// direct-to-LDS loads fill a ring of stages (512-byte row pieces, two rows per
// load; k-major V as its contiguous [256 k][r] block), and wave w reads k-slice
// w (32 k) of every stage.  Fetching the V fragments straight from global
// memory (16 rows x 64 bytes per load, the same lines for every workgroup)
// cost a third of the kernel's time; read from LDS they cost almost nothing.
// Other cases: eight waves take interleaved 128-byte chunks of the segment (up
// to four chunks in flight per wave) and load their fragments directly.
//
// k-major V (B in the backward pass): each wave copies the V rows of its chunk
// into a private LDS region and reads them back with ds_read_b64_tr_b16,
// which returns four consecutive k of one column per lane -- exactly the
// matrix-core operand -- instead of gathering 2-byte elements from global
// memory.
//
// Besides the fp32 partial sums the item writes the operand of the big GEMM's
// LoRA step, tail[m][p*r + j] = E(tail_mult * P_p), zero-padded to `ldt`
// columns, and its share of the optional copy job (the other LoRA factor
// repeated once per segment), shared out over a grid of gx * gy items.
#pragma once

#include "kernels.hpp"
#include "launch.hpp"

namespace lora {

typedef short rp_i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) rp_i16x4 rp_lds_i16x4;

constexpr int ROW_NW = 8;  // waves per workgroup

// Streamed through LDS (see above)?
template <class E, int JB, int VMODE>
constexpr bool row_streamed() {
  return sizeof(typename E::T) == 2 && JB <= 2 && (VMODE == V_ROW || VMODE == V_KMAJ_TR);
}
constexpr int ROW_KS = 256;  // k per stage of the streamed form
// Stage bytes and ring depth of the streamed form: 512-byte pieces of the 16 MB
// rows and of 16 JB rows of V (a k-major V block of 256 x r bf16 fits in them).
template <int JB, int MB>
constexpr int row_stage_bytes() { return (16 * MB + 16 * JB) * ROW_KS * 2; }
template <int JB, int MB>
constexpr int row_nbuf() { return row_stage_bytes<JB, MB>() <= 32768 ? 4 : 3; }

// LDS bytes of one item (NW waves).
template <class E, int JB, int VMODE, int U, int MB, int NW = ROW_NW>
constexpr int row_lds_bytes() {
  constexpr int CE = 128 / (int)sizeof(typename E::T);
  constexpr int REGION = U * CE * JB * 16 * 2;
  constexpr int RED = NW * 16 * MB * (JB * 16 + 1) * 4;
  if constexpr (row_streamed<E, JB, VMODE>()) {
    constexpr int RING = row_nbuf<JB, MB>() * row_stage_bytes<JB, MB>();
    return RING > RED ? RING : RED;
  }
  return (VMODE == V_KMAJ_TR && NW * REGION > RED) ? NW * REGION : RED;
}

// COH: the outputs (out, tail) are stored coherently at device scope (sc1):
// a consumer in another XCD reads them while the launch still runs.
// NW: waves of the workgroup, 8 or (streamed form only) 4; four waves take
// two k-slices of every stage each.
template <class E, int JB, int VMODE, int U, int MB, bool COH = false, int NW = ROW_NW>
__device__ __forceinline__ void row_item(const RowArgs &a, int bx, int by, int gx, int gy, char *smem) {
  constexpr int NT = 64 * NW;
  static_assert(NW == 8 || (NW == 4 && row_streamed<E, JB, VMODE>()), "eight waves, or four streaming");
  typedef typename E::T T;
  constexpr int VEC = E::VEC;
  constexpr int CE = 128 / (int)sizeof(T);  // elements per 128-byte chunk
  constexpr int R16 = JB * 16;
  constexpr int RSB = R16 * 2;              // LDS row of a staged B chunk (bf16)
  constexpr int REGION = U * CE * RSB;      // per-wave staging region
  constexpr int RM = 16 * MB;                // rows per workgroup

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int m0 = bx * RM;
  const int p = by;  // segment of the reduction axis
  const int row = m0 + (lane & 15);  // of row tile 0; tile mt adds 16 mt
  const int g = lane >> 4;
  const int M = a.M, r = a.r;
  const int k_lo = p * a.seg, k_hi = min(a.L, k_lo + a.seg);
  const T *Xp = (const T *)a.X;
  const T *Vp = (const T *)a.V;

  // Optional copy job (LoRA-step operands repeated once per segment).  In
  // 16-byte vectors when the repetition keeps whole vectors together: each
  // thread loads its first CPV vectors here and stores them after the main
  // work, so their latency hides behind the main loads instead of delaying
  // them; further vectors, and the element-wise form, are copied at the end.
  constexpr int CPV = 2;
  const T *csrc = (const T *)a.bcopy_src;
  T *cdst = (T *)a.bcopy_dst;
  const int64_t cg = ((int64_t)by * gx + bx) * NT + tid;
  const int64_t cstride = (int64_t)gx * gy * NT;
  const int crep = a.nsplit * r;
  const bool cvec = (a.bcopy_mode == BCOPY_COLS && r % VEC == 0 && a.ldt % VEC == 0) ||
                    (a.bcopy_mode == BCOPY_FLAT && a.bcopy_period % VEC == 0 && a.bcopy_elems % VEC == 0);
  const int64_t cnv = !cvec ? 0
                      : a.bcopy_mode == BCOPY_COLS ? (int64_t)a.bcopy_rows * (a.ldt / VEC)
                                                   : a.bcopy_elems / VEC;
  // vector v: destination element d, source element s (-1: zeros)
  auto cmap = [&](int64_t v, int64_t &d, int64_t &sidx) {
    if (a.bcopy_mode == BCOPY_COLS) {
      const int64_t n = v / (a.ldt / VEC);
      const int c0 = (int)(v % (a.ldt / VEC)) * VEC;
      d = n * a.ldt + c0;
      sidx = c0 < crep ? n * r + c0 % r : -1;
    } else {
      d = v * VEC;
      sidx = d % a.bcopy_period;
    }
  };
  u32x4 cval[CPV];
#pragma unroll
  for (int q = 0; q < CPV; ++q) {
    const int64_t v = cg + q * cstride;
    cval[q] = zero16();
    if (v < cnv) {
      int64_t d, si;
      cmap(v, d, si);
      if (si >= 0) cval[q] = ld16(csrc + si);
    }
  }

  f32x4 acc[MB][JB];
#pragma unroll
  for (int mt = 0; mt < MB; ++mt)
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) acc[mt][jb] = f32x4{0.f, 0.f, 0.f, 0.f};

  if constexpr (row_streamed<E, JB, VMODE>()) {
    // Stage layout: rows 0 .. 16 MB - 1 of the item, then V (row-major: 16 JB
    // rows; k-major: the [256][r] block), 512 bytes per row.  Row-major
    // pieces keep their 16-byte chunk c at c ^ (row & 15), so the fragment
    // reads of 16 rows at one k hit distinct banks.
    constexpr int KS = ROW_KS, PB = KS * 2;
    constexpr int XB = 16 * MB * PB;
    constexpr int STAGE = row_stage_bytes<JB, MB>(), NBUF = row_nbuf<JB, MB>();
    constexpr int F = ROW_NW / NW;     // k-slices per wave per stage
    constexpr int LPW = F * (MB + JB);  // loads per wave per stage
    constexpr uint32_t OOB = 0x80000000u;
    const int wv = __builtin_amdgcn_readfirstlane(wave);
    const int klen = k_hi - k_lo, nst = (klen + KS - 1) / KS;
    const int nrows = max(0, min(M - m0, 16 * MB));
    // (the values are uniform; readfirstlane keeps the resources in SGPRs)
    auto rsrc = [](const void *base, int64_t bytes) {
      const uint64_t b = (uint64_t)(uintptr_t)base;
      const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b);
      const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
      const int n = __builtin_amdgcn_readfirstlane((int)bytes);
      return __builtin_amdgcn_make_buffer_rsrc((void *)(uintptr_t)(((uint64_t)hi << 32) | lo), (short)0, n,
                                               0x00020000);
    };
    const __amdgpu_buffer_rsrc_t rsX = rsrc(Xp + (int64_t)m0 * a.ldx + k_lo, (int64_t)nrows * a.ldx * 2);
    const __amdgpu_buffer_rsrc_t rsV = VMODE == V_ROW ? rsrc(Vp + k_lo, (int64_t)r * a.ldv * 2)
                                                      : rsrc(Vp + (int64_t)k_lo * r, (int64_t)klen * r * 2);
    // Load q of this wave covers 1 KB piece ii = wv + NW q' of the stage's
    // rows (q < F MB, q' = q) or of V (after them, q' = q - F MB).  kq: k
    // (within a stage) of the lane's first element, or its k-row for k-major V.
    uint32_t offq[LPW];
    int kq[LPW];
#pragma unroll
    for (int q = 0; q < LPW; ++q) {
      const int ii = wv + NW * (q < F * MB ? q : q - F * MB);
      if (q < F * MB || VMODE == V_ROW) {
        const int rr = 2 * ii + (lane >> 5);
        const int c = (lane & 31) ^ (rr & 15);
        kq[q] = c * 8;
        offq[q] = (uint32_t)(rr * (q < F * MB ? a.ldx : a.ldv) * 2 + c * 16);
      } else {
        const int byte = ii * 1024 + lane * 16;
        kq[q] = byte / (2 * r) < KS ? byte / (2 * r) : KS + klen;  // past the block: never loaded
        offq[q] = (uint32_t)byte;
      }
    }
    auto issue = [&](int st) __attribute__((always_inline)) {
      char *buf = smem + (st % NBUF) * STAGE;
      const int k0 = st * KS;
#pragma unroll
      for (int q = 0; q < LPW; ++q) {
        const uint32_t vo = k0 + kq[q] < klen ? offq[q] : OOB;
        if (q < F * MB) dma16(rsX, buf + (wv + NW * q) * 1024, vo, k0 * 2);
        else dma16(rsV, buf + XB + (wv + NW * (q - F * MB)) * 1024, vo, VMODE == V_ROW ? k0 * 2 : k0 * r * 2);
      }
    };
#pragma unroll
    for (int st = 0; st < NBUF - 1; ++st) issue(st);
    for (int s = 0; s < nst; ++s) {
      constexpr int V = (NBUF - 2) * LPW;  // this wave's loads of stage s landed, LDS reads done
      __builtin_amdgcn_s_waitcnt((V & 15) | ((V >> 4) << 14) | (7 << 4));
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      issue(s + NBUF - 1);  // into the buffer of stage s - 1, which nobody reads any more
      const char *buf = smem + (s % NBUF) * STAGE;
#pragma unroll
      for (int h = 0; h < F; ++h) {
        const int w = wv + NW * h;                                // k-slice of the stage
        const int pos = (4 * w + (lane >> 4)) ^ (lane & 15);
        u32x4 xa[MB], vb[JB];
#pragma unroll
        for (int mt = 0; mt < MB; ++mt) xa[mt] = ld16(buf + (mt * 16 + (lane & 15)) * PB + pos * 16);
#pragma unroll
        for (int jb = 0; jb < JB; ++jb) {
          if constexpr (VMODE == V_ROW) {
            vb[jb] = ld16(buf + XB + (jb * 16 + (lane & 15)) * PB + pos * 16);
          } else {
            // four consecutive k of one column per lane (as in the other form)
            const int iq = lane & 15;
            const char *pp = buf + XB + (32 * w + 8 * g + (iq >> 2)) * (2 * r) + (jb * 16 + 4 * (iq & 3)) * 2;
            rp_i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((rp_lds_i16x4 *)pp);
            rp_i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((rp_lds_i16x4 *)(pp + 4 * (2 * r)));
            vb[jb] = u32x4{__builtin_bit_cast(uint2, lo).x, __builtin_bit_cast(uint2, lo).y,
                           __builtin_bit_cast(uint2, hi).x, __builtin_bit_cast(uint2, hi).y};
          }
        }
#pragma unroll
        for (int jb = 0; jb < JB; ++jb)
#pragma unroll
          for (int mt = 0; mt < MB; ++mt) mma16(E(), acc[mt][jb], xa[mt], vb[jb]);
      }
    }
    __builtin_amdgcn_s_waitcnt((7 << 4));  // the loads past the end (zeros) too
  } else {
  char *region = smem + wave * REGION;

  for (int kc0 = k_lo + wave * CE; kc0 < k_hi; kc0 += NW * CE * U) {
    u32x4 xf[U][MB][2];
    u32x4 vf[U][2][JB];
    // issue every global load of the U chunks first
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kc = kc0 + u * NW * CE;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int k = kc + h * 4 * VEC + g * VEC;
#pragma unroll
        for (int mt = 0; mt < MB; ++mt)
          xf[u][mt][h] = (row + 16 * mt < M && k < k_hi) ? ld16(Xp + (int64_t)(row + 16 * mt) * a.ldx + k)
                                                        : zero16();
        if constexpr (VMODE == V_ROW) {
#pragma unroll
          for (int jb = 0; jb < JB; ++jb) {
            const int j = jb * 16 + (lane & 15);
            vf[u][h][jb] = (j < r && k < k_hi) ? ld16(Vp + (int64_t)j * a.ldv + k) : zero16();
          }
        } else if constexpr (VMODE == V_KMAJ_GATHER) {
#pragma unroll
          for (int jb = 0; jb < JB; ++jb) {
            const int j = jb * 16 + (lane & 15);
            float f[VEC];
#pragma unroll
            for (int e = 0; e < VEC; ++e)
              f[e] = (j < r && k + e < k_hi) ? E::to_float(Vp[(int64_t)(k + e) * a.ldv + j]) : 0.0f;
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
          const u32x4 v = n < k_hi ? ld16(Vp + (int64_t)n * r + bc * 8) : zero16();
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
            rp_i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((rp_lds_i16x4 *)p);
            rp_i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((rp_lds_i16x4 *)(p + 4 * RSB));
            vf[u][h][jb] = u32x4{__builtin_bit_cast(uint2, lo).x, __builtin_bit_cast(uint2, lo).y,
                                 __builtin_bit_cast(uint2, hi).x, __builtin_bit_cast(uint2, hi).y};
          }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int jb = 0; jb < JB; ++jb)
#pragma unroll
          for (int mt = 0; mt < MB; ++mt) mma16(E(), acc[mt][jb], xf[u][mt][h], vf[u][h][jb]);
  }
  }

  // D[m][n]: m = 4 (lane / 16) + i, n = lane % 16.  Sum the waves' tiles.
  __syncthreads();
  float *red = (float *)smem;
#pragma unroll
  for (int mt = 0; mt < MB; ++mt)
#pragma unroll
    for (int jb = 0; jb < JB; ++jb)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        red[(wave * RM + mt * 16 + g * 4 + i) * (R16 + 1) + jb * 16 + (lane & 15)] = acc[mt][jb][i];
  __syncthreads();
  // Segment p owns columns p*r .. p*r + r-1 of the tail; the last segment
  // also writes its zero padding.
  T *tail = (T *)a.tail;
  float *out = a.out + (int64_t)p * a.out_stride;
  const int pad_lo = a.nsplit * r;
  const int ncol = (tail && p == a.nsplit - 1) ? r + (a.ldt - pad_lo) : r;
  for (int idx = tid; idx < RM * ncol; idx += NT) {
    const int mm = idx / ncol, c = idx % ncol;
    if (m0 + mm >= M) continue;
    auto put = [&](auto *dst, auto v) {
      if constexpr (COH) __hip_atomic_store(dst, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      else *dst = v;
    };
    if (c < r) {
      float s = red[(0 * RM + mm) * (R16 + 1) + c];
#pragma unroll
      for (int w = 1; w < NW; ++w) s += red[(w * RM + mm) * (R16 + 1) + c];
      put(out + (int64_t)(m0 + mm) * r + c, a.out_mult * s);
      if (tail) put(tail + (int64_t)(m0 + mm) * a.ldt + p * r + c, E::from_float(a.tail_mult * s));
    } else {
      put(tail + (int64_t)(m0 + mm) * a.ldt + pad_lo + (c - r), (T)0);
    }
  }
  // the copy job: held vectors, then the rest
#pragma unroll
  for (int q = 0; q < CPV; ++q) {
    const int64_t v = cg + q * cstride;
    if (v < cnv) {
      int64_t d, si;
      cmap(v, d, si);
      st16(cdst + d, cval[q]);
    }
  }
  for (int64_t v = cg + CPV * cstride; v < cnv; v += cstride) {
    int64_t d, si;
    cmap(v, d, si);
    st16(cdst + d, si >= 0 ? ld16(csrc + si) : zero16());
  }
  if (a.bcopy_mode != BCOPY_NONE && !cvec) {
    if (a.bcopy_mode == BCOPY_COLS) {
      const int64_t total = (int64_t)a.bcopy_rows * a.ldt;
      for (int64_t i = cg; i < total; i += cstride) {
        const int64_t n = i / a.ldt;
        const int c = (int)(i % a.ldt);
        cdst[i] = c < crep ? csrc[n * r + c % r] : (T)0;
      }
    } else {
      for (int64_t i = cg; i < a.bcopy_elems; i += cstride) cdst[i] = csrc[i % a.bcopy_period];
    }
  }
}

}  // namespace lora
