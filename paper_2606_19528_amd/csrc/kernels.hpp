// kernels.hpp -- shared device-side building blocks for the gfx950 kernels:
// element traits, 16-byte fragments and the matrix-core (MFMA) wrappers.
//
// Fragment convention (both element types): one lane holds 16 contiguous
// bytes of one operand row along the reduction index k.
//   32x32 tiles: a "k-slice" is 32 bytes of every row; lane l reads row
//                (l % 32) at byte offset (l / 32) * 16 of the slice.
//   16x16 tiles: a k-slice is 64 bytes; lane l reads row (l % 16) at byte
//                offset (l / 16) * 16.
// bf16: the 16 bytes are 8 consecutive k and feed one
//       v_mfma_f32_{32x32x16,16x16x32}_bf16.
// fp32: the 16 bytes are 4 consecutive k; element e of every lane feeds the
//       e-th of four v_mfma_f32_{32x32x2,16x16x4}_f32.  Operands A and B use
//       the same lane->k map, so the four products together cover the slice
//       exactly once (only the order of the additions differs).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lora {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

struct BF16 {
  typedef uint16_t T;             // storage: raw bf16 bits
  static constexpr int VEC = 8;   // elements per 16-byte vector
  static __device__ __forceinline__ T from_float(float f) {
    __bf16 h = (__bf16)f;         // round to nearest even (v_cvt_pk_bf16_f32)
    return __builtin_bit_cast(uint16_t, h);
  }
  static __device__ __forceinline__ float to_float(T v) {
    return __builtin_bit_cast(float, (uint32_t)v << 16);
  }
};

struct F32 {
  typedef float T;
  static constexpr int VEC = 4;
  static __device__ __forceinline__ T from_float(float f) { return f; }
  static __device__ __forceinline__ float to_float(T v) { return v; }
};

// acc(32x32) += A(32 x kslice) * B(kslice x 32); `a` holds the fragment of
// MFMA operand A (row = l % 32), `b` of operand B (column = l % 32).
__device__ __forceinline__ void mma32(BF16, f32x16 &acc, u32x4 a, u32x4 b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
}
// (The whole vector is bit-cast first: bit-casting a single element of an
// ext_vector_type value miscompiles to element 0 with this toolchain.)
__device__ __forceinline__ void mma32(F32, f32x16 &acc, u32x4 a, u32x4 b) {
  const f32x4 af = __builtin_bit_cast(f32x4, a), bf = __builtin_bit_cast(f32x4, b);
#pragma unroll
  for (int e = 0; e < 4; ++e) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(af[e], bf[e], acc, 0, 0, 0);
}

// acc(16x16) += A(16 x kslice) * B(kslice x 16).
__device__ __forceinline__ void mma16(BF16, f32x4 &acc, u32x4 a, u32x4 b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
}
__device__ __forceinline__ void mma16(F32, f32x4 &acc, u32x4 a, u32x4 b) {
  const f32x4 af = __builtin_bit_cast(f32x4, a), bf = __builtin_bit_cast(f32x4, b);
#pragma unroll
  for (int e = 0; e < 4; ++e) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(af[e], bf[e], acc, 0, 0, 0);
}

// Pack VEC floats into one 16-byte vector of element type E.
__device__ __forceinline__ u32x4 pack_vec(BF16, const float *f) {
  u32x4 r;
#pragma unroll
  for (int d = 0; d < 4; ++d)
    r[d] = (uint32_t)BF16::from_float(f[2 * d]) | ((uint32_t)BF16::from_float(f[2 * d + 1]) << 16);
  return r;
}
// Two floats to a bf16 pair (round to nearest even) in one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}
__device__ __forceinline__ u32x4 pack_vec(F32, const float *f) {
  u32x4 r;
#pragma unroll
  for (int d = 0; d < 4; ++d) r[d] = __builtin_bit_cast(uint32_t, f[d]);
  return r;
}

// Register transpose of a VEC x VEC block.  in[i] holds row i (VEC
// consecutive columns); out[c] receives column c (VEC consecutive rows).
__device__ __forceinline__ void transpose_block(BF16, const u32x4 *in, u32x4 *out) {
#pragma unroll
  for (int c = 0; c < 8; ++c) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      uint32_t lo = in[2 * p][c >> 1];
      uint32_t hi = in[2 * p + 1][c >> 1];
      out[c][p] = (c & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
    }
  }
}
__device__ __forceinline__ void transpose_block(F32, const u32x4 *in, u32x4 *out) {
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int p = 0; p < 4; ++p) out[c][p] = in[p][c];
}

typedef __attribute__((address_space(3))) void lds_void;

// One direct-to-LDS load: 16 bytes per lane from voffset + soffset of the
// resource into lds + 16 * lane (lds is the same for the whole wave; M0 holds
// it).  Written as assembly so that the compiler does not track these LDS
// writes: its own tracking makes some LDS reads wait for every such load in
// flight.  Every read of a stage is ordered after its loads by the explicit
// wait + barrier protocol of the main loop instead.  (No compiler-generated
// code of these kernels keeps a value in M0.)  The compiler does not look
// into the assembly for hazards, so it carries the one wait state the write
// of M0 needs before the load reads it.  The other hazard such a load has --
// five wait states after a vector instruction writes an SGPR the load reads
// (its resource or soffset) -- does not arise in these kernels: those
// operands come from scalar instructions, which the generated-code tests
// check for every load (a blanket s_nop 4 here cost 1-7 % of GEMM time).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t rs, char *lds, uint32_t voffset,
                                      int soffset) {
  const uint32_t base = (uint32_t)(uintptr_t)(lds_void *)lds;
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds" ::"s"(base),
               "v"(voffset),
               "s"(rs), "s"(soffset)
               : "memory", "m0");
}
// The 4-byte form: 4 bytes per lane into lds + 4 * lane.
__device__ __forceinline__ void dma4(__amdgpu_buffer_rsrc_t rs, char *lds, uint32_t voffset,
                                     int soffset) {
  const uint32_t base = (uint32_t)(uintptr_t)(lds_void *)lds;
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, %3 offen lds" ::"s"(base),
               "v"(voffset),
               "s"(rs), "s"(soffset)
               : "memory", "m0");
}
#pragma clang diagnostic pop

__device__ __forceinline__ u32x4 ld16(const void *p) { return *(const u32x4 *)p; }
__device__ __forceinline__ void st16(void *p, u32x4 v) { *(u32x4 *)p = v; }
__device__ __forceinline__ u32x4 zero16() { return u32x4{0u, 0u, 0u, 0u}; }

}  // namespace lora
