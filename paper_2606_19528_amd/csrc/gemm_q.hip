// gemm_q.hip -- launches of the quantized-B GEMM instances (the frozen W as
// codes plus per-group scale and offset, dequantized on chip): the
// direct-to-LDS dequantizing tiles, and the register-staged form for groups
// below 64 weights.  The kernel template is in gemm_kernel.hpp.
#include "gemm_kernel.hpp"

namespace lora {

// Dequantizing direct-to-LDS tiles (the shapes of the bf16 path; 256 x 128
// and 128 x 64 choices run 128 x 128 tiles).
template <int QB>
static hipError_t launch_q_dma(const GemmArgs &g, int shape, bool kmaj, const SideArgs *side, hipStream_t st) {
  if (kmaj) {
    switch (shape) {
      case 2:
        return launch_cfg<BF16, 256, 256, 2, 2, 1, B_KMAJ_TR, 64, 3, 3, 2, QB, EPI_STORE, 1>(g, side, st);
      case 4:
        return launch_cfg<BF16, 256, 192, 2, 2, 1, B_KMAJ_TR, 64, 3, 3, 2, QB, EPI_STORE, 1>(g, side, st);
      default:
        return launch_cfg<BF16, 128, 128, 2, 2, 2, B_KMAJ_TR, 128, 3, 3, 2, QB, EPI_STORE, 1>(g, side, st);
    }
  }
  switch (shape) {
    case 2:
      return launch_cfg<BF16, 256, 256, 2, 2, 1, B_ROW, 64, 3, 3, 2, QB, EPI_STORE, 1>(g, side, st);
    case 4:
      return launch_cfg<BF16, 256, 192, 2, 2, 1, B_ROW, 64, 3, 3, 2, QB, EPI_STORE, 1>(g, side, st);
    default:
      return launch_cfg<BF16, 128, 128, 2, 2, 2, B_ROW, 128, 3, 3, 2, QB, EPI_STORE, 1>(g, side, st);
  }
}

bool gemm_q_direct(const GemmArgs &g, int bits, bool b_kmajor, bool with_side) {
  // Groups of at least 64 weights (a row-major stage then holds one group per
  // row), the LoRA stages within the first three, and the scales (and, for
  // k-major B, the codes of all K rows) within 32-bit offsets.
  const int shape = pick_shape(g.M, g.N, b_kmajor, with_side);
  const int bke = shape == 2 || shape == 4 ? 32 : 64;
  const int64_t rowbytes = g.ldb * bits / 8, ldg = g.ldb >> g.qlog2g;
  const int64_t wrows = b_kmajor ? g.K : g.N;
  return (bits == 4 || bits == 8) && g.qlog2g >= 6 && g.r <= 3 * bke && wrows * ldg * 4 < (int64_t(1) << 31) &&
         (!b_kmajor || (int64_t)g.K * rowbytes < (int64_t(1) << 31));
}

hipError_t launch_gemm_q(const GemmArgs &g, int bits, bool b_kmajor, const SideArgs *side,
                         hipStream_t st) {
  if (gemm_q_direct(g, bits, b_kmajor, side != nullptr)) {
    const int shape = pick_shape(g.M, g.N, b_kmajor, side != nullptr);
    return bits == 4 ? launch_q_dma<4>(g, shape, b_kmajor, side, st) : launch_q_dma<8>(g, shape, b_kmajor, side, st);
  }
  if (bits == 4)
    return b_kmajor ? launch_cfg<BF16, 128, 128, 2, 2, 2, B_KMAJ_TR, 128, 2, 3, 2, 4>(g, side, st)
                    : launch_cfg<BF16, 128, 128, 2, 2, 2, B_ROW, 128, 2, 3, 2, 4>(g, side, st);
  if (bits == 8)
    return b_kmajor ? launch_cfg<BF16, 128, 128, 2, 2, 2, B_KMAJ_TR, 128, 2, 3, 2, 8>(g, side, st)
                    : launch_cfg<BF16, 128, 128, 2, 2, 2, B_ROW, 128, 2, 3, 2, 8>(g, side, st);
  return hipErrorInvalidValue;
}

}  // namespace lora
