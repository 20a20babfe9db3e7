// gemm.hip -- launches of the bf16 / fp32 GEMM instances (the kernel template
// and its launcher are in gemm_kernel.hpp; the quantized-B instances in
// gemm_q.hip): plain, fused with rank-r producers, and with epilogues.
#include <algorithm>

#include "gemm_kernel.hpp"

namespace lora {

int side_workgroups(SideArgs *s, Dtype dt) {
  const int cols = dt == DT_BF16 ? SideShape<BF16>::COLS : SideShape<F32>::COLS;
  int n = 0;
  for (int i = 0; i < s->njobs; ++i) {
    n += (s->job[i].L + cols - 1) / cols * ((s->r + 31) / 32);
    if (i == 0) s->n0 = n;
  }
  if (s->tparts < 1) s->tparts = 1;
  if (s->tparts == 1) s->tchunk = s->T;
  s->ntot = n * s->tparts;
  return (s->ntot + 7) / 8 * 8;
}

int side_item_count(int64_t d_in, int64_t d_out, int64_t r, Dtype dt) {
  const int64_t cols = dt == DT_BF16 ? SideShape<BF16>::COLS : SideShape<F32>::COLS;
  return (int)(((d_in + cols - 1) / cols + (d_out + cols - 1) / cols) * ((r + 31) / 32));
}

// An item over all T draws 40 - 55 GB/s (one workgroup per CU): at T = 4096
// (1.5 MB of x or dy and of du or u) it outlasts the tiles it runs beside in
// the dx launches of a 3072 -> 1024 linear (192 tiles of 256 x 256 over a
// reduction of 1024).  Where the tiles leave CUs idle, the items' parts take
// them.  Where the tiles fill the CUs, the items delay as many tiles by
// their own duration; parts of at least 2048 tokens (T >= 4096), one round
// of them, shorten that delay (8192 -> 3072 at T = 4096: 88 items as 176
// parts, 0.34 ms less per 28-layer step), while shorter parts were measured
// not to shrink with their token count (512-token parts of a 2048-token item
// took 10 - 17 us against 19.5 us for the whole item; about 5 us of it is a
// part's fixed cost: load ramp, LDS tree).
void side_split(int64_t T, int64_t d_in, int64_t d_out, int64_t r, Dtype dt, int *tparts, int *tchunk) {
  constexpr int64_t STEP = 8 * SideShape<BF16>::ROWS;  // one step of each virtual wave
  *tparts = 1;
  *tchunk = (int)T;
  if (dt != DT_BF16) return;
  int bm = 0, bn = 0;
  gemm_tile_shape((int)T, (int)d_in, true, true, dt, &bm, &bn);
  const int64_t tiles = ((T + bm - 1) / bm) * ((d_in + bn - 1) / bn);
  const int64_t items = side_item_count(d_in, d_out, r, dt);
  if (items < 1 || (tiles >= 256 && T < 4096)) return;
  int64_t p = tiles >= 256 ? std::min<int64_t>({8, T / STEP, 256 / items})
                           : std::min<int64_t>({4, T / STEP, (256 - tiles) / items});
  // The part tiles stay within an eighth of the fp32 dW the method never forms.
  while (p > 1 && items * p * SIDE_SLOT_FLOATS * 4 > d_in * d_out / 2) --p;
  if (p <= 1) return;
  const int64_t chunk = ((T + p - 1) / p + STEP - 1) / STEP * STEP;
  *tparts = (int)((T + chunk - 1) / chunk);
  *tchunk = (int)chunk;
}

void gemm_tile_shape(int M, int N, bool b_kmajor, bool with_side, Dtype dt, int *bm, int *bn) {
  static const int shp[5][2] = {{128, 128}, {256, 128}, {256, 256}, {128, 64}, {256, 192}};
  const int c = dt == DT_BF16 ? pick_shape(M, N, b_kmajor, with_side) : 0;
  *bm = shp[c][0];
  *bn = shp[c][1];
}

hipError_t launch_gemm_epi(const GemmArgs &g, int epi, hipStream_t st) {
  switch (epi) {
    case EPI_CE_STATS:
      return launch_cfg<BF16, 128, 128, 2, 2, 2, B_ROW, 128, 3, 3, 2, 0, EPI_CE_STATS, 1>(g, nullptr, st);
    case EPI_CE_DZ:
      return launch_cfg<BF16, 128, 128, 2, 2, 2, B_ROW, 128, 3, 3, 2, 0, EPI_CE_DZ, 1>(g, nullptr, st);
    case EPI_F32:
      return launch_cfg<BF16, 128, 128, 2, 2, 2, B_KMAJ_TR, 128, 4, 3, 2, 0, EPI_F32, 1>(g, nullptr, st);
    case EPI_TOPK:
      return launch_cfg<BF16, 128, 128, 2, 2, 2, B_ROW, 128, 3, 3, 2, 0, EPI_TOPK, 1>(g, nullptr, st);
  }
  return hipErrorInvalidValue;
}

// Producers only pay off on CUs the tiles leave idle: fused when the tile
// shape is direct-to-LDS and 32-row producers fit beside the tiles; beside
// the backward's 256 x 256 tiles (e.g. 64 producers of 64 rows beside 192
// tiles at 4096 rows) only over reductions of 2048 or more, where the tiles
// outlast the producers and the side items that follow them on the same
// CUs (over 1024 the fused launch measured 59 us against 47 + 6 us for the
// two launches, over 3072 78 against 74 + 10, over 8192 188 against 183 + 19).
bool gemm_fusable(int M, int N, int K, bool b_kmajor) {
  const int cfg = pick_shape(M, N, b_kmajor, b_kmajor);
  if (cfg == 4 || (cfg == 2 && !b_kmajor)) return false;
  if (cfg == 2) {  // the backward's 256 x 256 tiles, with producers of up to 64 rows
    const long tiles = (long)((M + 255) / 256) * ((N + 255) / 256);
    return K >= 2048 && tiles + ((M + 63) / 64 + 7) / 8 * 8 <= 256;
  }
  const long bm = cfg == 1 ? 256 : 128, bn = cfg == 3 ? 64 : 128;
  const long tiles = ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
  return tiles + ((M + 31) / 32 + 7) / 8 * 8 <= 256;
}

hipError_t launch_gemm_fused(const GemmArgs &g, FuseArgs *fz, const SideArgs *side, hipStream_t st) {
  const bool kmaj = fz && fz->row.vmode == V_KMAJ_TR;
  if (!fz || fz->nprod <= 0 || (fz->row.vmode != V_ROW && !kmaj) || fz->row.nsplit != 1 || fz->row.r < 1 ||
      fz->row.r > 32 || (kmaj && fz->row.r % 8) || g.r < 1 || g.M < 1 || !fz->sync || fz->gen == 0 ||
      (side && !kmaj))
    return hipErrorInvalidValue;
  if (kmaj) {
    switch (pick_shape(g.M, g.N, true, true)) {
      case 2:
        return launch_cfg<BF16, 256, 256, 2, 2, 1, B_KMAJ_TR, 64, 3, 3, 2, 0, EPI_STORE, 2>(g, side, st, fz);
      case 1:
        return launch_cfg<BF16, 256, 128, 4, 2, 1, B_KMAJ_TR, 128, 3, 3, 2, 0, EPI_STORE, 2>(g, side, st, fz);
      case 0:
        return launch_cfg<BF16, 128, 128, 2, 2, 2, B_KMAJ_TR, 128, 4, 3, 2, 0, EPI_STORE, 2>(g, side, st, fz);
      case 3:
        return launch_cfg<BF16, 128, 64, 2, 2, 2, B_KMAJ_TR, 128, 4, 3, 2, 0, EPI_STORE, 2>(g, side, st, fz);
    }
    return hipErrorInvalidValue;
  }
  switch (pick_shape(g.M, g.N, false, false)) {
    case 1:
      return launch_cfg<BF16, 256, 128, 4, 2, 1, B_ROW, 128, 3, 3, 2, 0, EPI_STORE, 2>(g, nullptr, st, fz);
    case 0:
      return launch_cfg<BF16, 128, 128, 2, 2, 2, B_ROW, 128, 3, 3, 2, 0, EPI_STORE, 2>(g, nullptr, st, fz);
    case 3:
      return launch_cfg<BF16, 128, 64, 2, 2, 2, B_ROW, 128, 3, 3, 2, 0, EPI_STORE, 2>(g, nullptr, st, fz);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gemm(const GemmArgs &g, Dtype dt, bool b_kmajor, const SideArgs *side,
                       hipStream_t st) {
  if (dt == DT_BF16) {
    switch (pick_shape(g.M, g.N, b_kmajor, side != nullptr)) {
      case 2:
        return b_kmajor ? launch_cfg<BF16, 256, 256, 2, 2, 1, B_KMAJ_TR, 64, 3, 3, 2, 0, EPI_STORE, 1>(g, side, st)
                        : launch_cfg<BF16, 256, 256, 2, 2, 1, B_ROW, 64, 4, 3, 2, 0, EPI_STORE, 1>(g, side, st);
      case 4:
        return b_kmajor ? launch_cfg<BF16, 256, 192, 2, 2, 1, B_KMAJ_TR, 64, 3, 3, 2, 0, EPI_STORE, 1>(g, side, st)
                        : launch_cfg<BF16, 256, 192, 2, 2, 1, B_ROW, 64, 4, 3, 2, 0, EPI_STORE, 1>(g, side, st);
      case 1:
        return b_kmajor ? launch_cfg<BF16, 256, 128, 4, 2, 1, B_KMAJ_TR, 128, 3, 3, 2, 0, EPI_STORE, 1>(g, side, st)
                        : launch_cfg<BF16, 256, 128, 4, 2, 1, B_ROW, 128, 3, 3, 2, 0, EPI_STORE, 1>(g, side, st);
      case 3:
        return b_kmajor ? launch_cfg<BF16, 128, 64, 2, 2, 2, B_KMAJ_TR, 128, 4, 3, 2, 0, EPI_STORE, 1>(g, side, st)
                        : launch_cfg<BF16, 128, 64, 2, 2, 2, B_ROW, 128, 3, 3, 2, 0, EPI_STORE, 1>(g, side, st);
      default:
        return b_kmajor ? launch_cfg<BF16, 128, 128, 2, 2, 2, B_KMAJ_TR, 128, 4, 3, 2, 0, EPI_STORE, 1>(g, side, st)
                        : launch_cfg<BF16, 128, 128, 2, 2, 2, B_ROW, 128, 3, 3, 2, 0, EPI_STORE, 1>(g, side, st);
    }
  }
  return b_kmajor ? launch_cfg<F32, 128, 128, 2, 4, 1, B_KMAJ_REG, 128, 2, 2, 0>(g, side, st)
                  : launch_cfg<F32, 128, 128, 2, 4, 1, B_ROW, 128, 2, 2, 0>(g, side, st);
}

hipError_t handover_giveups(unsigned *count, bool reset) {
  hipError_t e = hipMemcpyFromSymbol(count, HIP_SYMBOL(g_fz_giveups), sizeof(unsigned), 0,
                                     hipMemcpyDeviceToHost);
  if (e != hipSuccess || !reset) return e;
  const unsigned zero = 0;
  return hipMemcpyToSymbol(HIP_SYMBOL(g_fz_giveups), &zero, sizeof(unsigned), 0, hipMemcpyHostToDevice);
}

}  // namespace lora
