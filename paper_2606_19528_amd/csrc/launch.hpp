// launch.hpp -- host-side interface between the C ABI (api.cpp) and the
// kernel translation units.  Internal to the library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lora {

enum Dtype { DT_BF16 = 0, DT_F32 = 1 };

// Sets the text lora_last_error() returns to the calling thread.
void set_last_error(const char *msg);

// Side work run by extra workgroups of the backward GEMM launch (they
// overlap with the dx tiles): token-reduced products
//   job 0: dA = du^T x   out [r, L] (transposed store), scale 1
//   job 1: dB = s dy^T u out [L, r],                    scale s (scale1)
// out[l][j] = scale * sum_t X[t*L + l] * V[t*r + j], t < T (X has rows of
// L elements).  V may be given as `vparts` partial sums V_p = V + p * vstride
// (p < vparts), added in ascending p when loaded.  (Kept small: these
// arguments share the kernel's scalar registers with the tiles.)
// An item (column block, rank group) may run as `tparts` parts over
// consecutive ranges of `tchunk` tokens (unfused launches only).  A part
// stores its tile in its slot of `part` (SIDE_SLOT_FLOATS floats) with
// device-scope stores, waits until they have completed, and counts itself in
// cnt[item] (zero before the launch); the part that counts last reads the
// item's slots with ordinary loads, adds them in ascending part order and
// stores the result.  Why ordinary loads see the other parts' stores: as for
// the hand-over of FuseArgs below -- no cache holds a slot line from an
// earlier launch, each part owns whole lines, and no wave reads a slot
// before the count shows that every part's stores have completed.
// tparts = 1: each item over all T, no slots.
struct ColJob {
  const void *X;
  const float *V;
  float *out;
  int L;
  int vparts;
};
struct SideArgs {
  ColJob job[2];
  int njobs;
  int T, r;
  float scale1;
  int64_t vstride;
  int n0, ntot;  // work items of job 0, and parts of both jobs' items (set by the GEMM launcher)
  int tparts, tchunk;
  float *part;
  unsigned *cnt;
};
constexpr int SIDE_SLOT_FLOATS = 4096;  // a part's tile: 64 values per lane of one wave
// Side items of a backward with reduction lengths d_in (dA) and d_out (dB).
int side_item_count(int64_t d_in, int64_t d_out, int64_t r, Dtype dt);
// Token parts per side item of the unfused dx launch, and tokens per part:
// more than one where the launch's tiles leave CUs idle (fewer than 256
// tiles) and the parts fit on them, or, from 4096 tokens, one round of parts
// ahead of tiles that fill the CUs (bf16; fp32: one part).
void side_split(int64_t T, int64_t d_in, int64_t d_out, int64_t r, Dtype dt, int *tparts, int *tchunk);

// C[M, N] = sum_k Aop[m][k] Bop[n][k]  (+ LoRA step), rounded to the element type.
//   Aop[m][k] = A[m*lda + k]                         m < M, k < K
//   Bop[n][k] = B[n*ldb + k]   (b_kmajor = false)    n < N
//             = B[k*ldb + n]   (b_kmajor = true)
// LoRA step (r > 0), extra reduction over j < r appended to k, both operands
// already in the element type:
//   Aop2[m][j] = A2[m*lda2 + j]
//   Bop2[n][j] = B2[n*ldb2 + j] (b_kmajor = false)  or  B2[j*ldb2 + n] (true)
// Optional (usum_out != NULL): the workgroups also write
// usum_out[m][j] = sum_{p < usum_parts} usum_src[p][m][j] (ascending p) for
// m < M, j < usum_r -- the sum of a rank-r product computed in partial sums
// (usum_parts <= MAX_SPLIT; row-major B only).
struct GemmArgs {
  const void *A;
  int64_t lda;
  const void *B;
  int64_t ldb;
  int M, N, K;
  const void *A2;
  int64_t lda2;
  const void *B2;
  int64_t ldb2;
  int r;
  void *C;
  int64_t ldc;
  const float *usum_src;
  float *usum_out;
  int usum_parts, usum_r;
  // Quantized B (launch_gemm_q): B holds unsigned codes of W ([rows][ldb]
  // weights, bits/8 bytes each, two 4-bit codes per byte with the even weight
  // in the low nibble), w = qscale * code + qoffset with one scale and offset
  // per group of 2^qlog2g consecutive weights of a W row, group-major:
  // [ldb >> qlog2g][rows] (the scales of one group for consecutive rows are
  // contiguous).
  const float *qscale;
  const float *qoffset;
  int qlog2g;
  // Cross-entropy epilogues (launch_gemm_epi); this GEMM's output column n is
  // column col0 + n of the reduced vocabulary, tpos[m] the target's column.
  const int32_t *tpos;
  int col0;
  float *ce_max, *ce_sum, *ce_tgt;  // EPI_CE_STATS: [tiles_n][M], [tiles_n][M], [M]
  const float *lse;                 // EPI_CE_DZ
  float dscale;
  int c_accumulate;                 // EPI_F32: C fp32 += product instead of =
  // EPI_TOPK: cosine = z * rn_a[m] * rn_b[n]; appended (value, col0 + n) to
  // row m's list (tk_val / tk_idx, tk_cap slots, count tk_cnt[m]) when above
  // tk_thr[m].
  const float *rn_a, *rn_b;
  const float *tk_thr;
  int *tk_cnt;
  float *tk_val;
  int32_t *tk_idx;
  int tk_cap;
};

// Epilogues of launch_gemm_epi (bf16 operands, 128 x 128 tiles):
//   EPI_CE_STATS  no C; per row and 128-column tile t of logits z:
//                 ce_max[t][m] = max_n z, ce_sum[t][m] = sum_n exp(z - max),
//                 ce_tgt[m] = z at the target column (B row-major);
//   EPI_CE_DZ     C bf16 [M][ldc] = dscale (exp(z - lse[m]) - [n is the
//                 target]) for n < N, 0 for N <= n < ldc (B row-major);
//   EPI_F32       C fp32 [M][ldc] (+)= A B (B k-major);
//   EPI_TOPK      no C; candidates of the similarity table (B row-major).
enum { EPI_STORE = 0, EPI_CE_STATS = 1, EPI_CE_DZ = 2, EPI_F32 = 3, EPI_TOPK = 4 };
hipError_t launch_gemm_epi(const GemmArgs &g, int epi, hipStream_t st);

// Reduced vocabulary: J = sorted union over i < nrows of
// table[targets[rows[i]]][0 .. k-1]; pos_of[v] = position of v in J;
// tpos[i] = position of targets[rows[i]]; count[0] = |J| (device).
// mark: V words of scratch.  Indices outside their range (rows[i] not in
// [0, T), a target or table entry not in [0, V)) are skipped (tpos -1).
struct HeadVocabArgs {
  const int32_t *table;
  int64_t ldtab;
  int k, V, T;
  const int32_t *targets, *rows;
  int nrows;
  uint32_t *mark;
  int32_t *J, *pos_of, *tpos, *count;
};
hipError_t launch_vocab_build(const HeadVocabArgs &a, hipStream_t st);
// dst[i] = src[idx[i]] (bf16 rows of `cols`, a multiple of 8), i < n; zero
// rows for indices outside [0, nsrc).
hipError_t launch_gather_rows(const void *src, int64_t ld, int nsrc, const int32_t *idx, int n,
                              int cols, void *dst, hipStream_t st);
// lse / loss per row from the EPI_CE_STATS partials; total = sum of losses
// (if not NULL), all in a fixed order.
hipError_t launch_ce_combine(const float *tmax, const float *tsum, int ntiles, int M,
                             const float *ztgt, float *lse, float *loss, float *total,
                             hipStream_t st);
// Top-k similarity table: per-row candidate lists of a batch of rows.
// Candidate slots per row of the selection: a list holds TOPK_SLOTS - p2(k)
// entries rounded down to a multiple of 4, p2(k) the power of two at or
// above k (at least k + 4096 for every k <= 2048).
constexpr int TOPK_SLOTS = 8192;
struct TopkArgs {
  float *val;
  int32_t *idx;
  int *cnt;
  float *thr;
  int cap, k;
  int lazy;        // a non-final pass selects only rows with more candidates
                   // than this (the list then still has room for a chunk)
  int32_t *table;  // [V][k], rows row0 .. row0 + R - 1 written by the final select
  float *tvals;    // optional [V][k]
  int64_t row0;
};
hipError_t launch_row_rnorm(const void *W, int V, int D, float *rn, hipStream_t st);
hipError_t launch_topk_reset(float *thr, int *cnt, int R, hipStream_t st);
// keep each of the R rows' k best candidates (final = 0) or sort them into
// the table (final = 1); cap <= 8192, k <= 2048.
hipError_t launch_topk_select(const TopkArgs &a, int R, int final, hipStream_t st);

// p[0 .. n) = quiet NaN.
hipError_t launch_fill_nan(float *p, int64_t n, hipStream_t st);
// dh [T][D] bf16: row rows[i] = acc[i], every other row 0 (inv: T words scratch).
hipError_t launch_dh_finish(const float *acc, const int32_t *rows, int nrows, int32_t *inv, int T,
                            int D, void *dh, hipStream_t st);

// GEMM launch; `side` (may be NULL) adds the token-reduction workgroups.
hipError_t launch_gemm(const GemmArgs &g, Dtype dt, bool b_kmajor, const SideArgs *side,
                       hipStream_t st);
// bf16 GEMM whose B is the quantized frozen weight (bits = 4 or 8), dequantized
// into LDS; the LoRA step (r <= 64) runs first.
// Whether launch_gemm_q runs the dequantizing direct-to-LDS tiles for g.
bool gemm_q_direct(const GemmArgs &g, int bits, bool b_kmajor, bool with_side);
hipError_t launch_gemm_q(const GemmArgs &g, int bits, bool b_kmajor, const SideArgs *side,
                         hipStream_t st);

// Output tile (BM x BN) that launch_gemm / launch_gemm_fused run for an
// M x N product with this B layout, with or without side items.
void gemm_tile_shape(int M, int N, bool b_kmajor, bool with_side, Dtype dt, int *bm, int *bn);

// Counts the work items of `side` into s->n0 and their parts into s->ntot,
// and returns the number of side workgroups they need (a multiple of 8).
int side_workgroups(SideArgs *s, Dtype dt);

enum { V_ROW = 0, V_KMAJ_TR = 1, V_KMAJ_GATHER = 2 };
enum { BCOPY_NONE = 0, BCOPY_COLS = 1, BCOPY_FLAT = 2 };
// Row-skinny product, split over the reduction axis into `nsplit` segments of
// `seg` elements (seg a multiple of one 128-byte chunk of elements):
//   P_p[m][j] = sum_{k in segment p} X[m*ldx + k] * V(j, k),
//   V(j, k) = V[j*ldv + k] (V_ROW) or V[k*ldv + j] (k-major, ldv = r).
// Writes out[p * out_stride + m*r + j] = out_mult * P_p[m][j] and, if tail is
// set, tail[m][p*r + j] = E(tail_mult * P_p[m][j]), columns nsplit*r .. ldt-1
// zero.  Optional copy job:
//   BCOPY_COLS  dst[n][c] = src[n*r + c % r] for c < nsplit*r, 0 up to ldt,
//               n < bcopy_rows (B repeated once per segment, zero-padded);
//   BCOPY_FLAT  dst[i] = src[i % bcopy_period] for i < bcopy_elems.
struct RowArgs {
  const void *X;
  int64_t ldx;
  int M, L;
  const void *V;
  int64_t ldv;
  int vmode;
  int r;
  int nsplit, seg;
  float out_mult;
  float *out;
  int64_t out_stride;
  void *tail;
  int ldt;
  float tail_mult;
  int bcopy_mode;
  const void *bcopy_src;
  void *bcopy_dst;
  int bcopy_rows;
  int64_t bcopy_period, bcopy_elems;
  int mb;  // row tiles of 16 per workgroup: 1 (0), 2 or 4 (bf16, r <= 32)
  unsigned *zero;  // row_skinny only: workgroup (0, 0) also sets zero[0 .. nzero) to 0
  int nzero;
};
hipError_t launch_row_skinny(const RowArgs &a, Dtype dt, hipStream_t st);

// Fused rank-r pass: the first `nwg` workgroups of the GEMM launch (a
// multiple of 8, so the tiles keep their XCD mapping) are producers, one per
// 16 * row.mb rows, that compute the rank-r product over the whole reduction
// axis (row: nsplit = 1) -- forward: u = x A^T (V_ROW) and the LoRA-step
// operand E(s u); backward: du = s dy B (V_KMAJ_TR) and E(du) -- ahead of the
// tiles, which need them only in their last (LoRA) step.  In the backward the
// producers then run the dA / dB side items: each waits, after counting
// itself, until every producer has counted (dA = du^T x needs all of du).
// They hand over through two 8-byte words of the workspace (8-byte aligned;
// nothing else may use them during the launch):
//   sync[0] = (gen << 32) | producers counted, sync[1] = tiles that passed.
// Workgroup 0 arms the launch before its work (sync[0] = gen << 32, then,
// released after it, sync[1] = 0).  A producer stores its rows with
// device-scope atomic stores (relaxed; on gfx950 they carry the sc1 policy
// and write through to the point of coherence, with no L2 write-back that
// would stall the tiles of its XCD), waits until every wave's stores have
// completed (vmcnt 0), and counts itself in sync[0] once it sees the launch
// armed: sync[1] == 0, then the tag in sync[0].  A tile, in the step that
// issues its LoRA stage, waits until sync[1] < ncons and sync[0] holds the
// tag and all producers, reads the producers' rows with ordinary loads, and
// counts itself in sync[1] after its main loop.
// Why ordinary loads see the producers' stores without an acquire fence: a
// fence would make the reads fetch past any cache line older than the
// stores, and no such line can exist -- the caches hold no line of the
// workspace from an earlier launch (a kernel boundary writes back and
// invalidates the L1s and the per-XCD L2s), each producer owns whole
// 128-byte lines of the rows (16 or 32 rows of r >= 8 fp32, or of 64 bf16),
// and no wave of the launch reads any of those lines before its wait has
// seen every producer's count, i.e. after every producer's stores completed
// at the point of coherence.  The first read of such a line therefore
// misses in the reader's L1 and L2 and fetches the stored bytes.  (Measured
// at T = 1024: the tiles' device-scope acquire cost 10 us per fused launch,
// sc1 loads of the LoRA stage made the 256 x 128 tiles spill registers.)
// The side items on the producers read du after an invalidate of that
// kind, which costs them nothing measurable.
// A stale state left by an earlier launch with the same tag (a replayed
// graph) has sync[1] == ncons, so it never passes for armed; a workspace
// with arbitrary contents holds the tag only by a 2^-32 chance.
// Every wait gives up after 0.2 s (the 100 MHz real-time counter), so no
// launch can hang on a broken hand-over; each wave whose wait gave up adds
// one to a per-device counter once its work is done (handover_giveups),
// which callers and tests check, because that launch may have computed with
// incomplete producer rows.
struct FuseArgs {
  RowArgs row;
  int nprod;                 // producers (row blocks); 0: no fusion
  int nwg;                   // workgroups reserved for them
  unsigned long long *sync;  // sync[0], sync[1]
  unsigned int gen;          // this launch's tag, never 0
  int ncons;                 // consumers: the tiles (set by launch_gemm_fused)
  int hold;                  // 0; 1 only from a test: the tiles' waits then give up
};

// Reads (and, with reset, clears) this device's count of hand-over waits
// that gave up.  Synchronous.
hipError_t handover_giveups(unsigned *count, bool reset);

// Whether the bf16 GEMM of this shape (M x N, reduction K; forward:
// row-major B; backward: k-major B, carrying the dA / dB side items) runs a
// tile configuration that takes producer workgroups, and leaves the CUs for
// them.
bool gemm_fusable(int M, int N, int K, bool b_kmajor);
// The bf16 GEMM with producers at the front (fz->nprod > 0; chooses
// fz->row.mb and sets fz->nprod, fz->nwg and fz->ncons).  fz->row.vmode
// selects the forward (V_ROW, side must be null) or the backward (V_KMAJ_TR,
// side items run by the producers); dx rows are required (g.M >= 1).
hipError_t launch_gemm_fused(const GemmArgs &g, FuseArgs *fz, const SideArgs *side, hipStream_t st);

// Split of a row-skinny product over its reduction axis L, and rows per
// workgroup.  Short T (below 2048): one 16-row tile per workgroup, enough
// segments to give the T / 16 row blocks about one workgroup per CU, no more
// than fit in the 64-wide padded LoRA step (nsplit * r <= tail_ld(r)).  Long
// T (bf16, r <= 32 and a multiple of 8): up to four 16-row tiles per
// workgroup, so each chunk of
// the rank-r factor serves up to 64 rows, and up to 4 segments (the same
// LoRA-step bound) for about 256 workgroups.  Always: each segment at least
// one 128-byte chunk per wave, and at most MAX_SPLIT segments.
constexpr int MAX_SPLIT = 8;
struct RowSplit {
  int nsplit, seg, mb;
};
RowSplit row_split(int64_t T, int64_t L, int r, Dtype dt);

// Padded row length of the LoRA-step operands (a multiple of the GEMM stage).
inline int tail_ld(int r, Dtype dt) {
  const int s = dt == DT_BF16 ? 64 : 32;
  return (r + s - 1) / s * s;
}

}  // namespace lora
