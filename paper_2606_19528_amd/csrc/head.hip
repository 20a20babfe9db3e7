// head.hip -- the frozen LM head's reduced-vocabulary cross entropy with
// logits masking, apart from its GEMMs (which run in gemm.hip with the
// cross-entropy epilogues):
//   * the reduced vocabulary J: every entry of the first k columns of the
//     similarity table's rows of the trainable positions' targets is marked
//     in a bitmap over the vocabulary, and the marks are compacted in
//     ascending order (so J is sorted and each target's position in J is a
//     lookup);
//   * row gathers (hidden states of the trainable positions, embedding rows
//     of J) into contiguous operands;
//   * the combine of the per-tile (max, sum of exp) partials into log-sum-exp
//     and per-position losses, and their sum, in a fixed order;
//   * the finishing of dh: bf16 rows at the trainable positions, zero rows
//     elsewhere.
#include "kernels.hpp"
#include "launch.hpp"

namespace lora {

__global__ void fill_u32_kernel(uint32_t *p, int64_t n, uint32_t v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// mark[table[targets[rows[i]]][c]] = 1 for i < nrows, c < k.  Every writer
// stores the same value, so the result does not depend on their order.
__global__ void vocab_mark_kernel(const int32_t *table, int64_t ldtab, int k,
                                  const int32_t *targets, const int32_t *rows, int nrows, int T,
                                  int V, uint32_t *mark) {
  const int64_t total = (int64_t)nrows * k;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int i = (int)(e / k), c = (int)(e % k);
    const int32_t t = rows[i];
    if (t < 0 || t >= T) continue;  // invalid indices are skipped, never followed
    const int32_t y = targets[t];
    if (y < 0 || y >= V) continue;
    const int32_t v = table[(int64_t)y * ldtab + c];
    if (v >= 0 && v < V) mark[v] = 1u;
  }
}

// One workgroup: ascending compaction of the marked entries.  Thread t owns
// the contiguous slice [t*per, (t+1)*per) of the vocabulary; slice counts are
// scanned in LDS.  J[pos] = v and pos_of[v] = pos for every marked v;
// count[0] = |J|.
constexpr int COMPACT_NT = 1024;
__global__ __launch_bounds__(COMPACT_NT) void vocab_compact_kernel(const uint32_t *mark, int V,
                                                                    int32_t *J, int32_t *pos_of,
                                                                    int32_t *count) {
  __shared__ int part[COMPACT_NT];
  const int t = threadIdx.x;
  const int per = (V + COMPACT_NT - 1) / COMPACT_NT;
  const int lo = min(V, t * per), hi = min(V, lo + per);
  int c = 0;
  for (int v = lo; v < hi; ++v) c += mark[v] != 0u;
  part[t] = c;
  __syncthreads();
  // Hillis-Steele inclusive scan over the slice counts
  for (int off = 1; off < COMPACT_NT; off <<= 1) {
    const int add = t >= off ? part[t - off] : 0;
    __syncthreads();
    part[t] += add;
    __syncthreads();
  }
  int pos = part[t] - c;
  for (int v = lo; v < hi; ++v) {
    if (mark[v] != 0u) {
      J[pos] = v;
      pos_of[v] = pos;
      ++pos;
    }
  }
  if (t == COMPACT_NT - 1) count[0] = part[t];
}

// tpos[i] = position in J of the target of trainable position rows[i].
// (-1 for an invalid position or target).
__global__ void target_pos_kernel(const int32_t *targets, const int32_t *rows, int nrows, int T,
                                  int V, const uint32_t *mark, const int32_t *pos_of,
                                  int32_t *tpos) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= nrows) return;
  const int32_t t = rows[i];
  const int32_t y = (t >= 0 && t < T) ? targets[t] : -1;
  tpos[i] = (y >= 0 && y < V && mark[y] != 0u) ? pos_of[y] : -1;
}

// dst[i][:] = src[idx[i]][:] for i < n (zeros for an index outside [0, nsrc));
// rows of `cols` bf16, cols % 8 == 0.
__global__ void gather_rows_kernel(const uint16_t *src, int64_t ld, int nsrc, const int32_t *idx,
                                   int n, int cols, uint16_t *dst) {
  const int vpr = cols / 8;  // 16-byte vectors per row
  const int64_t total = (int64_t)n * vpr;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = e / vpr;
    const int v = (int)(e % vpr);
    const int32_t r = idx[i];
    st16(dst + i * cols + v * 8, (r >= 0 && r < nsrc) ? ld16(src + (int64_t)r * ld + v * 8) : zero16());
  }
}

// Per position m: lse = M + log(sum_t s_t exp(m_t - M)), M = max_t m_t over
// the vocabulary tiles t (ascending), and loss = lse - z_target.
__global__ void ce_combine_kernel(const float *tmax, const float *tsum, int ntiles, int M,
                                  const float *ztgt, float *lse, float *loss) {
  const int m = blockIdx.x * blockDim.x + threadIdx.x;
  if (m >= M) return;
  float mx = tmax[m];
  for (int t = 1; t < ntiles; ++t) mx = fmaxf(mx, tmax[(int64_t)t * M + m]);
  float s = 0.0f;
  for (int t = 0; t < ntiles; ++t) s += tsum[(int64_t)t * M + m] * __expf(tmax[(int64_t)t * M + m] - mx);
  const float l = mx + __logf(s);
  lse[m] = l;
  loss[m] = l - ztgt[m];
}

// total[0] = sum of loss[0..M) by one workgroup: fixed per-thread strides,
// then a fixed pairwise tree.
constexpr int SUM_NT = 1024;
__global__ __launch_bounds__(SUM_NT) void sum_kernel(const float *loss, int M, float *total) {
  __shared__ float part[SUM_NT];
  const int t = threadIdx.x;
  float s = 0.0f;
  for (int m = t; m < M; m += SUM_NT) s += loss[m];
  part[t] = s;
  __syncthreads();
  for (int h = SUM_NT / 2; h >= 1; h >>= 1) {
    if (t < h) part[t] += part[t + h];
    __syncthreads();
  }
  if (t == 0) total[0] = part[0];
}

// inv[t] = i for t = rows[i], -1 for positions that are not listed.  (A
// position listed twice keeps one of its entries; the entry points require
// distinct positions.)
__global__ void invert_rows_kernel(const int32_t *rows, int nrows, int T, int32_t *inv) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nrows && rows[i] >= 0 && rows[i] < T) inv[rows[i]] = i;
}

// dh[t][:] = bf16(acc[inv[t]][:]) for listed positions, 0 for the others.
__global__ void dh_finish_kernel(const float *acc, const int32_t *inv, int T, int D, uint16_t *dh) {
  const int vpr = D / 8;
  const int64_t total = (int64_t)T * vpr;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t t = e / vpr;
    const int v = (int)(e % vpr);
    const int i = inv[t];
    u32x4 out = zero16();
    if (i >= 0) {
      const float *src = acc + (int64_t)i * D + v * 8;
      out = pack_vec(BF16(), src);
    }
    st16(dh + t * D + v * 8, out);
  }
}

static int grid_for(int64_t work, int nt);

hipError_t launch_fill_nan(float *p, int64_t n, hipStream_t st) {
  hipLaunchKernelGGL(fill_u32_kernel, dim3((int)((n + 255) / 256 < 8192 ? (n + 255) / 256 : 8192)),
                     dim3(256), 0, st, (uint32_t *)p, n, 0x7FC00000u);
  return hipGetLastError();
}

static int grid_for(int64_t work, int nt) {
  const int64_t g = (work + nt - 1) / nt;
  return (int)(g < 1 ? 1 : (g > 8192 ? 8192 : g));
}

hipError_t launch_vocab_build(const HeadVocabArgs &a, hipStream_t st) {
  hipLaunchKernelGGL(fill_u32_kernel, dim3(grid_for(a.V, 256)), dim3(256), 0, st, a.mark,
                     (int64_t)a.V, 0u);
  hipLaunchKernelGGL(vocab_mark_kernel, dim3(grid_for((int64_t)a.nrows * a.k, 256)), dim3(256), 0,
                     st, a.table, a.ldtab, a.k, a.targets, a.rows, a.nrows, a.T, a.V, a.mark);
  hipLaunchKernelGGL(vocab_compact_kernel, dim3(1), dim3(COMPACT_NT), 0, st, a.mark, a.V, a.J,
                     a.pos_of, a.count);
  hipLaunchKernelGGL(target_pos_kernel, dim3((a.nrows + 255) / 256), dim3(256), 0, st, a.targets,
                     a.rows, a.nrows, a.T, a.V, a.mark, a.pos_of, a.tpos);
  return hipGetLastError();
}

hipError_t launch_gather_rows(const void *src, int64_t ld, int nsrc, const int32_t *idx, int n,
                              int cols, void *dst, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(gather_rows_kernel, dim3(grid_for((int64_t)n * (cols / 8), 256)), dim3(256), 0,
                     st, (const uint16_t *)src, ld, nsrc, idx, n, cols, (uint16_t *)dst);
  return hipGetLastError();
}

hipError_t launch_ce_combine(const float *tmax, const float *tsum, int ntiles, int M,
                             const float *ztgt, float *lse, float *loss, float *total,
                             hipStream_t st) {
  hipLaunchKernelGGL(ce_combine_kernel, dim3((M + 255) / 256), dim3(256), 0, st, tmax, tsum, ntiles,
                     M, ztgt, lse, loss);
  if (total) hipLaunchKernelGGL(sum_kernel, dim3(1), dim3(SUM_NT), 0, st, loss, M, total);
  return hipGetLastError();
}

hipError_t launch_dh_finish(const float *acc, const int32_t *rows, int nrows, int32_t *inv, int T,
                            int D, void *dh, hipStream_t st) {
  hipLaunchKernelGGL(fill_u32_kernel, dim3(grid_for(T, 256)), dim3(256), 0, st, (uint32_t *)inv,
                     (int64_t)T, 0xFFFFFFFFu);
  hipLaunchKernelGGL(invert_rows_kernel, dim3((nrows + 255) / 256), dim3(256), 0, st, rows, nrows,
                     T, inv);
  hipLaunchKernelGGL(dh_finish_kernel, dim3(grid_for((int64_t)T * (D / 8), 256)), dim3(256), 0, st,
                     acc, inv, T, D, (uint16_t *)dh);
  return hipGetLastError();
}

}  // namespace lora
