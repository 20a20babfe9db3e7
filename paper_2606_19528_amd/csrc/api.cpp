// api.cpp -- the C ABI: argument validation, workspace layout and the launch
// sequence of each entry point.  Every argument is checked before any work is
// enqueued; the library allocates no device memory.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <vector>

#include "../../include/lora_mi355x.h"
#include "launch.hpp"

using namespace lora;

namespace {
thread_local char g_err[256] = "";
}  // namespace

void lora::set_last_error(const char *msg) { std::snprintf(g_err, sizeof g_err, "%s", msg); }

namespace {

lora_status_t fail(lora_status_t s, const char *msg) {
  lora::set_last_error(msg);
  return s;
}

// ----- kernel timing hook ----------------------------------------------------
enum KernelId {
  K_GEMM_FWD = 0,     // y  = x W^T + (s u) B^T
  K_GEMM_BWD_DX,      // dx = dy W + du A, with the dA / dB token reductions alongside
  K_GEMM_FROZEN_DX,   // dx = dy W (rank 0)
  K_LORA_DOWN,        // u  = x A^T (+ LoRA-step operands)
  K_LORA_DY_B,        // du = s dy B (+ LoRA-step operand)
  K_GEMM_FWD_Q,       // gemm_fwd with the quantized W dequantized on the fly
  K_GEMM_BWD_DX_Q,    // gemm_bwd_dx, quantized W
  K_GEMM_FROZEN_DX_Q, // gemm_frozen_dx, quantized W
  K_HEAD_VOCAB,       // reduced vocabulary (mark, compact, target positions)
  K_HEAD_GATHER,      // gathers of the trainable hidden rows and of the rows of J
  K_HEAD_LOGITS,      // logits GEMM with the row-statistics epilogue (+ combine)
  K_HEAD_DZ,          // logits recomputed, softmax gradient epilogue
  K_HEAD_DH,          // dh += dz W_J (fp32), then the bf16 dh rows
  K_TOPK_SIM,         // similarity GEMM with the candidate epilogue (+ row norms)
  K_TOPK_SELECT,      // per-row selection of the k best candidates
  K_COUNT
};
const char *kKernelNames[K_COUNT] = {"gemm_fwd",   "gemm_bwd_dx",   "gemm_frozen_dx",
                                     "lora_down",  "lora_dy_b",     "gemm_fwd_q",
                                     "gemm_bwd_dx_q", "gemm_frozen_dx_q", "head_vocab",
                                     "head_gather", "head_logits", "head_dz", "head_dh",
                                     "topk_sim", "topk_select"};

struct EventPair {
  hipEvent_t a, b;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<EventPair> g_prof[K_COUNT];

struct Timed {
  int id;
  hipStream_t st;
  EventPair ev{nullptr, nullptr};
  bool on = false;
  Timed(int id_, hipStream_t st_) : id(id_), st(st_) {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    if (!g_prof_on) return;
    if (hipEventCreate(&ev.a) != hipSuccess || hipEventCreate(&ev.b) != hipSuccess) return;
    on = hipEventRecord(ev.a, st) == hipSuccess;
  }
  void done() {
    if (!on) return;
    if (hipEventRecord(ev.b, st) != hipSuccess) return;
    std::lock_guard<std::mutex> lk(g_prof_mu);
    g_prof[id].push_back(ev);
    on = false;
  }
};

// ----- validation helpers ------------------------------------------------------
constexpr int64_t kMaxElems = (int64_t(1) << 31) - 1;
constexpr int kMaxRank = 128;
constexpr int64_t kMaxDim = int64_t(1) << 20;  // keeps every tile's byte offsets within 32 bits

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Range {
  uintptr_t lo, hi;  // [lo, hi)
  bool set;
};
Range rng(const void *p, int64_t bytes) {
  if (!p || bytes <= 0) return {0, 0, false};
  uintptr_t lo = reinterpret_cast<uintptr_t>(p);
  return {lo, lo + (uintptr_t)bytes, true};
}
bool overlap(const Range &a, const Range &b) {
  return a.set && b.set && a.lo < b.hi && b.lo < a.hi;
}
bool any_overlap(const std::vector<Range> &outs, const std::vector<Range> &ins) {
  for (size_t i = 0; i < outs.size(); ++i) {
    for (const Range &x : ins)
      if (overlap(outs[i], x)) return true;
    for (size_t j = i + 1; j < outs.size(); ++j)
      if (overlap(outs[i], outs[j])) return true;
  }
  return false;
}

size_t esize(lora_dtype_t dt) { return dt == LORA_BF16 ? 2 : 4; }
size_t round256(size_t b) { return (b + 255) & ~size_t(255); }

lora_status_t check_shapes(int64_t T, int64_t d_in, int64_t d_out, int64_t r, lora_dtype_t dt) {
  if (dt != LORA_BF16 && dt != LORA_F32) return fail(LORA_EINVAL, "unknown dtype");
  if (T < 1 || d_in < 1 || d_out < 1) return fail(LORA_EINVAL, "T, d_in and d_out must be >= 1");
  if (r < 0 || r > kMaxRank) return fail(LORA_EINVAL, "rank r must be in [0, 128]");
  if (d_in % 8 || d_out % 8) return fail(LORA_EUNSUPPORTED, "d_in and d_out must be multiples of 8");
  if (T > kMaxElems / d_in || T > kMaxElems / d_out || d_in > kMaxElems / d_out)
    return fail(LORA_EUNSUPPORTED, "a matrix has 2^31 or more elements");
  if (d_in > kMaxDim || d_out > kMaxDim)
    return fail(LORA_EUNSUPPORTED, "d_in and d_out must be at most 2^20");
  return LORA_OK;
}

// Workspace layouts (offsets in bytes, 256-byte aligned).  The rank-r row
// products are computed as `nsplit` partial sums over their reduction axis
// (row_split); the LoRA-step operands hold one column block per partial.
//
// The rank-r pass of either direction (forward u = x A^T, backward
// du = s dy B) runs fused into its GEMM launch -- as producer workgroups
// ahead of the tiles, each over whole rows -- when the operands are bf16, r
// is a multiple of 8 up to 32 and the GEMM takes a direct-to-LDS tile
// configuration that leaves the producers room beside the tiles; it then
// needs no partial sums and no padded copy of B (A), and the workspace starts
// with the hand-over words of the launch.  In the backward the producers then
// run the dA / dB side items, so those take no CUs of their own.
// (N, K: the GEMM's output columns and reduction length.)
bool fuse_ok(int64_t T, int64_t N, int64_t K, int64_t r, lora_dtype_t dt, bool b_kmajor = false) {
  return dt == LORA_BF16 && r >= 8 && r <= 32 && r % 8 == 0 && gemm_fusable((int)T, (int)N, (int)K, b_kmajor);
}
// Tag of a fused launch: distinct for every call of this process, never 0.
unsigned int next_gen() {
  static std::atomic<unsigned int> g{0};
  unsigned int v;
  do {
    v = ++g;
  } while (v == 0);
  return v;
}
// Test hook (lora_debug_set_handover): 1 makes every tile's hand-over wait
// of the following fused launches give up.
std::atomic<int> g_fz_hold{0};
void handover_params(FuseArgs &fz) { fz.hold = g_fz_hold.load(); }
// One segment over the whole reduction axis L, 16 rows per workgroup.
RowSplit whole_rows(int64_t L, Dtype d) {
  const int64_t ce = d == DT_BF16 ? 64 : 32;
  return RowSplit{1, (int)((L + ce - 1) / ce * ce), 1};
}

struct FwdLayout {
  size_t sync, u, utail, bpad, total;
  int ldt;
  bool fused;
  RowSplit sp;
};
FwdLayout fwd_layout(int64_t T, int64_t K, int64_t N, int64_t r, lora_dtype_t dt) {
  FwdLayout L{};
  if (r == 0) return L;
  const Dtype d = dt == LORA_BF16 ? DT_BF16 : DT_F32;
  L.fused = fuse_ok(T, N, K, r, dt);
  if (L.fused) {
    L.sp = whole_rows(K, d);
    L.ldt = tail_ld((int)r, d);
    size_t off = 0;
    L.sync = off;  // hand-over words
    off += 256;
    L.u = off;  // u = x A^T when the caller does not keep it, [T][r] fp32
    off += round256((size_t)T * r * 4);
    L.utail = off;  // [T][ldt]: E(s * u), zero-padded
    off += round256((size_t)T * L.ldt * esize(dt));
    L.total = off;
    return L;
  }
  L.sp = row_split(T, K, (int)r, d);
  L.ldt = tail_ld(L.sp.nsplit * (int)r, d);
  size_t off = 0;
  L.u = off;  // partial sums of u = x A^T, [nsplit][T][r] fp32
  off += round256((size_t)L.sp.nsplit * T * r * 4);
  L.utail = off;  // [T][ldt]: E(s * partial p) in columns p*r ..
  off += round256((size_t)T * L.ldt * esize(dt));
  L.bpad = off;  // [N][ldt]: B repeated once per partial, zero-padded
  off += round256((size_t)N * L.ldt * esize(dt));
  L.total = off;
  return L;
}

struct BwdLayout {
  size_t sync, u, du, dutail, acat, scnt, spart, total;
  int ldt;
  bool fused;
  RowSplit sp_u, sp_du;
  int tparts, tchunk;  // token parts of the dA / dB side items (unfused dx launch)
};
BwdLayout bwd_layout(int64_t T, int64_t K, int64_t N, int64_t r, lora_dtype_t dt) {
  BwdLayout L{};
  if (r == 0) return L;
  const Dtype d = dt == LORA_BF16 ? DT_BF16 : DT_F32;
  // A recomputed u is summed exactly as the forward pass summed it (whole
  // rows when the forward runs fused), so it is bitwise the saved one.
  L.sp_u = fuse_ok(T, N, K, r, dt) ? whole_rows(K, d) : row_split(T, K, (int)r, d);
  L.fused = fuse_ok(T, K, N, r, dt, true);
  L.sp_du = L.fused ? whole_rows(N, d) : row_split(T, N, (int)r, d);
  L.ldt = tail_ld(L.sp_du.nsplit * (int)r, d);
  size_t off = 0;
  L.sync = off;  // hand-over words of a fused launch
  off += L.fused ? 256 : 0;
  L.u = off;  // partial sums of u (when it is recomputed)
  off += round256((size_t)L.sp_u.nsplit * T * r * 4);
  L.du = off;  // partial sums of du = s dy B
  off += round256((size_t)L.sp_du.nsplit * T * r * 4);
  L.dutail = off;  // [T][ldt]: E(partial p of du) in columns p*r ..
  off += round256((size_t)T * L.ldt * esize(dt));
  L.acat = off;  // [nsplit * r][K]: A repeated once per partial
  off += L.sp_du.nsplit > 1 ? round256((size_t)L.sp_du.nsplit * r * K * esize(dt)) : 0;
  L.tparts = 1;
  L.tchunk = (int)T;
  if (!L.fused) side_split(T, K, N, r, d, &L.tparts, &L.tchunk);
  const size_t items = L.tparts > 1 ? (size_t)side_item_count(K, N, r, d) : 0;
  L.scnt = off;  // [items] part counts of the side items
  off += round256(items * 4);
  L.spart = off;  // [items][tparts] part tiles
  off += items * L.tparts * SIDE_SLOT_FLOATS * 4;
  L.total = off;
  return L;
}

// LM head workspaces.
constexpr int64_t kHeadChunk = 8192;  // vocabulary columns per backward chunk (multiple of 128)
struct VocabLayout {
  size_t mark, pos_of, count, total;
};
VocabLayout vocab_layout(int64_t V) {
  VocabLayout L{};
  size_t off = 0;
  L.mark = off;
  off += round256((size_t)V * 4);
  L.pos_of = off;
  off += round256((size_t)V * 4);
  L.count = off;
  off += 256;
  L.total = off;
  return L;
}
struct CeLayout {
  size_t hT, WJ, tmax, tsum, ztgt, lse, dz, dhacc, inv, total;
  int64_t tiles;
};
CeLayout ce_layout(int64_t T, int64_t D, int64_t nrows, int64_t nJ, bool want_dh) {
  CeLayout L{};
  L.tiles = (nJ + 127) / 128;
  size_t off = 0;
  L.hT = off;
  off += round256((size_t)nrows * D * 2);
  L.WJ = off;
  off += round256((size_t)nJ * D * 2);
  L.tmax = off;
  off += round256((size_t)L.tiles * nrows * 4);
  L.tsum = off;
  off += round256((size_t)L.tiles * nrows * 4);
  L.ztgt = off;
  off += round256((size_t)nrows * 4);
  L.lse = off;
  off += round256((size_t)nrows * 4);
  if (want_dh) {
    const int64_t ch = nJ < kHeadChunk ? (nJ + 7) / 8 * 8 : kHeadChunk;
    L.dz = off;
    off += round256((size_t)nrows * ch * 2);
    L.dhacc = off;
    off += round256((size_t)nrows * D * 4);
    L.inv = off;
    off += round256((size_t)T * 4);
  }
  L.total = off;
  return L;
}

// Top-k table workspace: row norms, and per batch of rows a threshold, a
// count and a candidate list per row (TOPK_SLOTS minus the sort slots of the
// final pass: room for k plus at least one column chunk, so that most chunks
// need no selection).
constexpr int64_t kTopkChunk = 4096, kTopkBatch = 16384;
struct TopkLayout {
  size_t rn, thr, cnt, val, idx, total;
  int64_t R, cap, lazy;
};
TopkLayout topk_layout(int64_t V, int64_t k) {
  TopkLayout L{};
  L.R = std::min(V, kTopkBatch);
  int64_t p2 = 1;
  while (p2 < k) p2 <<= 1;
  L.cap = (TOPK_SLOTS - p2) & ~3;  // >= k + kTopkChunk for every k <= 2048; whole vectors of 4
  L.lazy = L.cap - kTopkChunk;
  size_t off = 0;
  L.rn = off;
  off += round256((size_t)V * 4);
  L.thr = off;
  off += round256((size_t)L.R * 4);
  L.cnt = off;
  off += round256((size_t)L.R * 4);
  L.val = off;
  off += round256((size_t)L.R * L.cap * 4);
  L.idx = off;
  off += round256((size_t)L.R * L.cap * 4);
  L.total = off;
  return L;
}

lora_status_t check_ws(void *ws, size_t ws_bytes, size_t need) {
  if (need == 0) return LORA_OK;
  if (!ws) return fail(LORA_EWORKSPACE, "workspace required but ws is NULL");
  if (ws_bytes < need) return fail(LORA_EWORKSPACE, "workspace too small");
  if (!aligned16(ws)) return fail(LORA_EINVAL, "workspace not 16-byte aligned");
  return LORA_OK;
}

// A quantized frozen weight W [d_out, d_in]: unsigned codes of `bits` bits
// ([d_out][d_in * bits / 8] bytes; two 4-bit codes per byte, the even input in
// the low nibble), W = scale * code + offset with one fp32 scale and offset per
// group of `group` consecutive inputs of a row ([d_out][d_in / group]).
struct QWeight {
  const void *codes;
  const float *scale, *offset;
  int bits, log2g;
};

lora_status_t check_qweight(const void *codes, const float *scale, const float *offset, int bits,
                            int64_t group, int64_t d_in, int64_t d_out, int64_t r,
                            lora_dtype_t dt, QWeight *q, std::vector<Range> *ins) {
  if (dt != LORA_BF16) return fail(LORA_EUNSUPPORTED, "a quantized weight needs dt = LORA_BF16");
  if (bits != 4 && bits != 8) return fail(LORA_EINVAL, "bits must be 4 or 8");
  if (!codes || !scale || !offset) return fail(LORA_EINVAL, "codes, scale and offset are required");
  if (!aligned16(codes) || !aligned16(scale) || !aligned16(offset))
    return fail(LORA_EINVAL, "pointers must be 16-byte aligned");
  if (group < 16 || (group & (group - 1)) != 0 || d_in % group != 0)
    return fail(LORA_EUNSUPPORTED, "group must be a power of two >= 16 that divides d_in");
  if (r > 64) return fail(LORA_EUNSUPPORTED, "rank r must be at most 64 with a quantized weight");
  int log2g = 0;
  while ((int64_t(1) << log2g) < group) ++log2g;
  *q = QWeight{codes, scale, offset, bits, log2g};
  ins->push_back(rng(codes, d_out * d_in * bits / 8));
  ins->push_back(rng(scale, d_out * (d_in / group) * 4));
  ins->push_back(rng(offset, d_out * (d_in / group) * 4));
  return LORA_OK;
}

void set_qweight(GemmArgs &g, const QWeight *q) {
  if (!q) return;
  g.B = q->codes;
  g.qscale = q->scale;
  g.qoffset = q->offset;
  g.qlog2g = q->log2g;
}

hipError_t run_gemm(const GemmArgs &g, Dtype d, const QWeight *q, bool kmajor, const SideArgs *side,
                    hipStream_t st) {
  return q ? launch_gemm_q(g, q->bits, kmajor, side, st) : launch_gemm(g, d, kmajor, side, st);
}

lora_status_t hip_fail(hipError_t e, const char *what) {
  std::snprintf(g_err, sizeof g_err, "%s: %s", what, hipGetErrorString(e));
  return LORA_EHIP;
}

// Forward with a bf16/fp32 W, or (qc != NULL) a quantized one.
lora_status_t fwd_impl(const void *x, const void *W, const void *qc, const float *qs,
                       const float *qo, int bits, int64_t group, const void *A, const void *B,
                       void *y, float *u_save, int64_t T, int64_t d_in, int64_t d_out, int64_t r,
                       float scale, lora_dtype_t dt, void *ws, size_t ws_bytes, void *hip_stream) {
  lora_status_t s = check_shapes(T, d_in, d_out, r, dt);
  if (s != LORA_OK) return s;
  QWeight qw{};
  std::vector<Range> qins;
  if (qc) {
    if ((s = check_qweight(qc, qs, qo, bits, group, d_in, d_out, r, dt, &qw, &qins)) != LORA_OK)
      return s;
    W = qc;
  }
  if (!x || !W || !y) return fail(LORA_EINVAL, "x, W and y are required");
  if (r > 0 && (!A || !B)) return fail(LORA_EINVAL, "A and B are required when r > 0");
  if (r > 0 && !std::isfinite(scale)) return fail(LORA_EINVAL, "scale must be finite");
  const void *ptrs[] = {x, W, y, r > 0 ? A : nullptr, r > 0 ? B : nullptr,
                        r > 0 ? (const void *)u_save : nullptr};
  for (const void *p : ptrs)
    if (p && !aligned16(p)) return fail(LORA_EINVAL, "pointers must be 16-byte aligned");
  const size_t es = esize(dt);
  const size_t need = lora_linear_workspace_bytes(LORA_OP_FWD, T, d_in, d_out, r, dt);
  if ((s = check_ws(ws, ws_bytes, need)) != LORA_OK) return s;
  std::vector<Range> ins = {rng(x, T * d_in * es)};
  if (qc) ins.insert(ins.end(), qins.begin(), qins.end());
  else ins.push_back(rng(W, d_out * d_in * es));
  std::vector<Range> outs = {rng(y, T * d_out * es)};
  if (r > 0) {
    ins.push_back(rng(A, r * d_in * es));
    ins.push_back(rng(B, d_out * r * es));
    if (u_save) outs.push_back(rng(u_save, T * r * 4));
    if (need) outs.push_back(rng(ws, (int64_t)need));
  }
  if (any_overlap(outs, ins)) return fail(LORA_EINVAL, "an output overlaps an input or another output");

  hipStream_t st = (hipStream_t)hip_stream;
  const Dtype d = dt == LORA_BF16 ? DT_BF16 : DT_F32;
  GemmArgs g{};
  g.A = x; g.lda = d_in;
  g.B = W; g.ldb = d_in;
  g.M = (int)T; g.N = (int)d_out; g.K = (int)d_in;
  g.C = y; g.ldc = d_out;
  if (r > 0 && !qc && fwd_layout(T, d_in, d_out, r, dt).fused) {
    const FwdLayout L = fwd_layout(T, d_in, d_out, r, dt);
    char *wsb = (char *)ws;
    FuseArgs fz{};
    RowArgs &ra = fz.row;
    ra.X = x; ra.ldx = d_in; ra.M = (int)T; ra.L = (int)d_in;
    ra.V = A; ra.ldv = d_in; ra.vmode = V_ROW; ra.r = (int)r;
    ra.nsplit = 1; ra.seg = L.sp.seg; ra.mb = 1;
    ra.out_mult = 1.0f; ra.out = u_save ? u_save : (float *)(wsb + L.u); ra.out_stride = T * r;
    ra.tail = wsb + L.utail; ra.ldt = L.ldt; ra.tail_mult = scale;
    fz.nprod = (int)((T + 15) / 16);
    fz.sync = (unsigned long long *)(wsb + L.sync);
    fz.gen = next_gen();
    handover_params(fz);
    g.A2 = wsb + L.utail; g.lda2 = L.ldt;
    g.B2 = B; g.ldb2 = r;  // rows of r bf16: whole 16-byte vectors
    g.r = (int)r;
    Timed t(K_GEMM_FWD, st);
    hipError_t e = launch_gemm_fused(g, &fz, nullptr, st);
    t.done();
    if (e != hipSuccess) return hip_fail(e, "gemm_fwd launch");
    return LORA_OK;
  }
  if (r > 0) {
    const FwdLayout L = fwd_layout(T, d_in, d_out, r, dt);
    const int ns = L.sp.nsplit;
    char *wsb = (char *)ws;
    float *upart = (float *)(wsb + L.u);
    RowArgs ra{};
    ra.X = x; ra.ldx = d_in; ra.M = (int)T; ra.L = (int)d_in;
    ra.V = A; ra.ldv = d_in; ra.vmode = V_ROW; ra.r = (int)r;
    ra.nsplit = ns; ra.seg = L.sp.seg; ra.mb = L.sp.mb;
    ra.out_mult = 1.0f; ra.out = (ns == 1 && u_save) ? u_save : upart; ra.out_stride = T * r;
    ra.tail = wsb + L.utail; ra.ldt = L.ldt; ra.tail_mult = scale;
    // B itself serves as the LoRA-step operand when there is one partial and
    // its rows are whole 16-byte vectors; otherwise the kernel writes B
    // repeated once per partial, zero-padded.
    const bool pad_b = ns > 1 || r % (16 / (int64_t)esize(dt)) != 0;
    if (pad_b) {
      ra.bcopy_mode = BCOPY_COLS; ra.bcopy_src = B; ra.bcopy_dst = wsb + L.bpad;
      ra.bcopy_rows = (int)d_out;
    }
    Timed t(K_LORA_DOWN, st);
    hipError_t e = launch_row_skinny(ra, d, st);
    t.done();
    if (e != hipSuccess) return hip_fail(e, "lora_down launch");
    g.A2 = wsb + L.utail; g.lda2 = L.ldt;
    g.B2 = pad_b ? (const void *)(wsb + L.bpad) : B;
    g.ldb2 = pad_b ? L.ldt : r;
    g.r = (int)(ns * r);
    if (ns > 1 && u_save) {
      g.usum_src = upart; g.usum_out = u_save; g.usum_parts = ns; g.usum_r = (int)r;
    }
  }
  set_qweight(g, qc ? &qw : nullptr);
  Timed t(qc ? K_GEMM_FWD_Q : K_GEMM_FWD, st);
  hipError_t e = run_gemm(g, d, qc ? &qw : nullptr, false, nullptr, st);
  t.done();
  if (e != hipSuccess) return hip_fail(e, "gemm_fwd launch");
  return LORA_OK;
}

lora_status_t bwd_impl(const void *x, const void *W, const void *qc, const float *qs,
                       const float *qo, int bits, int64_t group, const void *A, const void *B,
                       const float *u_saved, const void *dy, void *dx, float *dA, float *dB,
                       int64_t T, int64_t d_in, int64_t d_out, int64_t r, float scale,
                       lora_dtype_t dt, void *ws, size_t ws_bytes, void *hip_stream) {
  lora_status_t s = check_shapes(T, d_in, d_out, r, dt);
  if (s != LORA_OK) return s;
  QWeight qw{};
  std::vector<Range> qins;
  if (qc) {
    if ((s = check_qweight(qc, qs, qo, bits, group, d_in, d_out, r, dt, &qw, &qins)) != LORA_OK)
      return s;
    W = qc;
  }
  if (!dy || !W) return fail(LORA_EINVAL, "dy and W are required");
  if (r > 0 && (!x || !A || !B || !dA || !dB))
    return fail(LORA_EINVAL, "x, A, B, dA and dB are required when r > 0");
  if (r == 0 && !dx) return fail(LORA_EINVAL, "nothing to compute: r = 0 and dx is NULL");
  if (r > 0 && !std::isfinite(scale)) return fail(LORA_EINVAL, "scale must be finite");
  const void *ptrs[] = {x, qc ? nullptr : W, A, B, u_saved, dy, dx, dA, dB};
  for (const void *p : ptrs)
    if (p && !aligned16(p)) return fail(LORA_EINVAL, "pointers must be 16-byte aligned");
  const size_t es = esize(dt);
  const size_t need = lora_linear_workspace_bytes(LORA_OP_BWD, T, d_in, d_out, r, dt);
  if ((s = check_ws(ws, ws_bytes, need)) != LORA_OK) return s;
  std::vector<Range> ins = {rng(dy, T * d_out * es)};
  if (qc) ins.insert(ins.end(), qins.begin(), qins.end());
  else ins.push_back(rng(W, d_out * d_in * es));
  std::vector<Range> outs;
  if (dx) outs.push_back(rng(dx, T * d_in * es));
  if (r > 0) {
    ins.push_back(rng(x, T * d_in * es));
    ins.push_back(rng(A, r * d_in * es));
    ins.push_back(rng(B, d_out * r * es));
    if (u_saved) ins.push_back(rng(u_saved, T * r * 4));
    outs.push_back(rng(dA, r * d_in * 4));
    outs.push_back(rng(dB, d_out * r * 4));
    if (need) outs.push_back(rng(ws, (int64_t)need));
  }
  if (any_overlap(outs, ins)) return fail(LORA_EINVAL, "an output overlaps an input or another output");

  hipStream_t st = (hipStream_t)hip_stream;
  const Dtype d = dt == LORA_BF16 ? DT_BF16 : DT_F32;
  hipError_t e;
  GemmArgs g{};
  g.A = dy; g.lda = d_out;
  g.B = W; g.ldb = d_in;
  g.M = dx ? (int)T : 0; g.N = (int)d_in; g.K = (int)d_out;
  g.C = dx; g.ldc = d_in;
  set_qweight(g, qc ? &qw : nullptr);
  if (r == 0) {
    Timed t(qc ? K_GEMM_BWD_DX_Q : K_GEMM_BWD_DX, st);
    e = run_gemm(g, d, qc ? &qw : nullptr, true, nullptr, st);
    t.done();
    return e == hipSuccess ? LORA_OK : hip_fail(e, "gemm_bwd_dx launch");
  }

  const BwdLayout L = bwd_layout(T, d_in, d_out, r, dt);
  char *wsb = (char *)ws;
  const float *u = u_saved;
  int u_parts = 1;
  if (!u) {  // rematerialise u = x A^T instead of having stored it
    RowArgs ra{};
    ra.X = x; ra.ldx = d_in; ra.M = (int)T; ra.L = (int)d_in;
    ra.V = A; ra.ldv = d_in; ra.vmode = V_ROW; ra.r = (int)r;
    ra.nsplit = L.sp_u.nsplit; ra.seg = L.sp_u.seg; ra.mb = L.sp_u.mb;
    ra.out_mult = 1.0f; ra.out = (float *)(wsb + L.u); ra.out_stride = T * r;
    Timed t(K_LORA_DOWN, st);
    e = launch_row_skinny(ra, d, st);
    t.done();
    if (e != hipSuccess) return hip_fail(e, "lora_down launch");
    u = (const float *)(wsb + L.u);
    u_parts = L.sp_u.nsplit;
  }
  const int ns = L.sp_du.nsplit;
  float *du = (float *)(wsb + L.du);
  if (L.fused && !qc && dx) {
    // du = s dy B by the producer workgroups of the dx launch, which then run
    // the dA / dB side items.
    FuseArgs fz{};
    RowArgs &ra = fz.row;
    ra.X = dy; ra.ldx = d_out; ra.M = (int)T; ra.L = (int)d_out;
    ra.V = B; ra.ldv = r; ra.vmode = V_KMAJ_TR; ra.r = (int)r;
    ra.nsplit = 1; ra.seg = L.sp_du.seg; ra.mb = 1;
    ra.out_mult = scale; ra.out = du; ra.out_stride = T * r;
    ra.tail = wsb + L.dutail; ra.ldt = L.ldt; ra.tail_mult = scale;
    fz.nprod = (int)((T + 15) / 16);
    fz.sync = (unsigned long long *)(wsb + L.sync);
    fz.gen = next_gen();
    handover_params(fz);
    SideArgs sd{};
    sd.T = (int)T; sd.r = (int)r; sd.njobs = 2; sd.scale1 = scale; sd.vstride = T * r;
    sd.job[0] = ColJob{x, du, dA, (int)d_in, 1};
    sd.job[1] = ColJob{dy, u, dB, (int)d_out, u_parts};
    g.A2 = wsb + L.dutail; g.lda2 = L.ldt;
    g.B2 = A; g.ldb2 = d_in;
    g.r = (int)r;
    Timed t(K_GEMM_BWD_DX, st);
    e = launch_gemm_fused(g, &fz, &sd, st);
    t.done();
    if (e != hipSuccess) return hip_fail(e, "gemm_bwd_dx launch");
    return LORA_OK;
  }
  {
    RowArgs ra{};
    ra.X = dy; ra.ldx = d_out; ra.M = (int)T; ra.L = (int)d_out;
    ra.V = B; ra.ldv = r; ra.vmode = V_KMAJ_TR; ra.r = (int)r;
    ra.nsplit = ns; ra.seg = L.sp_du.seg; ra.mb = L.sp_du.mb;
    ra.out_mult = scale; ra.out = du; ra.out_stride = T * r;
    ra.tail = wsb + L.dutail; ra.ldt = L.ldt; ra.tail_mult = scale;
    if (ns > 1) {  // A repeated once per partial of du
      ra.bcopy_mode = BCOPY_FLAT; ra.bcopy_src = A; ra.bcopy_dst = wsb + L.acat;
      ra.bcopy_period = r * d_in; ra.bcopy_elems = ns * r * d_in;
    }
    if (L.tparts > 1) {  // the dx launch's side parts count from zero
      ra.zero = (unsigned *)(wsb + L.scnt);
      ra.nzero = side_item_count(d_in, d_out, r, d);
    }
    Timed t(K_LORA_DY_B, st);
    e = launch_row_skinny(ra, d, st);
    t.done();
    if (e != hipSuccess) return hip_fail(e, "lora_dy_b launch");
  }
  SideArgs sd{};
  sd.T = (int)T; sd.r = (int)r; sd.njobs = 2; sd.scale1 = scale; sd.vstride = T * r;
  sd.job[0] = ColJob{x, du, dA, (int)d_in, ns};
  sd.job[1] = ColJob{dy, u, dB, (int)d_out, u_parts};
  sd.tparts = L.tparts; sd.tchunk = L.tchunk;
  sd.cnt = (unsigned *)(wsb + L.scnt);
  sd.part = (float *)(wsb + L.spart);
  g.A2 = wsb + L.dutail; g.lda2 = L.ldt;
  g.B2 = ns > 1 ? (const void *)(wsb + L.acat) : A; g.ldb2 = d_in;
  g.r = (int)(ns * r);
  Timed t(qc ? K_GEMM_BWD_DX_Q : K_GEMM_BWD_DX, st);
  e = run_gemm(g, d, qc ? &qw : nullptr, true, &sd, st);
  t.done();
  if (e != hipSuccess) return hip_fail(e, "gemm_bwd_dx launch");
  return LORA_OK;
}

lora_status_t frozen_impl(const void *dy, const void *W, const void *qc, const float *qs,
                          const float *qo, int bits, int64_t group, void *dx, int64_t T,
                          int64_t d_in, int64_t d_out, lora_dtype_t dt, void *hip_stream) {
  lora_status_t s = check_shapes(T, d_in, d_out, 0, dt);
  if (s != LORA_OK) return s;
  QWeight qw{};
  std::vector<Range> ins;
  if (qc) {
    if ((s = check_qweight(qc, qs, qo, bits, group, d_in, d_out, 0, dt, &qw, &ins)) != LORA_OK)
      return s;
    W = qc;
  }
  if (!dy || !W || !dx) return fail(LORA_EINVAL, "dy, W and dx are required");
  if (!aligned16(dy) || !aligned16(W) || !aligned16(dx))
    return fail(LORA_EINVAL, "pointers must be 16-byte aligned");
  const size_t es = esize(dt);
  if (!qc) ins.push_back(rng(W, d_out * d_in * es));
  ins.push_back(rng(dy, T * d_out * es));
  std::vector<Range> outs = {rng(dx, T * d_in * es)};
  if (any_overlap(outs, ins)) return fail(LORA_EINVAL, "an output overlaps an input");
  hipStream_t st = (hipStream_t)hip_stream;
  GemmArgs g{};
  g.A = dy; g.lda = d_out;
  g.B = W; g.ldb = d_in;
  g.M = (int)T; g.N = (int)d_in; g.K = (int)d_out;
  g.C = dx; g.ldc = d_in;
  set_qweight(g, qc ? &qw : nullptr);
  Timed t(qc ? K_GEMM_FROZEN_DX_Q : K_GEMM_FROZEN_DX, st);
  hipError_t e = run_gemm(g, dt == LORA_BF16 ? DT_BF16 : DT_F32, qc ? &qw : nullptr, true, nullptr, st);
  t.done();
  return e == hipSuccess ? LORA_OK : hip_fail(e, "gemm_frozen_dx launch");
}

}  // namespace

extern "C" {

size_t lora_linear_workspace_bytes(lora_op_t op, int64_t T, int64_t d_in, int64_t d_out,
                                   int64_t r, lora_dtype_t dt) {
  if (check_shapes(T, d_in, d_out, op == LORA_OP_FROZEN_DX ? 0 : r, dt) != LORA_OK)
    return (size_t)-1;
  switch (op) {
    case LORA_OP_FWD:
      return fwd_layout(T, d_in, d_out, r, dt).total;
    case LORA_OP_BWD:
      return bwd_layout(T, d_in, d_out, r, dt).total;
    case LORA_OP_FROZEN_DX:
      return 0;
  }
  return (size_t)-1;
}

lora_status_t lora_linear_fwd(const void *x, const void *W, const void *A, const void *B,
                              void *y, float *u_save, int64_t T, int64_t d_in, int64_t d_out,
                              int64_t r, float scale, lora_dtype_t dt, void *ws,
                              size_t ws_bytes, void *hip_stream) {
  return fwd_impl(x, W, nullptr, nullptr, nullptr, 0, 0, A, B, y, u_save, T, d_in, d_out, r,
                  scale, dt, ws, ws_bytes, hip_stream);
}

lora_status_t lora_linear_fwd_q(const void *x, const void *W_codes, const float *W_scale,
                                const float *W_offset, int bits, int64_t group, const void *A,
                                const void *B, void *y, float *u_save, int64_t T, int64_t d_in,
                                int64_t d_out, int64_t r, float scale, void *ws, size_t ws_bytes,
                                void *hip_stream) {
  if (!W_codes) return fail(LORA_EINVAL, "codes, scale and offset are required");
  return fwd_impl(x, nullptr, W_codes, W_scale, W_offset, bits, group, A, B, y, u_save, T, d_in,
                  d_out, r, scale, LORA_BF16, ws, ws_bytes, hip_stream);
}

lora_status_t lora_linear_bwd(const void *x, const void *W, const void *A, const void *B,
                              const float *u_saved, const void *dy, void *dx, float *dA,
                              float *dB, int64_t T, int64_t d_in, int64_t d_out, int64_t r,
                              float scale, lora_dtype_t dt, void *ws, size_t ws_bytes,
                              void *hip_stream) {
  return bwd_impl(x, W, nullptr, nullptr, nullptr, 0, 0, A, B, u_saved, dy, dx, dA, dB, T, d_in,
                  d_out, r, scale, dt, ws, ws_bytes, hip_stream);
}

lora_status_t lora_linear_bwd_q(const void *x, const void *W_codes, const float *W_scale,
                                const float *W_offset, int bits, int64_t group, const void *A,
                                const void *B, const float *u_saved, const void *dy, void *dx,
                                float *dA, float *dB, int64_t T, int64_t d_in, int64_t d_out,
                                int64_t r, float scale, void *ws, size_t ws_bytes,
                                void *hip_stream) {
  if (!W_codes) return fail(LORA_EINVAL, "codes, scale and offset are required");
  return bwd_impl(x, nullptr, W_codes, W_scale, W_offset, bits, group, A, B, u_saved, dy, dx, dA,
                  dB, T, d_in, d_out, r, scale, LORA_BF16, ws, ws_bytes, hip_stream);
}

lora_status_t frozen_linear_bwd_dx(const void *dy, const void *W, void *dx, int64_t T,
                                   int64_t d_in, int64_t d_out, lora_dtype_t dt, void *ws,
                                   size_t ws_bytes, void *hip_stream) {
  (void)ws;
  (void)ws_bytes;
  return frozen_impl(dy, W, nullptr, nullptr, nullptr, 0, 0, dx, T, d_in, d_out, dt, hip_stream);
}

lora_status_t frozen_linear_bwd_dx_q(const void *dy, const void *W_codes, const float *W_scale,
                                     const float *W_offset, int bits, int64_t group, void *dx,
                                     int64_t T, int64_t d_in, int64_t d_out, void *ws,
                                     size_t ws_bytes, void *hip_stream) {
  (void)ws;
  (void)ws_bytes;
  if (!W_codes) return fail(LORA_EINVAL, "codes, scale and offset are required");
  return frozen_impl(dy, nullptr, W_codes, W_scale, W_offset, bits, group, dx, T, d_in, d_out,
                     LORA_BF16, hip_stream);
}

size_t lm_head_workspace_bytes(int op, int64_t T, int64_t V, int64_t D, int64_t nrows,
                               int64_t nJ) {
  if (T < 1 || V < 1 || D < 8 || D % 8 || nrows < 1 || nrows > T || V > kMaxElems || D > kMaxDim ||
      T > kMaxElems / D || V > kMaxElems / D)
    return (size_t)-1;
  if (op == LM_HEAD_OP_VOCAB) return vocab_layout(V).total;
  if (nJ < 1 || nJ > V) return (size_t)-1;
  if (op == LM_HEAD_OP_LOSS) return ce_layout(T, D, nrows, nJ, false).total;
  if (op == LM_HEAD_OP_LOSS_DH) return ce_layout(T, D, nrows, nJ, true).total;
  return (size_t)-1;
}

lora_status_t lm_head_build_vocab(const int32_t *table, int64_t V, int64_t ldtab, int64_t k,
                                  const int32_t *targets, int64_t T, const int32_t *rows,
                                  int64_t nrows, int32_t *J, int32_t *tpos, int64_t *nJ, void *ws,
                                  size_t ws_bytes, void *hip_stream) {
  if (!table || !targets || !rows || !J || !tpos || !nJ)
    return fail(LORA_EINVAL, "table, targets, rows, J, tpos and nJ are required");
  if (V < 1 || V > kMaxElems || T < 1 || T > kMaxElems || nrows < 1 || nrows > T)
    return fail(LORA_EINVAL, "need V >= 1, T >= 1 and 1 <= nrows <= T");
  if (k < 1 || k > ldtab || ldtab > kMaxElems / V || (int64_t)nrows * k > kMaxElems)
    return fail(LORA_EINVAL, "need 1 <= k <= ldtab and a table below 2^31 entries");
  const void *ptrs[] = {table, targets, rows, J, tpos};
  for (const void *p : ptrs)
    if (!aligned16(p)) return fail(LORA_EINVAL, "pointers must be 16-byte aligned");
  const VocabLayout L = vocab_layout(V);
  lora_status_t s;
  if ((s = check_ws(ws, ws_bytes, L.total)) != LORA_OK) return s;
  std::vector<Range> ins = {rng(table, V * ldtab * 4), rng(targets, T * 4), rng(rows, nrows * 4)};
  std::vector<Range> outs = {rng(J, V * 4), rng(tpos, nrows * 4), rng(ws, (int64_t)L.total)};
  if (any_overlap(outs, ins)) return fail(LORA_EINVAL, "an output overlaps an input or another output");
  hipStream_t st = (hipStream_t)hip_stream;
  char *wsb = (char *)ws;
  HeadVocabArgs a{};
  a.table = table; a.ldtab = ldtab; a.k = (int)k; a.V = (int)V; a.T = (int)T;
  a.targets = targets; a.rows = rows; a.nrows = (int)nrows;
  a.mark = (uint32_t *)(wsb + L.mark); a.J = J; a.pos_of = (int32_t *)(wsb + L.pos_of);
  a.tpos = tpos; a.count = (int32_t *)(wsb + L.count);
  Timed t(K_HEAD_VOCAB, st);
  hipError_t e = launch_vocab_build(a, st);
  t.done();
  if (e != hipSuccess) return hip_fail(e, "head_vocab launch");
  int32_t count = 0;
  if ((e = hipMemcpyAsync(&count, a.count, 4, hipMemcpyDeviceToHost, st)) != hipSuccess)
    return hip_fail(e, "reading |J|");
  if ((e = hipStreamSynchronize(st)) != hipSuccess) return hip_fail(e, "reading |J|");
  *nJ = count;
  return LORA_OK;
}

lora_status_t lm_head_reduced_ce(const void *h, const void *W, int64_t T, int64_t V, int64_t D,
                                 const int32_t *rows, int64_t nrows, const int32_t *J, int64_t nJ,
                                 const int32_t *tpos, float *loss_rows, float *loss_total,
                                 void *dh, float dscale, void *ws, size_t ws_bytes,
                                 void *hip_stream) {
  if (!h || !W || !rows || !J || !tpos || !loss_rows)
    return fail(LORA_EINVAL, "h, W, rows, J, tpos and loss_rows are required");
  if (T < 1 || V < 1 || nrows < 1 || nrows > T || nJ < 1 || nJ > V)
    return fail(LORA_EINVAL, "need 1 <= nrows <= T and 1 <= nJ <= V");
  if (D < 8 || D % 8) return fail(LORA_EUNSUPPORTED, "D must be a positive multiple of 8");
  if (D > kMaxDim || T > kMaxElems / D || V > kMaxElems / D)
    return fail(LORA_EUNSUPPORTED, "D at most 2^20 and h, W below 2^31 elements");
  if (dh && !std::isfinite(dscale)) return fail(LORA_EINVAL, "dscale must be finite");
  const void *ptrs[] = {h, W, rows, J, tpos, loss_rows, loss_total, dh};
  for (const void *p : ptrs)
    if (p && !aligned16(p)) return fail(LORA_EINVAL, "pointers must be 16-byte aligned");
  const CeLayout L = ce_layout(T, D, nrows, nJ, dh != nullptr);
  lora_status_t s;
  if ((s = check_ws(ws, ws_bytes, L.total)) != LORA_OK) return s;
  std::vector<Range> ins = {rng(h, T * D * 2), rng(W, V * D * 2), rng(rows, nrows * 4),
                            rng(J, nJ * 4), rng(tpos, nrows * 4)};
  std::vector<Range> outs = {rng(loss_rows, nrows * 4), rng(ws, (int64_t)L.total)};
  if (loss_total) outs.push_back(rng(loss_total, 4));
  if (dh) outs.push_back(rng(dh, T * D * 2));
  if (any_overlap(outs, ins)) return fail(LORA_EINVAL, "an output overlaps an input or another output");

  hipStream_t st = (hipStream_t)hip_stream;
  char *wsb = (char *)ws;
  void *hT = wsb + L.hT, *WJ = wsb + L.WJ;
  float *tmax = (float *)(wsb + L.tmax), *tsum = (float *)(wsb + L.tsum);
  float *ztgt = (float *)(wsb + L.ztgt), *lse = (float *)(wsb + L.lse);
  hipError_t e;
  {
    Timed t(K_HEAD_GATHER, st);
    e = launch_gather_rows(h, D, (int)T, rows, (int)nrows, (int)D, hT, st);
    if (e == hipSuccess) e = launch_gather_rows(W, D, (int)V, J, (int)nJ, (int)D, WJ, st);
    t.done();
    if (e != hipSuccess) return hip_fail(e, "head_gather launch");
  }
  // logits z = h_T W_J^T, never stored: per-tile row max / sum of exp, target logit
  GemmArgs g{};
  g.A = hT; g.lda = D;
  g.B = WJ; g.ldb = D;
  g.M = (int)nrows; g.N = (int)nJ; g.K = (int)D;
  g.tpos = tpos; g.col0 = 0;
  g.ce_max = tmax; g.ce_sum = tsum; g.ce_tgt = ztgt;
  {
    Timed t(K_HEAD_LOGITS, st);
    e = launch_fill_nan(ztgt, nrows, st);  // a target outside J leaves its loss NaN
    if (e == hipSuccess) e = launch_gemm_epi(g, EPI_CE_STATS, st);
    if (e == hipSuccess)
      e = launch_ce_combine(tmax, tsum, (int)L.tiles, (int)nrows, ztgt, lse, loss_rows, loss_total, st);
    t.done();
    if (e != hipSuccess) return hip_fail(e, "head_logits launch");
  }
  if (!dh) return LORA_OK;
  // dh_T = sum over chunks of the vocabulary of dz_chunk W_J[chunk], with
  // dz = dscale (softmax - one-hot(target)) recomputed per chunk.
  const int64_t ch = nJ < kHeadChunk ? (nJ + 7) / 8 * 8 : kHeadChunk;
  float *dhacc = (float *)(wsb + L.dhacc);
  for (int64_t c0 = 0; c0 < nJ; c0 += ch) {
    const int64_t w = std::min<int64_t>(ch, nJ - c0);
    const int64_t ldz = (w + 7) / 8 * 8;
    GemmArgs z{};
    z.A = hT; z.lda = D;
    z.B = (const char *)WJ + c0 * D * 2; z.ldb = D;
    z.M = (int)nrows; z.N = (int)w; z.K = (int)D;
    z.C = wsb + L.dz; z.ldc = ldz;
    z.tpos = tpos; z.col0 = (int)c0; z.lse = lse; z.dscale = dscale;
    {
      Timed t(K_HEAD_DZ, st);
      e = launch_gemm_epi(z, EPI_CE_DZ, st);
      t.done();
      if (e != hipSuccess) return hip_fail(e, "head_dz launch");
    }
    GemmArgs d{};
    d.A = wsb + L.dz; d.lda = ldz;
    d.B = (const char *)WJ + c0 * D * 2; d.ldb = D;
    d.M = (int)nrows; d.N = (int)D; d.K = (int)w;
    d.C = dhacc; d.ldc = D; d.c_accumulate = c0 > 0;
    Timed t(K_HEAD_DH, st);
    e = launch_gemm_epi(d, EPI_F32, st);
    t.done();
    if (e != hipSuccess) return hip_fail(e, "head_dh launch");
  }
  Timed t(K_HEAD_DH, st);
  e = launch_dh_finish(dhacc, rows, (int)nrows, (int32_t *)(wsb + L.inv), (int)T, (int)D, dh, st);
  t.done();
  return e == hipSuccess ? LORA_OK : hip_fail(e, "head_dh launch");
}

size_t topk_table_workspace_bytes(int64_t V, int64_t D, int64_t k) {
  if (V < 1 || D < 8 || D % 8 || k < 1 || k > std::min<int64_t>(V, 2048) || D > kMaxDim ||
      V > kMaxElems / D || V > kMaxElems / k)
    return (size_t)-1;
  return topk_layout(V, k).total;
}

lora_status_t topk_table_build(const void *W, int64_t V, int64_t D, int64_t k, int32_t *table,
                               float *values, void *ws, size_t ws_bytes, void *hip_stream) {
  if (!W || !table) return fail(LORA_EINVAL, "W and table are required");
  if (V < 1 || k < 1 || k > std::min<int64_t>(V, 2048))
    return fail(LORA_EINVAL, "need V >= 1 and 1 <= k <= min(V, 2048)");
  if (D < 8 || D % 8) return fail(LORA_EUNSUPPORTED, "D must be a positive multiple of 8");
  if (D > kMaxDim || V > kMaxElems / D || V > kMaxElems / k)
    return fail(LORA_EUNSUPPORTED, "D at most 2^20 and W, table below 2^31 elements");
  if (!aligned16(W) || !aligned16(table) || (values && !aligned16(values)))
    return fail(LORA_EINVAL, "pointers must be 16-byte aligned");
  const TopkLayout L = topk_layout(V, k);
  lora_status_t s;
  if ((s = check_ws(ws, ws_bytes, L.total)) != LORA_OK) return s;
  std::vector<Range> ins = {rng(W, V * D * 2)};
  std::vector<Range> outs = {rng(table, V * k * 4), rng(ws, (int64_t)L.total)};
  if (values) outs.push_back(rng(values, V * k * 4));
  if (any_overlap(outs, ins)) return fail(LORA_EINVAL, "an output overlaps an input or another output");
  hipStream_t st = (hipStream_t)hip_stream;
  char *wsb = (char *)ws;
  float *rn = (float *)(wsb + L.rn);
  TopkArgs ta{};
  ta.val = (float *)(wsb + L.val); ta.idx = (int32_t *)(wsb + L.idx);
  ta.cnt = (int *)(wsb + L.cnt); ta.thr = (float *)(wsb + L.thr);
  ta.cap = (int)L.cap; ta.k = (int)k; ta.lazy = (int)L.lazy; ta.table = table; ta.tvals = values;
  hipError_t e;
  {
    Timed t(K_TOPK_SIM, st);
    e = launch_row_rnorm(W, (int)V, (int)D, rn, st);
    t.done();
    if (e != hipSuccess) return hip_fail(e, "topk_sim launch");
  }
  for (int64_t r0 = 0; r0 < V; r0 += L.R) {
    const int rb = (int)std::min<int64_t>(L.R, V - r0);
    if ((e = launch_topk_reset(ta.thr, ta.cnt, rb, st)) != hipSuccess) return hip_fail(e, "topk reset");
    ta.row0 = r0;
    for (int64_t c0 = 0; c0 < V; c0 += kTopkChunk) {
      GemmArgs g{};
      g.A = (const char *)W + r0 * D * 2; g.lda = D;
      g.B = (const char *)W + c0 * D * 2; g.ldb = D;
      g.M = rb; g.N = (int)std::min<int64_t>(kTopkChunk, V - c0); g.K = (int)D;
      g.col0 = (int)c0; g.rn_a = rn + r0; g.rn_b = rn + c0;
      g.tk_thr = ta.thr; g.tk_cnt = ta.cnt; g.tk_val = ta.val; g.tk_idx = ta.idx;
      g.tk_cap = (int)L.cap;
      {
        Timed t(K_TOPK_SIM, st);
        e = launch_gemm_epi(g, EPI_TOPK, st);
        t.done();
        if (e != hipSuccess) return hip_fail(e, "topk_sim launch");
      }
      const int final = c0 + kTopkChunk >= V;
      Timed t(K_TOPK_SELECT, st);
      e = launch_topk_select(ta, rb, final, st);
      t.done();
      if (e != hipSuccess) return hip_fail(e, "topk_select launch");
    }
  }
  return LORA_OK;
}

lora_status_t lora_linear_plan(int64_t T, int64_t d_in, int64_t d_out, int64_t r, lora_dtype_t dt,
                               lora_plan_t *plan) {
  if (!plan) return fail(LORA_EINVAL, "plan is NULL");
  lora_status_t s = check_shapes(T, d_in, d_out, r, dt);
  if (s != LORA_OK) return s;
  const Dtype d = dt == LORA_BF16 ? DT_BF16 : DT_F32;
  lora_plan_t p{};
  gemm_tile_shape((int)T, (int)d_out, false, false, d, &p.fwd_tile_m, &p.fwd_tile_n);
  gemm_tile_shape((int)T, (int)d_in, true, r > 0, d, &p.bwd_tile_m, &p.bwd_tile_n);
  if (r > 0) {
    const FwdLayout F = fwd_layout(T, d_in, d_out, r, dt);
    const BwdLayout B = bwd_layout(T, d_in, d_out, r, dt);
    p.fwd_fused = F.fused;
    p.fwd_u_parts = F.sp.nsplit;
    p.bwd_fused = B.fused;
    p.bwd_du_parts = B.sp_du.nsplit;
    p.bwd_side_parts = B.tparts;
  }
  *plan = p;
  return LORA_OK;
}

lora_status_t lora_handover_giveups(uint64_t *count, int reset) {
  if (!count) return fail(LORA_EINVAL, "count is NULL");
  unsigned c = 0;
  hipError_t e = handover_giveups(&c, reset != 0);
  if (e != hipSuccess) return hip_fail(e, "reading the hand-over give-up count");
  *count = c;
  return LORA_OK;
}

lora_status_t lora_debug_set_handover(int hold) {
  if (hold != 0 && hold != 1) return fail(LORA_EINVAL, "hold must be 0 or 1");
  g_fz_hold.store(hold);
  return LORA_OK;
}

const char *lora_status_str(lora_status_t status) {
  switch (status) {
    case LORA_OK: return "ok";
    case LORA_EINVAL: return "invalid argument";
    case LORA_EUNSUPPORTED: return "unsupported shape";
    case LORA_EWORKSPACE: return "workspace missing or too small";
    case LORA_EHIP: return "HIP launch error";
  }
  return "unknown status";
}

const char *lora_last_error(void) { return g_err; }

lora_status_t lora_profiler_enable(int on) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_on = on != 0;
  return LORA_OK;
}

lora_status_t lora_profiler_reset(void) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (auto &v : g_prof) {
    for (auto &p : v) {
      (void)hipEventDestroy(p.a);
      (void)hipEventDestroy(p.b);
    }
    v.clear();
  }
  return LORA_OK;
}

lora_status_t lora_profiler_read(int kernel_id, double *total_ms, int64_t *launches) {
  if (kernel_id < 0 || kernel_id >= K_COUNT || !total_ms || !launches)
    return fail(LORA_EINVAL, "bad kernel id or NULL output");
  std::vector<EventPair> recs;
  {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    recs = g_prof[kernel_id];
  }
  double sum = 0.0;
  for (auto &p : recs) {
    hipError_t e = hipEventSynchronize(p.b);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    float ms = 0.0f;
    e = hipEventElapsedTime(&ms, p.a, p.b);
    if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
    sum += ms;
  }
  *total_ms = sum;
  *launches = (int64_t)recs.size();
  return LORA_OK;
}

const char *lora_kernel_name(int kernel_id) {
  return (kernel_id >= 0 && kernel_id < K_COUNT) ? kKernelNames[kernel_id] : nullptr;
}

int lora_kernel_count(void) { return K_COUNT; }

}  // extern "C"
