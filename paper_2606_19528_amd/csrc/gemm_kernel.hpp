// gemm_kernel.hpp -- LDS-tiled matrix-core GEMM for the two big contractions of the
// LoRA linear, each with the rank-r LoRA term folded in as extra reduction
// steps (so y and dx are rounded exactly once):
//   forward   y  = [x | s*u] [W | B]^T          (NT: both operands k-contiguous)
//   backward  dx = [dy | du] [W ; A]            (NN: W and A are k-major, i.e.
//                                                 the reduction index is the row)
//   frozen    dx = dy W                          (NN, no tail)
//
// Structure of one workgroup (4 or 8 waves, one BM x BN output tile):
//  * k advances in stages of BKB bytes per row.  Global loads go through
//    buffer resources (hardware bounds checks instead of per-load branches).
//  * DMA = 1 or 2 (every bf16 tile shape; 2 with producer workgroups of a
//    fused rank-r pass in front): the loads write LDS directly
//    (buffer_load ... lds), into a ring of NBUF stages with NBUF - 1 stages
//    in flight behind the one being read; no registers or LDS-write
//    instructions are spent on staging.  One load moves 1 KB in lane order, so
//    the lanes pick their source chunks to produce an XOR-swizzled layout whose
//    fragment reads are bank-conflict free.  With a quantized B (QB = 4 or 8,
//    DMA = 1) the codes, scales and offsets are loaded into LDS the same way,
//    into slots of their own, and each step dequantizes one stage from them
//    into the bf16 B area of the ring.
//  * DMA = 0: loads go into a ring of RD register sets, then into an LDS ring
//    of NBUF buffers; a stage's loads are issued RD - 1 steps before its LDS
//    write, which covers the latency of reads that miss L2 (the fp32 check
//    mode, and a quantized B with groups of fewer than 64 weights, which is
//    dequantized in registers on the way into LDS).
//  * NBUF = 3: a stage is written to LDS two steps before it is consumed, so
//    the first k-slice's MFMA fragments of the next stage can be read before
//    the end-of-step barrier and the MFMAs of a step start without waiting on
//    LDS.  NBUF = 2: classic double buffering.  One barrier per step.
//  * The waves form a WM x WN x WK grid: WM x WN split the tile, WK splits
//    each stage's 16-deep k-slices; with WK > 1 the partial accumulators are
//    summed through LDS in a fixed order at the end.
//  * k-major operands (W and A in the backward pass) keep their memory layout
//    in LDS ([k][n]) and are read with ds_read_b64_tr_b16, which hands each
//    lane four consecutive k of one column (bf16).  In the fp32 check mode
//    they are transposed in registers on the way into LDS instead.
//  * Workgroups are mapped to tiles XCD by XCD (the dispatcher deals workgroup
//    ids round-robin over the 8 XCDs, each with its own L2), and each XCD's
//    share of tiles is a compact block of GM tile rows.
#pragma once

#include <type_traits>

#include "colred.hpp"
#include "rowprod.hpp"
#include "kernels.hpp"
#include "launch.hpp"

namespace lora {

enum { B_ROW = 0, B_KMAJ_REG = 1, B_KMAJ_TR = 2 };

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// ---- hand-over of a fused rank-r pass (protocol in launch.hpp, FuseArgs) ------
constexpr unsigned long long FZ_BUDGET = 20000000ull;  // 0.2 s of the 100 MHz real-time counter

// Waits that gave up (their condition not met within FZ_BUDGET), summed over
// every launch on this device; read and cleared from the host
// (handover_giveups).  A give-up means the launch may have computed with
// incomplete producer rows.
static __device__ unsigned int g_fz_giveups;

// A wait that gives up marks its wave by raising the wave's scheduling
// priority (s_setprio), a flag that costs no register while the tile's
// main loop still runs; fz_report counts marked waves once their work is
// done.  (Every other form of recording at the point of the give-up --
// a store, an atomic, an extra live value -- made the fused kernels spill.)
constexpr int FZ_MARK = 3;
__device__ __forceinline__ void fz_mark() { __builtin_amdgcn_s_setprio(FZ_MARK); }
// The wave's user priority: bits 4:3 of the STATUS hardware register.
__device__ __forceinline__ int fz_prio() {
  return __builtin_amdgcn_s_getreg((1 << 11) | (3 << 6) | 2);  // size 2, offset 3, STATUS
}
// After a wave's last use of producer data: count it if a wait of it gave up,
// and drop the mark.
__device__ __forceinline__ void fz_report() {
  if (fz_prio() == FZ_MARK) {
    if ((threadIdx.x & 63) == 0)
      __hip_atomic_fetch_add(&g_fz_giveups, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __builtin_amdgcn_s_setprio(0);
  }
}

__device__ __forceinline__ unsigned long long fz_load(unsigned long long *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Workgroup 0, one thread, before its work: tag the launch, then open it.
__device__ __forceinline__ void fz_arm(unsigned long long *sync, unsigned gen) {
  __hip_atomic_store(sync, (unsigned long long)gen << 32, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(sync + 1, 0ull, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}
// A producer, one thread, after every wave's stores have completed: count
// this producer once the launch is open.
__device__ __forceinline__ void fz_produced(unsigned long long *sync, unsigned gen) {
  const unsigned long long t0 = __builtin_amdgcn_s_memrealtime();
  for (;;) {
    if (fz_load(sync + 1) == 0 && (fz_load(sync) >> 32) == gen) break;
    if (__builtin_amdgcn_s_memrealtime() - t0 > FZ_BUDGET) {
      fz_mark();
      break;
    }
    __builtin_amdgcn_s_sleep(4);
  }
  __hip_atomic_fetch_add(sync, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// A consumer wave, before it reads producer data: wait until every producer
// of this launch has counted itself (ncons 0: never -- a test's way of
// forcing every wait to give up).
__device__ __forceinline__ void fz_wait(unsigned long long *sync, unsigned gen, int nprod, int ncons) {
  const unsigned long long t0 = __builtin_amdgcn_s_memrealtime();
  for (;;) {
    if (fz_load(sync + 1) < (unsigned long long)ncons) {
      const unsigned long long v = fz_load(sync);
      if ((v >> 32) == gen && (unsigned)v >= (unsigned)nprod) break;
    }
    if (__builtin_amdgcn_s_memrealtime() - t0 > FZ_BUDGET) {
      fz_mark();
      break;
    }
    __builtin_amdgcn_s_sleep(4);
  }
}
// A producer that then runs side items, one thread, after counting itself:
// wait until every producer of this launch has counted itself.  Its own
// count followed this launch's arming, so the count it reads is this
// launch's and no condition on the tiles' count is needed.
__device__ __forceinline__ void fz_wait_producers(unsigned long long *sync, unsigned gen, int nprod) {
  const unsigned long long t0 = __builtin_amdgcn_s_memrealtime();
  for (;;) {
    const unsigned long long v = fz_load(sync);
    if ((v >> 32) == gen && (unsigned)v >= (unsigned)nprod) break;
    if (__builtin_amdgcn_s_memrealtime() - t0 > FZ_BUDGET) {
      fz_mark();
      break;
    }
    __builtin_amdgcn_s_sleep(4);
  }
}
// A producer about to run side items, after its wait has seen every
// producer's count: invalidate the caches that could hold lines older than
// the other producers' device-scope stores of du (this CU's vector L1, and
// the L2 lines not kept coherent across XCDs) -- the cache action of a
// device-scope acquire, without its wait for every load in flight (the
// count's own load has returned: its value decided the wait).  64 producers
// pay it at no measurable cost; in the tiles it cost 10 us per launch at
// T = 1024, so they rely on the argument in launch.hpp (FuseArgs) instead.
__device__ __forceinline__ void fz_acquire() { asm volatile("buffer_inv sc1" ::: "memory"); }
// A consumer, one thread, once it has passed.
__device__ __forceinline__ void fz_done(unsigned long long *sync) {
  __hip_atomic_fetch_add(sync + 1, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

constexpr int cmax(int a, int b) { return a > b ? a : b; }

template <int V>
struct IC {
  static constexpr int value = V;
};

// Calls f(IC<I>()) for I = B .. E-1.
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F &&f) {
  if constexpr (B < E) {
    f(IC<B>());
    static_for<B + 1, E>(f);
  }
}

template <class E, int BM, int BN, int WM, int WN, int WK, int BMODE, int BKB, int NBUF, int RD, int FS,
          int QB = 0, int EPI = EPI_STORE, int DMA = 0>
__global__ __launch_bounds__(64 * WM * WN * WK) void gemm_kernel(GemmArgs g, int group_m,
                                                                 SideArgs side, int nside,
                                                                 FuseArgs fz) {
  typedef typename E::T T;
  constexpr int NT = 64 * WM * WN * WK;
  constexpr int VEC = E::VEC;
  constexpr int ES = (int)sizeof(T);
  constexpr int BKE = BKB / ES;              // k elements per stage
  constexpr int SLICES = BKB / 32;           // k-slices of 32 bytes per stage
  constexpr int SPW = SLICES / WK;           // slices per wave
  constexpr int ROWA = BKB + 16;             // padded LDS row of a k-contiguous operand
  constexpr int ROWT = BN * 2 + 32;          // padded LDS row of a k-major bf16 operand
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int FM = WTM / 32, FN = WTN / 32, NB = FM * FN;
  constexpr int CPR = BKB / 16;              // 16-byte chunks per k-contiguous row
  constexpr int A_CH = BM * CPR, A_PER = (A_CH + NT - 1) / NT;
  constexpr int NBV = BN / VEC;
  constexpr int B_CH = BMODE == B_KMAJ_TR ? BKE * NBV : BN * CPR;
  constexpr int B_PER = (B_CH + NT - 1) / NT;
  constexpr int KB_BLK = (BKE / VEC) * NBV, KB_PER = (KB_BLK + NT - 1) / NT;
  constexpr int RB = BMODE == B_KMAJ_REG ? KB_PER * VEC : B_PER;
  constexpr int A_BYTES = BM * ROWA;
  constexpr int B_BYTES = BMODE == B_KMAJ_TR ? BKE * ROWT : BN * ROWA;
  constexpr int STAGE = A_BYTES + B_BYTES;
  constexpr int OWN = (NB + WK - 1) / WK;    // accumulator blocks owned per wave (k-split)
  constexpr int RED_BYTES = WK > 1 ? WM * WN * WK * OWN * 4096 : 0;
  // Direct-to-LDS stages (DMA): unpadded rows, chunks swizzled (see dma_stage).
  constexpr int NWV = NT / 64;
  // Row-major B is loaded in whole loads per wave (rows past BN read zeros);
  // k-major B rows take 256 bytes in LDS (columns past BN read zeros).
  constexpr int DB_ROWS = (BN + (1024 / BKB) * NWV - 1) / ((1024 / BKB) * NWV) * ((1024 / BKB) * NWV);
  constexpr int DBRB = (BN * 2 + 255) / 256 * 256;
  constexpr int DA_BYTES = BM * BKB;
  constexpr int DB_BYTES = BMODE == B_KMAJ_TR ? BKE * DBRB : DB_ROWS * BKB;
  constexpr int DSTAGE = DA_BYTES + DB_BYTES;
  constexpr int DA_PW = DA_BYTES / 1024 / NWV, DB_PW = DB_BYTES / 1024 / NWV;  // loads per wave per stage
  constexpr int IPS = DA_PW + DB_PW;
  // Quantized B on the direct-to-LDS path (DMA = 1, QB = 4 or 8; groups of at
  // least 64 weights, so a stage of a row-major B holds one group per row):
  // the stage's codes and the scales and offsets it needs are loaded straight
  // into LDS too, into a ring of three slots of their own, two stages ahead
  // of the stage's A loads; each step then dequantizes one stage from its
  // slot into the bf16 B area of the ring (same layout as the bf16 path).
  // A code slot holds the stage's runs of 16 weights (one W row, one group)
  // in order: row-major B run = tile row * (BKE / 16) + k / 16, k-major B run
  // = k row * (BN / 16) + n / 16, at 2 * QB bytes each.  Scales and offsets
  // (group-major in memory, so those of one group and consecutive W rows are
  // contiguous): k-major B, one slot per stage holding, per group touched by
  // the tile's columns, its BKE k rows (group - first group) * BKE + k row;
  // row-major B, whose tile rows keep a group for G / BKE stages, one slot
  // per group (group % 4) holding the group's BN tile rows, loaded with the
  // codes of the group's first stage.  Wave 0 issues them (two 16-byte
  // loads), first in their step, and only in the steps that have some; the
  // wait at the top of the next step counts them only where that step
  // issued them.
  constexpr bool QD = DMA == 1 && QB != 0;
  constexpr int QCW = QD ? 128 / QB : 16;                               // weights per 16-byte code chunk
  constexpr int QCHUNKS = QD ? BKE * BN / QCW : 0;                      // code chunks per stage
  constexpr int QC_PW = (QCHUNKS + 64 * NWV - 1) / (64 * NWV);          // code loads per wave per stage
  constexpr int QSLOT = QC_PW * NWV * 1024;                             // bytes of a code slot
  constexpr int QSO = 1024;                                             // bytes of a slot's scales (or offsets)
  constexpr int QRUNS = QD ? BKE * BN / 16 : 0;                         // runs of 16 weights per stage
  constexpr int QRPT = QD ? (QRUNS + NT - 1) / NT : 1;                  // runs per thread
  constexpr int QIPS = QC_PW + DA_PW;                                   // counted loads per wave per step
  constexpr int QSOSLOTS = BMODE == B_ROW ? 4 : 3;                        // scale / offset slots
  constexpr int QAREA = QD ? 3 * QSLOT + QSOSLOTS * 2 * QSO : 0;
  constexpr int RING = DMA ? NBUF * DSTAGE + QAREA : NBUF * STAGE;
  constexpr int LDS0 = RING > RED_BYTES ? RING : RED_BYTES;
  constexpr int SIDE = side_lds_bytes<E, WM * WN * WK>();
  // Producer workgroups of a fused rank-r pass ahead of the bf16
  // direct-to-LDS tiles: u = x A^T (forward, row-major A) or du = s dy B
  // (backward, k-major B).
  // (DMA = 2: a separate instance, so launches without producers carry none
  // of their code or registers.)
  constexpr bool FUSE = DMA == 2;
  static_assert(!FUSE || (QB == 0 && EPI == EPI_STORE && ES == 2 && (BMODE == B_ROW || BMODE == B_KMAJ_TR)),
                "producers: bf16 direct-to-LDS tiles that store C");
  constexpr int PV = BMODE == B_ROW ? V_ROW : V_KMAJ_TR;
  // (Only the 256 x 256 tiles, which leave 64 CUs to the producers at 4096
  // rows, need producers of 64 rows.)
  constexpr bool PROD4 = FUSE && BM == 256 && BN == 256;
  constexpr int PNW = NT / 64;  // the producers' waves: the tile's
  constexpr int PROD =
      FUSE ? cmax(cmax(cmax(row_lds_bytes<E, 1, PV, 4, 1, PNW>(), row_lds_bytes<E, 2, PV, 4, 1, PNW>()),
                       cmax(row_lds_bytes<E, 1, PV, 4, 2, PNW>(), row_lds_bytes<E, 2, PV, 4, 2, PNW>())),
                  PROD4 ? cmax(row_lds_bytes<E, 1, PV, 4, 4, PNW>(), row_lds_bytes<E, 2, PV, 4, 4, PNW>()) : 0)
           : 0;
  constexpr int LDS1 = LDS0 > SIDE ? LDS0 : SIDE;
  constexpr int LDS = LDS1 > PROD ? LDS1 : PROD;
  constexpr uint32_t OOB = 0x80000000u;      // offset past every buffer: loads return 0
  static_assert(WM * WN * WK == 4 || WM * WN * WK == 8, "four or eight waves");
  static_assert(SLICES % WK == 0, "k split");
  static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tile");
  static_assert(BMODE != B_KMAJ_TR || ES == 2, "transposed LDS reads are bf16");
  static_assert(DMA ? (NBUF == 3 || NBUF == 4) : (NBUF == 2 || NBUF == 3), "LDS ring depth");
  static_assert(!QD || (NBUF == 3 && BN <= 256 && (BN / 64 + 1) * BKE <= 256 && QCW * QC_PW * 64 * NWV >= BKE * BN &&
                        QRUNS * 2 * QB <= QSLOT && QRPT * NT * 2 * QB <= QSLOT && EPI == EPI_STORE &&
                        BKE % 16 == 0 && BN % 16 == 0 && QIPS < 64),
                "quantized direct-to-LDS stages: a ring of three, whole runs of 16 weights");
  static_assert(!DMA || ((QB == 0 || DMA == 1) && ES == 2 && FS == 2 && (BKB == 128 || BKB == 64) && BMODE != B_KMAJ_REG &&
                         DA_BYTES % (1024 * NWV) == 0 && DB_BYTES % (1024 * NWV) == 0 &&
                         (BMODE != B_KMAJ_TR || DBRB == 256 || DBRB == 512)),
                "direct-to-LDS stages: bf16, 64- or 32-deep stages, whole 1 KB loads per wave");
  static_assert(RD >= 2 && RD <= 4, "register ring depth");
  static_assert(!FS || DMA || NBUF == 2, "staged fragments use two LDS buffers");
  // Quantized B (QB = 4 or 8 bits): each thread dequantizes one piece of 16
  // consecutive weights of a W row per stage.
  constexpr int QPIECES = BMODE == B_ROW ? BN * (BKE / 16) : BKE * (BN / 16);
  static_assert(QB == 0 || QB == 4 || QB == 8, "code width");
  static_assert(EPI == EPI_STORE || (ES == 2 && FS), "cross-entropy / fp32 epilogues: bf16 kernels");
  static_assert((EPI != EPI_CE_STATS && EPI != EPI_TOPK) || (NT == 4 * BM && BM * (BN + 1) * 4 + BN * 4 <= LDS),
                "row statistics / candidates: four threads per tile row, the fp32 tile in LDS");
  static_assert(QB == 0 || QD || (ES == 2 && FS && BMODE != B_KMAJ_REG && QPIECES == NT),
                "quantized B: bf16, staged fragments, one 16-weight piece per thread");

  __shared__ __align__(16) char smem[LDS];
  auto ring_a = [&](auto BUF) -> char * { return smem + decltype(BUF)::value * DSTAGE; };
  auto ring_b = [&](auto BUF) -> char * { return smem + decltype(BUF)::value * DSTAGE + DA_BYTES; };

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wk = wave % WK;
  const int wn = (wave / WK) % WN;
  const int wm = wave / (WK * WN);

  // ---- tile of this workgroup: XCD-contiguous, grouped by GM tile rows ----
  const int tiles_m = (g.M + BM - 1) / BM;
  const int tiles_n = (g.N + BN - 1) / BN;
  const int ntiles = tiles_m * tiles_n;
  // The first `nside` workgroups (a multiple of 8, so the XCD of a tile
  // workgroup is unchanged) run the token-reduction side items; they start
  // first and overlap with the tiles.
  // With a fused rank-r pass, the `fz.nwg` producer workgroups come first.
  const bool coh = FUSE && fz.nprod > 0;
  const int bid = (int)blockIdx.x - (FUSE ? fz.nwg : 0);
  if constexpr (FUSE) {
    if (bid < 0) {
      if ((int)blockIdx.x < fz.nprod) {
        if (blockIdx.x == 0 && tid == 0) fz_arm(fz.sync, fz.gen);
        // Coherent stores, complete in every wave before the count: no L2
        // write-back (which would stall every tile of the XCD) is needed.
        auto prod = [&](auto JB, auto MB) {
          row_item<E, decltype(JB)::value, PV, 4, decltype(MB)::value, true, NT / 64>(fz.row, blockIdx.x, 0, fz.nprod, 1,
                                                                             smem);
        };
        if (fz.row.r <= 16) {
          if (PROD4 && fz.row.mb == 4) prod(IC<1>(), IC<PROD4 ? 4 : 1>());
          else if (fz.row.mb == 2) prod(IC<1>(), IC<2>());
          else prod(IC<1>(), IC<1>());
        } else {
          if (PROD4 && fz.row.mb == 4) prod(IC<2>(), IC<PROD4 ? 4 : 1>());
          else if (fz.row.mb == 2) prod(IC<2>(), IC<2>());
          else prod(IC<2>(), IC<1>());
        }
        __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
        __syncthreads();
        if (tid == 0) fz_produced(fz.sync, fz.gen);
        // Backward: the producers then run the dA / dB side items (dA needs
        // all of du), on CUs the tiles leave to them.
        const int nitems = BMODE == B_KMAJ_TR ? side_items_total<E>(side) : 0;
        if constexpr (BMODE == B_KMAJ_TR) if (nitems > 0) {
          if (tid == 0) {
            fz_wait_producers(fz.sync, fz.gen, fz.nprod);
            fz_acquire();
          }
          __syncthreads();
          for (int it = blockIdx.x; it < nitems; it += fz.nprod) {
            side_item<E, WM * WN * WK, false>(side, it, smem);
            __syncthreads();
          }
        }
        fz_report();
      }
      return;
    }
  }
  // (A fused launch runs its side items on the producers: nside = 0.  Only
  // the dx launches, k-major B, carry side items.)
  if constexpr (!FUSE && BMODE != B_ROW) {
    if (bid < nside) {
      if (bid < side_items_total<E>(side)) side_item<E, WM * WN * WK, true>(side, bid, smem);
      return;
    }
  }
  int t;
  {
    const int id = bid - nside;
    const int xcd = id & 7, local = id >> 3;
    const int base = ntiles >> 3, rem = ntiles & 7;
    t = xcd * base + (xcd < rem ? xcd : rem) + local;
  }
  const int gsize = group_m * tiles_n;
  const int first_m = (t / gsize) * group_m;
  const int gm = min(tiles_m - first_m, group_m);
  const int mt = first_m + (t % gsize) % gm;
  const int nt = (t % gsize) / gm;
  const int m0 = mt * BM, n0 = nt * BN;

  // Optional sum of partial rank-r products for the rows of this tile row:
  // its BM x r elements are shared out over the tile row's workgroups, one
  // per thread; the loads are issued here and the sum stored after the main
  // loop, so their latency is hidden.
  // (Tiles larger than 128 x 128 have no registers to spare across the loop:
  // they issue the loads after it.)
  constexpr bool US_EARLY = BM * BN <= 128 * 128;
  float us_part[MAX_SPLIT];
  int64_t us_idx = -1;
  int us_first = 0, us_last = 0;
  auto us_load = [&]() {
    const int64_t plane = (int64_t)g.M * g.usum_r;
#pragma unroll
    for (int q = 0; q < MAX_SPLIT; ++q) us_part[q] = q < g.usum_parts ? g.usum_src[q * plane + us_idx] : 0.0f;
  };
  // Only the forward GEMM (row-major B) carries this job.
  if (BMODE == B_ROW && g.usum_out) {
    const int total = min(BM, g.M - m0) * g.usum_r;
    const int chunk = (total + tiles_n - 1) / tiles_n;
    us_first = nt * chunk + tid;
    us_last = min(total, (nt + 1) * chunk);
    if (us_first < us_last) {
      us_idx = (int64_t)(m0 + us_first / g.usum_r) * g.usum_r + us_first % g.usum_r;
      if constexpr (US_EARLY) us_load();
    }
  }

  const int nk_main = (g.K + BKE - 1) / BKE;
  const int nk_lora = g.r > 0 ? (g.r + BKE - 1) / BKE : 0;
  const int nk = nk_main + nk_lora;
  // Stage order: the LoRA steps follow the main ones, except with a quantized
  // B, where they come first (stage 0, loaded and stored by the prologue), so
  // that the main loop only ever runs the dequantizing path.

  // Buffer resources.  The tile's rows past M (and, for row-major B, past N)
  // lie beyond num_records; k past K (or j past r) is masked per stage by
  // selecting OOB.  The LoRA step reads A2 / B2 through resources of its own.
  const int mrows = min(g.M - m0, BM);
  const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc(
      (void *)((const char *)g.A + (int64_t)m0 * g.lda * ES), (short)0, (int)(mrows * g.lda * ES),
      0x00020000);
  const __amdgpu_buffer_rsrc_t rsA2 = __builtin_amdgcn_make_buffer_rsrc(
      (void *)((const char *)g.A2 + (int64_t)m0 * g.lda2 * ES), (short)0,
      g.r > 0 ? (int)(mrows * g.lda2 * ES) : 0, 0x00020000);
  __amdgpu_buffer_rsrc_t rsB, rsB2;
  if constexpr (BMODE == B_ROW) {
    const int nrows = min(g.N - n0, BN);
    rsB = __builtin_amdgcn_make_buffer_rsrc((void *)((const char *)g.B + (int64_t)n0 * g.ldb * ES),
                                            (short)0, (int)(nrows * g.ldb * ES), 0x00020000);
    rsB2 = __builtin_amdgcn_make_buffer_rsrc(
        (void *)((const char *)g.B2 + (int64_t)n0 * g.ldb2 * ES), (short)0,
        g.r > 0 ? (int)(nrows * g.ldb2 * ES) : 0, 0x00020000);
  }
  // k-major B whole (columns of the tile from n0), for the loads of full main
  // stages: their k-rows all lie below K, the stage start goes in soffset.
  __amdgpu_buffer_rsrc_t rsBk;
  if constexpr (BMODE == B_KMAJ_TR)
    rsBk = __builtin_amdgcn_make_buffer_rsrc((void *)((const char *)g.B + (int64_t)n0 * ES), (short)0,
                                             (int)((int64_t)g.K * g.ldb * ES), 0x00020000);
  uint32_t va[A_PER], va2[A_PER], vb[BMODE == B_KMAJ_REG ? KB_PER : B_PER], vb2[B_PER];
  int kca[A_PER], kcb[B_PER];
#pragma unroll
  for (int i = 0; i < A_PER; ++i) {
    const int c = tid + i * NT;
    kca[i] = (c % CPR) * VEC;
    va[i] = c < A_CH ? (uint32_t)((c / CPR) * g.lda * ES + (c % CPR) * 16) : OOB;
    va2[i] = c < A_CH ? (uint32_t)((c / CPR) * g.lda2 * ES + (c % CPR) * 16) : OOB;
  }
  if constexpr (BMODE == B_ROW) {
#pragma unroll
    for (int i = 0; i < B_PER; ++i) {
      const int c = tid + i * NT;
      kcb[i] = (c % CPR) * VEC;
      vb[i] = c < B_CH ? (uint32_t)((c / CPR) * g.ldb * ES + (c % CPR) * 16) : OOB;
      vb2[i] = c < B_CH ? (uint32_t)((c / CPR) * g.ldb2 * ES + (c % CPR) * 16) : OOB;
    }
  } else if constexpr (BMODE == B_KMAJ_TR) {
#pragma unroll
    for (int i = 0; i < B_PER; ++i) {
      const int c = tid + i * NT;
      const int kr = c / NBV, nc = c % NBV;
      vb[i] = (c < B_CH && n0 + nc * VEC < g.N) ? (uint32_t)(kr * g.ldb * ES + nc * 16) : OOB;
      vb2[i] = (c < B_CH && n0 + nc * VEC < g.N) ? (uint32_t)(kr * g.ldb2 * ES + nc * 16) : OOB;
    }
  } else {
#pragma unroll
    for (int i = 0; i < KB_PER; ++i) {
      const int b = tid + i * NT;
      const int kb = b % (BKE / VEC), nb = b / (BKE / VEC);
      vb[i] = (b < KB_BLK && n0 + nb * VEC < g.N) ? (uint32_t)(kb * VEC * g.ldb * ES + nb * 16)
                                                   : OOB;
    }
  }

  // Direct-to-LDS loads: one load instruction of a wave moves 64 x 16 bytes
  // into 1 KB of LDS in lane order, so the LDS layout is fixed and the lanes
  // choose which global chunk lands where.  k-contiguous operands (A; B when
  // row-major): load q of a stage covers tile rows RPK q .. RPK q + RPK - 1
  // (RPK = 8 rows of BKB = 128 bytes, or 16 rows of 64 bytes), and row r keeps
  // its 16-byte chunk c at chunk c ^ swz(r): swz(r) = (r & 7) ^ ((r >> 3) & 1)
  // for 128-byte rows, (r >> 2) & 3 for 64-byte rows, which puts the fragment
  // reads of sixteen consecutive rows in distinct banks.  k-major B: load q
  // covers k-rows KPK q .. KPK q + KPK - 1 (DBRB = 256 or 512 bytes each, KPK
  // = 4 or 2), chunk c at c ^ 4 (r & 3).
  // (Written out per layout: the general forms cost the fused kernels
  // registers, and spills, that these do not.)
  auto chunk_row = [&](int q, int &r, int &c) __attribute__((always_inline)) {
    if constexpr (CPR == 8) {
      r = 8 * q + (lane >> 3);
      c = (lane & 7) ^ (lane >> 3) ^ (q & 1);
    } else {
      r = 16 * q + (lane >> 2);
      c = (lane & 3) ^ ((lane >> 4) & 3);
    }
  };
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  uint32_t dA[DMA ? DA_PW : 1], dA2[DMA ? DA_PW : 1], dB[DMA ? DB_PW : 1], dB2[DMA ? DB_PW : 1];
  int dkA[DMA ? DA_PW : 1], dkB[DMA ? DB_PW : 1];
  if constexpr (DMA) {
#pragma unroll
    for (int i = 0; i < DA_PW; ++i) {
      const int q = wv + i * NWV;
      int r, c;
      chunk_row(q, r, c);
      dkA[i] = c * 8;
      dA[i] = (uint32_t)(r * g.lda * ES + c * 16);
      dA2[i] = (uint32_t)(r * g.lda2 * ES + c * 16);
    }
#pragma unroll
    for (int i = 0; i < DB_PW; ++i) {
      const int q = wv + i * NWV;
      if constexpr (BMODE == B_ROW) {
        int r, c;
        chunk_row(q, r, c);
        dkB[i] = c * 8;
        dB[i] = (uint32_t)(r * g.ldb * ES + c * 16);
        dB2[i] = (uint32_t)(r * g.ldb2 * ES + c * 16);
      } else {
        const int r = DBRB == 256 ? 4 * q + (lane >> 4) : 2 * q + (lane >> 5);
        const int c = DBRB == 256 ? (lane & 15) ^ (4 * ((lane >> 4) & 3)) : (lane & 31) ^ (4 * (r & 3));
        const bool ok = c * 8 < BN && n0 + c * 8 < g.N;
        dkB[i] = 0;
        // (k-major B2 has B's row length, so its offsets are B's.)
        dB[i] = ok ? (uint32_t)(r * g.ldb * ES + c * 16) : OOB;
      }
    }
  }

  // Quantized B: the thread's piece of 16 weights (W row `qrow`, first weight
  // of the piece `qcol` within the stage or tile), codes through one buffer
  // resource, per-group scale and offset through two more.  Scales and
  // offsets are group-major: [groups per W row][W rows] (q_wrows W rows: N
  // for row-major B, K for k-major B).
  const int qrow = BMODE == B_ROW ? tid / (BKE / 16) : tid / (BN / 16);
  const int qcol = BMODE == B_ROW ? (tid % (BKE / 16)) * 16 : (tid % (BN / 16)) * 16;
  const int64_t q_rowbytes = (int64_t)g.ldb * (QB ? QB : 8) / 8;
  const int64_t q_ldg = g.ldb >> g.qlog2g;  // groups per W row
  const int q_wrows = BMODE == B_ROW ? g.N : g.K;
  __amdgpu_buffer_rsrc_t rsQ, rsQs, rsQo;
  if constexpr (QB) {
    if constexpr (BMODE == B_ROW) {
      const int nrows = min(g.N - n0, BN);
      rsQ = __builtin_amdgcn_make_buffer_rsrc((void *)((const char *)g.B + n0 * q_rowbytes), (short)0,
                                              (int)(nrows * q_rowbytes), 0x00020000);
    }
    rsQs = __builtin_amdgcn_make_buffer_rsrc((void *)g.qscale, (short)0, (int)(q_ldg * q_wrows * 4), 0x00020000);
    rsQo = __builtin_amdgcn_make_buffer_rsrc((void *)g.qoffset, (short)0, (int)(q_ldg * q_wrows * 4), 0x00020000);
  }
  // Quantized direct-to-LDS loads (QD): per lane, the offset of its code
  // chunk relative to the stage's first weight and the k position (row-major
  // B) or k row (k-major B) that masks it against K; row-major codes go
  // through rsQ (the tile's W rows, stage k in soffset), k-major codes
  // through a resource over all K rows (stage row in soffset).  Scales and
  // offsets: one 16-byte load per lane covering four W rows of one group --
  // row-major B, tile rows 4 lane .. 4 lane + 3 (group in soffset); k-major
  // B, k rows 4 kq .. 4 kq + 3 of group q_g0 + gg, lane = gg (BKE / 4) + kq
  // (stage row in soffset).  Out of range: rows past N (row-major), groups
  // past the row's last, k rows past K (per stage).
  const int q_ngk = BMODE == B_KMAJ_TR ? (BN >> g.qlog2g) + 1 : 1;  // groups of a k row the tile touches
  const int q_g0 = n0 >> g.qlog2g;                                  // the first of them
  uint32_t dQ[QD ? QC_PW : 1], dS = OOB;
  int dkQ[QD ? QC_PW : 1], dkS = 0;
  __amdgpu_buffer_rsrc_t rsQk;
  if constexpr (QD) {
#pragma unroll
    for (int i = 0; i < QC_PW; ++i) {
      const int c = (wv + i * NWV) * 64 + lane;
      if constexpr (BMODE == B_ROW) {
        constexpr int CPRQ = BKE / QCW;  // chunks per W row per stage
        const int n = c / CPRQ, kc = (c % CPRQ) * QCW;
        dQ[i] = c < QCHUNKS ? (uint32_t)(n * q_rowbytes + kc * QB / 8) : OOB;
        dkQ[i] = kc;
      } else {
        constexpr int CPRQ = BN / QCW;  // chunks per k row of the tile
        const int kk = c / CPRQ, nc = (c % CPRQ) * QCW;
        dQ[i] = c < QCHUNKS && n0 + nc < g.N ? (uint32_t)(kk * q_rowbytes + (int64_t)(n0 + nc) * QB / 8) : OOB;
        dkQ[i] = kk;
      }
    }
    if constexpr (BMODE == B_ROW) {
      dS = 4 * lane < BN && n0 + 4 * lane < g.N ? (uint32_t)((n0 + 4 * lane) * 4) : OOB;
    } else {
      constexpr int LPG = BKE / 4;  // lanes per group
      const int gg = lane / LPG, kq = lane % LPG;
      dS = gg < q_ngk && q_g0 + gg < q_ldg ? (uint32_t)(((q_g0 + gg) * q_wrows + 4 * kq) * 4) : OOB;
      dkS = 4 * kq;
      rsQk = __builtin_amdgcn_make_buffer_rsrc((void *)g.B, (short)0, (int)(g.K * q_rowbytes), 0x00020000);
    }
  }

  constexpr int QW = QB == 4 ? 2 : 4;  // dwords of codes per piece
  uint32_t rqc[QB ? RD : 1][QW];
  float rqs[QB ? RD : 1], rqo[QB ? RD : 1];

  u32x4 ra[RD][A_PER];
  u32x4 rb[QB ? 1 : RD][RB];  // quantized B: only the LoRA stage is bf16

  // ---- global -> register set S for stage kt (zeros past the end) ----------
  // Stages kt < nk_main stream x/dy and W; the following ones stream the LoRA
  // operands (j = (kt - nk_main) * BKE ...).  The choice is a uniform select
  // of resources and offsets, so the step stays branch-free.
  auto is_lora = [&](int kt) { return QB ? kt < nk_lora : kt >= nk_main; };
  auto stage_k0 = [&](int kt) {
    return (QB ? (kt < nk_lora ? kt : kt - nk_lora) : (kt >= nk_main ? kt - nk_main : kt)) * BKE;
  };
  auto load_A = [&](auto SET, int kt) {
    constexpr int S = decltype(SET)::value;
    const bool lora = is_lora(kt);
    const int k0 = stage_k0(kt);
    const int krem = (lora ? g.r : g.K) - k0;  // valid k remaining (uniform)
    const int soff = k0 * ES;
    const __amdgpu_buffer_rsrc_t ra_rs = lora ? rsA2 : rsA;
#pragma unroll
    for (int i = 0; i < A_PER; ++i)
      ra[S][i] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                     ra_rs, kca[i] < krem ? (lora ? va2[i] : va[i]) : OOB, soff, 0));
  };
  // Codes, scale and offset of the thread's piece (main stages only); a piece
  // past the end of W reads zero codes, scale and offset, i.e. weight 0.
  auto load_Bq = [&](auto SET, int kt) {
    constexpr int S = decltype(SET)::value;
    if constexpr (QB) {
      const int k0 = stage_k0(kt);
      const int krem = g.K - k0;
      __amdgpu_buffer_rsrc_t rq, rs, ro;
      uint32_t vq, vs;
      if constexpr (BMODE == B_ROW) {
        const bool ok = k0 + qcol < g.K;
        rq = rsQ; rs = rsQs; ro = rsQo;
        vq = ok ? (uint32_t)(qrow * q_rowbytes + (int64_t)(k0 + qcol) * QB / 8) : OOB;
        vs = ok && n0 + qrow < g.N ? (uint32_t)((((k0 + qcol) >> g.qlog2g) * q_wrows + n0 + qrow) * 4) : OOB;
      } else {
        // W rows k0 .. k0 + BKE - 1 (rows past K out of range), columns of the tile
        const int rows = krem > 0 ? min(krem, BKE) : 0;
        rq = __builtin_amdgcn_make_buffer_rsrc((void *)((const char *)g.B + k0 * q_rowbytes), (short)0,
                                               (int)(rows * q_rowbytes), 0x00020000);
        rs = rsQs;
        ro = rsQo;
        const bool ok = n0 + qcol < g.N;
        vq = ok ? (uint32_t)(qrow * q_rowbytes + (int64_t)(n0 + qcol) * QB / 8) : OOB;
        vs = ok && qrow < rows ? (uint32_t)((((n0 + qcol) >> g.qlog2g) * q_wrows + k0 + qrow) * 4) : OOB;
      }
      if constexpr (QB == 4) {
        const auto c = __builtin_amdgcn_raw_buffer_load_b64(rq, vq, 0, 0);
        rqc[S][0] = c[0];
        rqc[S][1] = c[1];
      } else {
        const auto c = __builtin_amdgcn_raw_buffer_load_b128(rq, vq, 0, 0);
#pragma unroll
        for (int d = 0; d < 4; ++d) rqc[S][d] = c[d];
      }
      rqs[S] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, vs, 0, 0));
      rqo[S] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(ro, vs, 0, 0));
    }
  };
  auto load_B = [&](auto SET, int kt) {
    constexpr int S = QB ? 0 : decltype(SET)::value;
    const bool lora = is_lora(kt);
    const int k0 = stage_k0(kt);
    const int krem = (lora ? g.r : g.K) - k0;  // valid k remaining (uniform)
    const int soff = k0 * ES;
    if constexpr (BMODE == B_ROW) {
      const __amdgpu_buffer_rsrc_t rb_rs = lora ? rsB2 : rsB;
#pragma unroll
      for (int i = 0; i < B_PER; ++i)
        rb[S][i] = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                       rb_rs, kcb[i] < krem ? (lora ? vb2[i] : vb[i]) : OOB, soff, 0));
    } else {
      // k-major: rebase on this stage's first k row; rows past K (r) are out of range.
      const char *base = lora ? (const char *)g.B2 + ((int64_t)k0 * g.ldb2 + n0) * ES
                              : (const char *)g.B + ((int64_t)k0 * g.ldb + n0) * ES;
      const int64_t ld = lora ? g.ldb2 : g.ldb;
      const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
          (void *)base, (short)0, (int)(krem > 0 ? min(krem, BKE) * ld * ES : 0), 0x00020000);
      if constexpr (BMODE == B_KMAJ_TR) {
#pragma unroll
        for (int i = 0; i < B_PER; ++i)
          rb[S][i] = __builtin_bit_cast(
              u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, lora ? vb2[i] : vb[i], 0, 0));
      } else {
        // fp32 check mode: W and A have the same row length (d_in), so one
        // set of offsets serves both.
#pragma unroll
        for (int i = 0; i < KB_PER; ++i)
#pragma unroll
          for (int e = 0; e < VEC; ++e)
            rb[S][i * VEC + e] = __builtin_bit_cast(
                u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                           rs, vb[i] == OOB ? OOB : vb[i] + (uint32_t)(e * ld * ES), 0, 0));
      }
    }
  };

  auto load_stage = [&](auto SET, int kt) {
    load_A(SET, kt);
    if constexpr (QB) load_Bq(SET, kt);
    else load_B(SET, kt);
  };

  // ---- register set S -> LDS buffer `buf` -----------------------------------
  auto store_A = [&](auto SET, int buf) {
    constexpr int S = decltype(SET)::value;
    char *sA = smem + buf * STAGE;
#pragma unroll
    for (int i = 0; i < A_PER; ++i) {
      const int c = tid + i * NT;
      if (A_CH % NT == 0 || c < A_CH) st16(sA + (c / CPR) * ROWA + (c % CPR) * 16, ra[S][i]);
    }
  };
  // Dequantize the thread's piece: w = scale * code + offset, rounded to bf16,
  // two 16-byte chunks at the piece's place in the B tile.
  auto store_Bq = [&](auto SET, int buf) {
    constexpr int S = decltype(SET)::value;
    if constexpr (QB) {
      char *sB = smem + buf * STAGE + A_BYTES;
      float f[16];
      if constexpr (QB == 4) {
        // dword d holds weights 8d .. 8d+7; byte j of it has weight 8d+2j in
        // its low nibble and 8d+2j+1 in its high nibble.
#pragma unroll
        for (int d = 0; d < 2; ++d) {
          const uint32_t lo = rqc[S][d] & 0x0F0F0F0Fu, hi = (rqc[S][d] >> 4) & 0x0F0F0F0Fu;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            f[8 * d + 2 * j] = fmaf(rqs[S], (float)((lo >> (8 * j)) & 0xFFu), rqo[S]);
            f[8 * d + 2 * j + 1] = fmaf(rqs[S], (float)((hi >> (8 * j)) & 0xFFu), rqo[S]);
          }
        }
      } else {
#pragma unroll
        for (int d = 0; d < 4; ++d)
#pragma unroll
          for (int j = 0; j < 4; ++j) f[4 * d + j] = fmaf(rqs[S], (float)((rqc[S][d] >> (8 * j)) & 0xFFu), rqo[S]);
      }
      char *dst = BMODE == B_ROW ? sB + qrow * ROWA + qcol * 2 : sB + qrow * ROWT + qcol * 2;
      st16(dst, pack_vec(E(), f));
      st16(dst + 16, pack_vec(E(), f + 8));
    }
  };
  auto store_B = [&](auto SET, int buf) {
    constexpr int S = QB ? 0 : decltype(SET)::value;
    char *sB = smem + buf * STAGE + A_BYTES;
    if constexpr (BMODE == B_ROW) {
#pragma unroll
      for (int i = 0; i < B_PER; ++i) {
        const int c = tid + i * NT;
        if (B_CH % NT == 0 || c < B_CH) st16(sB + (c / CPR) * ROWA + (c % CPR) * 16, rb[S][i]);
      }
    } else if constexpr (BMODE == B_KMAJ_TR) {
#pragma unroll
      for (int i = 0; i < B_PER; ++i) {
        const int c = tid + i * NT;
        if (B_CH % NT == 0 || c < B_CH) st16(sB + (c / NBV) * ROWT + (c % NBV) * 16, rb[S][i]);
      }
    } else {
#pragma unroll
      for (int i = 0; i < KB_PER; ++i) {
        const int b = tid + i * NT;
        if (KB_BLK % NT == 0 || b < KB_BLK) {
          const int kb = b % (BKE / VEC), nb = b / (BKE / VEC);
          u32x4 tr[VEC];
          transpose_block(E(), &rb[S][i * VEC], tr);
#pragma unroll
          for (int c = 0; c < VEC; ++c) st16(sB + (nb * VEC + c) * ROWA + kb * 16, tr[c]);
        }
      }
    }
  };

  auto store_stage = [&](auto SET, int buf) {
    store_A(SET, buf);
    if constexpr (QB) store_Bq(SET, buf);
    else store_B(SET, buf);
  };

  // ---- direct-to-LDS loads of stage kt into ring buffer BUF --------------------
  auto dma_stage = [&](auto BUF, int kt) {
    if constexpr (DMA) {
      char *sA = ring_a(BUF);
      char *sB = ring_b(BUF);
      const bool lora = is_lora(kt);
      const int k0 = stage_k0(kt);
      const int krem = (lora ? g.r : g.K) - k0;  // valid k remaining (uniform)
      const int soff = k0 * ES;
      const __amdgpu_buffer_rsrc_t ra_rs = lora ? rsA2 : rsA;
#pragma unroll
      for (int i = 0; i < DA_PW; ++i) {
        const uint32_t vo = dkA[i] < krem ? (lora ? dA2[i] : dA[i]) : (uint32_t)OOB;
        dma16(ra_rs, sA + (wv + i * NWV) * 1024, vo, soff);
      }
      // (Quantized B: only the LoRA stages' B is loaded here, as bf16.)
      if (QD && !lora) return;
      if constexpr (BMODE == B_ROW) {
        const __amdgpu_buffer_rsrc_t rb_rs = lora ? rsB2 : rsB;
#pragma unroll
        for (int i = 0; i < DB_PW; ++i) {
          const uint32_t vo = dkB[i] < krem ? (lora ? dB2[i] : dB[i]) : (uint32_t)OOB;
          dma16(rb_rs, sB + (wv + i * NWV) * 1024, vo, soff);
        }
      } else {
        const char *base = lora ? (const char *)g.B2 + ((int64_t)k0 * g.ldb2 + n0) * ES
                                : (const char *)g.B + ((int64_t)k0 * g.ldb + n0) * ES;
        const int64_t ld = lora ? g.ldb2 : g.ldb;
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            (void *)base, (short)0, (int)(krem > 0 ? min(krem, BKE) * ld * ES : 0), 0x00020000);
#pragma unroll
        for (int i = 0; i < DB_PW; ++i) {
          dma16(rs, sB + (wv + i * NWV) * 1024, dB[i], 0);
        }
      }
    }
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.0f;

  // ---- MFMA fragments of one k-slice ------------------------------------------
  struct Frag {
    u32x4 a[FM], b[FN];
  };
  const int lrow = lane & 31;
  const int lko = (lane >> 5) * 16;
  // transposed-read addressing: 16-lane group gq, lane iq within it
  const int gq = lane >> 4, iq = lane & 15;
  const int tr_k = 8 * (gq >> 1) + (iq >> 2);
  const int tr_n = 16 * (gq & 1) + 4 * (iq & 3);

  auto read_frags = [&](int buf, int s, Frag &f) {
    const char *sA = smem + buf * STAGE;
    const char *sB = sA + A_BYTES;
    const int sl = wk * SPW + s;
#pragma unroll
    for (int i = 0; i < FM; ++i) f.a[i] = ld16(sA + (wm * WTM + i * 32 + lrow) * ROWA + sl * 32 + lko);
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      if constexpr (BMODE == B_KMAJ_TR) {
        const char *p = sB + (sl * 16 + tr_k) * ROWT + (wn * WTN + j * 32 + tr_n) * 2;
        i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)p);
        i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(p + 4 * ROWT));
        f.b[j] = u32x4{__builtin_bit_cast(uint2, lo).x, __builtin_bit_cast(uint2, lo).y,
                       __builtin_bit_cast(uint2, hi).x, __builtin_bit_cast(uint2, hi).y};
      } else {
        f.b[j] = ld16(sB + (wn * WTN + j * 32 + lrow) * ROWA + sl * 32 + lko);
      }
    }
  };
  // Fragment reads from a direct-to-LDS stage (swizzled chunks, see dma_stage).
  const int swz_a = CPR == 8 ? (lrow & 7) ^ ((lrow >> 3) & 1) : (lrow >> 2) & 3;  // the lane's rows' swizzle
  const int swz_t = 4 * ((iq >> 2) & 3);
  auto read_frags_d = [&](auto BUF, int s, Frag &f) {
    const char *sA = ring_a(BUF);
    const char *sB = ring_b(BUF);
    const int sl = wk * SPW + s;
    const int ca = ((sl * 2 + (lane >> 5)) ^ swz_a) * 16;
#pragma unroll
    for (int i = 0; i < FM; ++i) f.a[i] = ld16(sA + (wm * WTM + i * 32 + lrow) * BKB + ca);
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      if constexpr (BMODE == B_KMAJ_TR) {
        const int n = wn * WTN + j * 32 + tr_n;
        const char *p = sB + (sl * 16 + tr_k) * DBRB + (((n >> 3) ^ swz_t) * 16) + (n & 7) * 2;
        i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)p);
        i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(p + 4 * DBRB));
        f.b[j] = u32x4{__builtin_bit_cast(uint2, lo).x, __builtin_bit_cast(uint2, lo).y,
                       __builtin_bit_cast(uint2, hi).x, __builtin_bit_cast(uint2, hi).y};
      } else {
        f.b[j] = ld16(sB + (wn * WTN + j * 32 + lrow) * BKB + ca);
      }
    }
  };
  // One direct-to-LDS load (q < IPS) of stage kt into ring buffer BUF.  With
  // MASK = 0 the stage is a full main stage (every k below K, no LoRA step),
  // so the lanes' precomputed offsets need no per-load selection.
  auto dma_one = [&](auto BUF, int kt, auto QI, auto MASK) __attribute__((always_inline)) {
    if constexpr (DMA && !decltype(MASK)::value) {
      constexpr int q = decltype(QI)::value;
      const int k0 = stage_k0(kt);
      if constexpr (q < DA_PW) {
        dma16(rsA, ring_a(BUF) + (wv + q * NWV) * 1024, dA[q], k0 * ES);
      } else {
        constexpr int i = q - DA_PW;
        if constexpr (BMODE == B_ROW) dma16(rsB, ring_b(BUF) + (wv + i * NWV) * 1024, dB[i], k0 * ES);
        else dma16(rsBk, ring_b(BUF) + (wv + i * NWV) * 1024, dB[i], (int)((int64_t)k0 * g.ldb * ES));
      }
    } else if constexpr (DMA) {
      constexpr int q = decltype(QI)::value;
      const bool lora = is_lora(kt);
      const int k0 = stage_k0(kt);
      const int krem = (lora ? g.r : g.K) - k0;
      const int soff = k0 * ES;
      if constexpr (q < DA_PW) {
        const __amdgpu_buffer_rsrc_t ra_rs = lora ? rsA2 : rsA;
        const uint32_t vo = dkA[q] < krem ? (lora ? dA2[q] : dA[q]) : (uint32_t)OOB;
        dma16(ra_rs, ring_a(BUF) + (wv + q * NWV) * 1024, vo, soff);
      } else {
        constexpr int i = q - DA_PW;
        if constexpr (BMODE == B_ROW) {
          const __amdgpu_buffer_rsrc_t rb_rs = lora ? rsB2 : rsB;
          const uint32_t vo = dkB[i] < krem ? (lora ? dB2[i] : dB[i]) : (uint32_t)OOB;
          dma16(rb_rs, ring_b(BUF) + (wv + i * NWV) * 1024, vo, soff);
        } else {
          const char *base = lora ? (const char *)g.B2 + ((int64_t)k0 * g.ldb2 + n0) * ES
                                  : (const char *)g.B + ((int64_t)k0 * g.ldb + n0) * ES;
          const int64_t ld = lora ? g.ldb2 : g.ldb;
          const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
              (void *)base, (short)0, (int)(krem > 0 ? min(krem, BKE) * ld * ES : 0), 0x00020000);
          dma16(rs, ring_b(BUF) + (wv + i * NWV) * 1024, dB[i], 0);
        }
      }
    }
  };
  // One fragment read (ri < SPW * (FM + FN)) of a direct-to-LDS stage.
  auto read_one_d = [&](auto BUF, auto RI, Frag *f) __attribute__((always_inline)) {
    constexpr int ri = decltype(RI)::value;
    constexpr int s2 = ri / (FM + FN), w = ri % (FM + FN);
    const char *sA = ring_a(BUF);
    const char *sB = ring_b(BUF);
    const int sl = wk * SPW + s2;
    if constexpr (w < FM) {
      const int ca = ((sl * 2 + (lane >> 5)) ^ swz_a) * 16;
      f[s2].a[w] = ld16(sA + (wm * WTM + w * 32 + lrow) * BKB + ca);
    } else {
      constexpr int j = w - FM;
      if constexpr (BMODE == B_KMAJ_TR) {
        const int n = wn * WTN + j * 32 + tr_n;
        const char *pp = sB + (sl * 16 + tr_k) * DBRB + (((n >> 3) ^ swz_t) * 16) + (n & 7) * 2;
        i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)pp);
        i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(pp + 4 * DBRB));
        f[s2].b[j] = u32x4{__builtin_bit_cast(uint2, lo).x, __builtin_bit_cast(uint2, lo).y,
                           __builtin_bit_cast(uint2, hi).x, __builtin_bit_cast(uint2, hi).y};
      } else {
        const int ca = ((sl * 2 + (lane >> 5)) ^ swz_a) * 16;
        f[s2].b[j] = ld16(sB + (wn * WTN + j * 32 + lrow) * BKB + ca);
      }
    }
  };
  // ---- quantized direct-to-LDS stages (QD) --------------------------------------
  auto qcode_slot = [&](auto S) -> char * { return smem + NBUF * DSTAGE + decltype(S)::value * QSLOT; };
  // Scale / offset slot of quantized stage kt (k-major: the stage's ring
  // slot S; row-major: its group's slot).
  auto qso_slot = [&](auto S, int kt) -> char * {
    const int slot = BMODE == B_ROW ? (stage_k0(kt) >> g.qlog2g) & 3 : decltype(S)::value;
    return smem + NBUF * DSTAGE + 3 * QSLOT + slot * 2 * QSO;
  };
  // Whether this wave loads scales and offsets (two loads) for quantized
  // stage kt: wave 0, for k-major B every stage, for row-major B the first
  // stage of every group.
  auto so_loads = [&](int kt) -> bool {
    if constexpr (BMODE == B_ROW) {
      const int k0 = stage_k0(kt);
      return wv == 0 && !is_lora(kt) && k0 < g.K && (k0 & ((1 << g.qlog2g) - 1)) == 0;
    } else {
      return wv == 0;
    }
  };
  // Those loads, into slot S; issued first in their step.
  auto dma_so = [&](auto S, int kt) __attribute__((always_inline)) {
    if constexpr (QD) {
      if (so_loads(kt)) {
        const int k0 = stage_k0(kt);
        char *dst = qso_slot(S, kt);
        int so;
        uint32_t vo = dS;
        if constexpr (BMODE == B_ROW) {
          so = (k0 >> g.qlog2g) * q_wrows * 4;
        } else {
          const int krem = is_lora(kt) ? 0 : g.K - k0;
          so = k0 * 4;
          vo = dkS < krem ? dS : (uint32_t)OOB;
        }
        dma16(rsQs, dst, vo, so);
        dma16(rsQo, dst + QSO, vo, so);
      }
    }
  };
  // Code load q (< QC_PW) of quantized stage kt into code slot S.  With MASK
  // = 0 the stage is a full main stage; else lanes past K read zeros, and so
  // does a LoRA stage (no codes).
  auto dma_code = [&](auto S, int kt, auto QI, auto MASK) __attribute__((always_inline)) {
    if constexpr (QD) {
      constexpr int i = decltype(QI)::value;
      const int k0 = stage_k0(kt);
      const int krem = is_lora(kt) ? 0 : g.K - k0;
      char *dst = qcode_slot(S) + (wv + i * NWV) * 1024;
      const uint32_t vo = !decltype(MASK)::value || dkQ[i] < krem ? dQ[i] : (uint32_t)OOB;
      if constexpr (BMODE == B_ROW)
        dma16(rsQ, dst, vo, k0 * QB / 8);
      else
        dma16(rsQk, dst, vo, (int)((int64_t)k0 * q_rowbytes));
    }
  };
  // Load q (< DA_PW) of main stage kt's A into ring buffer BUF.
  auto dma_a_one = [&](auto BUF, int kt, auto QI, auto MASK) __attribute__((always_inline)) {
    constexpr int q = decltype(QI)::value;
    const int k0 = stage_k0(kt);
    const uint32_t vo = !decltype(MASK)::value || dkA[q] < g.K - k0 ? dA[q] : (uint32_t)OOB;
    dma16(rsA, ring_a(BUF) + (wv + q * NWV) * 1024, vo, k0 * ES);
  };
  // Dequantization of the stage in slot S into the B area of ring buffer BUF:
  // w = scale * code + offset (one fp32 fma), rounded to bf16, in the layout
  // the bf16 direct-to-LDS loads produce.  Thread t takes runs t, t + NT, ...
  struct QRun {
    uint32_t c[QB == 8 ? 4 : 2];
    float s, o;
  };
  auto dq_read = [&](auto S, int kt, QRun(&q)[QRPT]) __attribute__((always_inline)) {
    if constexpr (QD) {
      const char *cs = qcode_slot(S);
      const float *ss = (const float *)qso_slot(S, kt);
#pragma unroll
      for (int j = 0; j < QRPT; ++j) {
        int rho = tid + j * NT;
        if (QRUNS % NT) rho = rho < QRUNS ? rho : 0;
        if constexpr (QB == 8) {
          const u32x4 v = ld16(cs + rho * 16);
#pragma unroll
          for (int d = 0; d < 4; ++d) q[j].c[d] = v[d];
        } else {
          const uint2 v = *(const uint2 *)(cs + rho * 8);
          q[j].c[0] = v.x;
          q[j].c[1] = v.y;
        }
        int pr;
        if constexpr (BMODE == B_ROW) {
          pr = rho / (BKE / 16);  // tile row
        } else {
          const int kk = rho / (BN / 16), nr = rho % (BN / 16);
          pr = (((n0 + nr * 16) >> g.qlog2g) - q_g0) * BKE + kk;
        }
        q[j].s = ss[pr];
        q[j].o = ss[QSO / 4 + pr];
      }
    }
  };
  auto dq_write = [&](auto BUF, const QRun(&q)[QRPT]) __attribute__((always_inline)) {
    if constexpr (QD) {
      char *sB = ring_b(BUF);
#pragma unroll
      for (int j = 0; j < QRPT; ++j) {
        const int rho = tid + j * NT;
        if (QRUNS % NT == 0 || rho < QRUNS) {
          // w = fma(scale, code, offset) per weight, rounded to bf16 in pairs.
          // Each code byte converts with one v_cvt_f32_ubyteN: for 4-bit codes
          // the low and the high nibbles are first spread to bytes of their
          // own (an empty asm hides their known-zero bits, which would
          // otherwise turn each conversion into a bit-field extract plus a
          // conversion).
          const float qs = q[j].s, qo = q[j].o;
          uint32_t w[8];
          if constexpr (QB == 4) {
            // dword d: weights 8d .. 8d + 7, weight 8d + 2i in the low nibble of byte i
#pragma unroll
            for (int d = 0; d < 2; ++d) {
              uint32_t lo = q[j].c[d] & 0x0F0F0F0Fu, hi = (q[j].c[d] >> 4) & 0x0F0F0F0Fu;
              asm("" : "+v"(lo), "+v"(hi));
#pragma unroll
              for (int i = 0; i < 4; ++i)
                w[4 * d + i] = pack_bf16x2(fmaf(qs, (float)((lo >> (8 * i)) & 0xFFu), qo),
                                           fmaf(qs, (float)((hi >> (8 * i)) & 0xFFu), qo));
            }
          } else {
#pragma unroll
            for (int d = 0; d < 4; ++d)
#pragma unroll
              for (int i = 0; i < 2; ++i)
                w[2 * d + i] = pack_bf16x2(fmaf(qs, (float)((q[j].c[d] >> (16 * i)) & 0xFFu), qo),
                                           fmaf(qs, (float)((q[j].c[d] >> (16 * i + 8)) & 0xFFu), qo));
          }
          const u32x4 lo = u32x4{w[0], w[1], w[2], w[3]}, hi = u32x4{w[4], w[5], w[6], w[7]};
          if constexpr (BMODE == B_ROW) {
            // row n, 16-byte chunks 2 kr and 2 kr + 1, chunk c kept at c ^ swz(n)
            const int n = rho / (BKE / 16), kr = rho % (BKE / 16);
            const int swz = CPR == 8 ? (n & 7) ^ ((n >> 3) & 1) : (n >> 2) & 3;
            st16(sB + n * BKB + ((2 * kr) ^ swz) * 16, lo);
            st16(sB + n * BKB + ((2 * kr + 1) ^ swz) * 16, hi);
          } else {
            // k row kk, chunks 2 nr and 2 nr + 1, chunk c kept at c ^ 4 (kk & 3)
            const int kk = rho / (BN / 16), nr = rho % (BN / 16);
            const int swz = 4 * (kk & 3);
            st16(sB + kk * DBRB + ((2 * nr) ^ swz) * 16, lo);
            st16(sB + kk * DBRB + ((2 * nr + 1) ^ swz) * 16, hi);
          }
        }
      }
    }
  };
  // D = Bop * Aop^T: D rows are output columns n, D columns are rows m, so each
  // lane ends up holding runs of 4 consecutive n of one output row.
  auto mma_frags = [&](const Frag &f) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) mma32(E(), acc[i][j], f.b[j], f.a[i]);
  };
  // All slices of the stage in `buf`; slice 0's fragments arrive in f0.
  auto compute = [&](int buf, const Frag &f0) {
    Frag cur = f0;
#pragma unroll
    for (int s = 0; s < SPW; ++s) {
      Frag nxt;
      if (s + 1 < SPW) read_frags(buf, s + 1, nxt);
      mma_frags(cur);
      if (s + 1 < SPW) cur = nxt;
    }
  };

  // ---- main loop -------------------------------------------------------------
  // Step kt: issue the global loads of stage kt + D into register set
  // (kt + D) % RD, write register set (kt + E) % RD (loaded RD - 1 steps
  // earlier, so the loads have RD - 1 steps to land) into LDS buffer
  // (kt + E) % NBUF, then run the MFMAs of stage kt.  With NBUF = 3, E = 2 and
  // the first fragments of stage kt + 1 are read before the barrier; with
  // NBUF = 2, E = 1.  Unrolled by RD so the register sets are static; the LDS
  // buffer index is a run-time value.  Each step is branch-free: loads of
  // stages past the end select out-of-range offsets (zeros, no memory traffic)
  // and stores of such stages land in an LDS buffer that is never read again.
  static_assert(!QB || FS, "quantized B runs the staged-fragment schedule");
  if constexpr (DMA) {
    // Ring of NBUF stages filled by direct-to-LDS loads, fragments staged in
    // registers one step ahead.  Step kt: wait for this wave's loads of stage
    // kt + 1 and for its LDS reads of the previous step, barrier (stage kt + 1
    // is then complete for every wave and nobody reads the buffer of stage kt
    // any more), issue the loads of stage kt + NBUF into that buffer, read the
    // fragments of stage kt + 1 while the MFMAs of stage kt run.  NBUF - 1
    // stages stay in flight behind the one being read.  The waits are explicit
    // (the loads write LDS behind the compiler's back as far as the barrier is
    // concerned): vmcnt counts this wave's loads in issue order.
    constexpr int UN = NBUF % 2 == 0 ? NBUF : 2 * NBUF;  // ring buffers and fragment sets static
    constexpr int W_ENC = (7 << 4) | (15 << 8);           // expcnt, lgkmcnt: no wait
    Frag F[2][SPW];
    auto read_stage_d = [&](auto BUF, Frag(&f)[SPW]) {
#pragma unroll
      for (int s2 = 0; s2 < SPW; ++s2) read_frags_d(BUF, s2, f[s2]);
    };
    auto mma_stage = [&](const Frag(&f)[SPW]) {
#pragma unroll
      for (int s2 = 0; s2 < SPW; ++s2) mma_frags(f[s2]);
    };
    if constexpr (QD) {
      // Quantized B.  Step kt: wait for its loads of stage kt + 1 and of the
      // codes of stage kt + NBUF (both issued two steps earlier), barrier,
      // dequantize stage kt + NBUF into the B area of the buffer that stage
      // kt vacated, issue the codes, scales and offsets of stage kt + NBUF + 2
      // and the A loads of stage kt + NBUF, read the fragments of stage kt + 1
      // and run the MFMAs of stage kt.  The LoRA stages come first (all
      // within the prologue, as bf16).
      constexpr int QL = QC_PW;  // counted loads of a stage's codes
      constexpr int W_LGKM = 15 | (7 << 4) | (3 << 14);  // lgkmcnt(0) only
      static_for<0, NBUF>([&](auto SI) {
        dma_so(SI, decltype(SI)::value);
        dma_stage(SI, decltype(SI)::value);
        static_for<0, QL>([&](auto QI) { dma_code(SI, decltype(SI)::value, QI, IC<1>()); });
      });
      __builtin_amdgcn_s_waitcnt(0 | W_ENC);
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      static_for<0, NBUF>([&](auto SI) {
        if (decltype(SI)::value >= nk_lora) {
          QRun q[QRPT];
          dq_read(SI, decltype(SI)::value, q);
          dq_write(SI, q);
        }
      });
      __builtin_amdgcn_s_waitcnt(W_LGKM);
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      static_for<0, 2>([&](auto SI) {
        dma_so(SI, NBUF + decltype(SI)::value);
        static_for<0, QL>([&](auto QI) { dma_code(SI, NBUF + decltype(SI)::value, QI, IC<1>()); });
      });
      __builtin_amdgcn_s_waitcnt((QL & 15) | ((QL >> 4) << 14) | W_ENC);  // stage NBUF's codes landed
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      read_stage_d(IC<0>(), F[0]);
      auto qstep = [&](auto PH, int kt, auto MASK) __attribute__((always_inline)) {
        constexpr int P = decltype(PH)::value;  // kt % UN
        // the loads of the last step (with its scale loads, if any) may be in flight
        constexpr int V = QIPS, V2 = QIPS + 2;
        if (so_loads(kt + NBUF + 1))
          __builtin_amdgcn_s_waitcnt((V2 & 15) | ((V2 >> 4) << 14) | (7 << 4));  // and lgkmcnt(0)
        else
          __builtin_amdgcn_s_waitcnt((V & 15) | ((V >> 4) << 14) | (7 << 4));
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        QRun q[QRPT];
        dq_read(IC<P % NBUF>(), kt + NBUF, q);
        dma_so(IC<(P + 2) % NBUF>(), kt + NBUF + 2);
        constexpr int NRO = SPW * (FM + FN);
        static_for<0, NRO>([&](auto RI) {
          constexpr int ri = decltype(RI)::value;
          read_one_d(IC<(P + 1) % NBUF>(), RI, F[(P + 1) % 2]);
          static_for<ri * QIPS / NRO, (ri + 1) * QIPS / NRO>([&](auto QI) {
            constexpr int qi = decltype(QI)::value;
            if constexpr (qi < QL)
              dma_code(IC<(P + 2) % NBUF>(), kt + NBUF + 2, QI, MASK);
            else
              dma_a_one(IC<P % NBUF>(), kt + NBUF, IC<qi - QL>(), MASK);
          });
        });
        dq_write(IC<P % NBUF>(), q);
        mma_stage(F[P % 2]);
        constexpr int NM = SPW * FM * FN;
        constexpr int NR = SPW * (FM + FN * (BMODE == B_KMAJ_TR ? 2 : 1));
        constexpr int NQR = QRPT * 3;                     // dequant LDS reads
        constexpr int NQV = QRPT * (QB == 4 ? 46 : 40);   // dequant vector instructions (about)
        constexpr int NQW = QRPT * 2;                     // dequant LDS writes
        // The dequantization's LDS reads go first and its arithmetic starts
        // two MFMAs later, so the first MFMAs do not wait for those reads.
        constexpr int M0 = NM > 4 ? 2 : 1;
        static_for<0, NM>([&](auto MI) {
          constexpr int m = decltype(MI)::value;
          constexpr int r = (m + 1) * NR / NM - m * NR / NM;
          constexpr int v = m < M0 ? 0 : (m - M0 + 1) * NQV / (NM - M0) - (m - M0) * NQV / (NM - M0);
          if constexpr (m == 0) __builtin_amdgcn_sched_group_barrier(0x100, NQR, 0);  // DS read
          if constexpr (r > 0) __builtin_amdgcn_sched_group_barrier(0x100, r, 0);   // DS read
          if constexpr (v > 0) __builtin_amdgcn_sched_group_barrier(0x002, v, 0);   // VALU
          if constexpr (m >= NM - NQW) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // DS write
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                        // MFMA
        });
        __builtin_amdgcn_sched_barrier(0);
      };
      // Steps whose loads are all of full main stages run unmasked.
      const int nb = nk_lora + g.K / BKE - NBUF - 2;
      int kt = 0;
      for (; kt + UN <= nb; kt += UN)
        static_for<0, UN>([&](auto PH) { qstep(PH, kt + decltype(PH)::value, IC<0>()); });
      for (; kt + UN <= nk; kt += UN)
        static_for<0, UN>([&](auto PH) { qstep(PH, kt + decltype(PH)::value, IC<1>()); });
      static_for<0, UN - 1>([&](auto PH) {
        constexpr int P = decltype(PH)::value;
        if (kt + P < nk) qstep(PH, kt + P, IC<1>());
      });
    } else {
      // A fused launch's LoRA-step operands come from its producers: wait for
      // them before the first load of a LoRA stage (here when the prologue
      // already issues one, else in the step that does).
      if (coh && nk_main < NBUF) fz_wait(fz.sync, fz.gen, fz.nprod, fz.ncons);
      static_for<0, NBUF>([&](auto SI) { dma_stage(SI, decltype(SI)::value); });
      {
        constexpr int V = (NBUF - 1) * IPS;  // stage 0 landed
        __builtin_amdgcn_s_waitcnt((V & 15) | ((V >> 4) << 14) | W_ENC);
      }
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      read_stage_d(IC<0>(), F[0]);
      auto step = [&](auto PH, int kt, auto MASK) __attribute__((always_inline)) {
        constexpr int P = decltype(PH)::value;  // kt % UN
        constexpr int V = (NBUF - 2) * IPS;     // stage kt + 1 landed
        __builtin_amdgcn_s_waitcnt((V & 15) | ((V >> 4) << 14) | (7 << 4));  // and lgkmcnt(0)
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        // A fused launch's LoRA stage holds its producers' output: wait for them
        // before the step that issues its loads.
        if (FUSE && coh && kt + NBUF == nk_main) fz_wait(fz.sync, fz.gen, fz.nprod, fz.ncons);
        __builtin_amdgcn_sched_barrier(0);
        // The loads of stage kt + NBUF are spread between the fragment reads of
        // stage kt + 1 (in source order: an LDS read cannot pass the load
        // assembly), so the load path, the LDS and the matrix cores work side by
        // side instead of all loads queueing at the top of the step.
        constexpr int NRO = SPW * (FM + FN);
        static_for<0, NRO>([&](auto RI) {
          constexpr int ri = decltype(RI)::value;
          read_one_d(IC<(P + 1) % NBUF>(), RI, F[(P + 1) % 2]);
          static_for<ri * IPS / NRO, (ri + 1) * IPS / NRO>(
              [&](auto QI) { dma_one(IC<P % NBUF>(), kt + NBUF, QI, MASK); });
        });
        mma_stage(F[P % 2]);
        constexpr int NM = SPW * FM * FN;
        constexpr int NR = SPW * (FM + FN * (BMODE == B_KMAJ_TR ? 2 : 1));
        static_for<0, NM>([&](auto MI) {
          constexpr int m = decltype(MI)::value;
          constexpr int r = (m + 1) * NR / NM - m * NR / NM;
          if constexpr (r > 0) __builtin_amdgcn_sched_group_barrier(0x100, r, 0);  // DS read
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                       // MFMA
        });
        __builtin_amdgcn_sched_barrier(0);
      };
      // Steps whose loads fill a full main stage (stage kt + NBUF below the K
      // tail) run unmasked; the K tail, the LoRA stages and the stages past the
      // end (zeros) run masked.
      // (Launches with producers, and the 256 x 128 tile with k-major B, keep
      // one loop: the second copy of the steps costs them registers and spills.)
      constexpr bool SPLIT = !FUSE && !(BM == 256 && BN == 128 && BMODE == B_KMAJ_TR);
      const bool whole_ok = BMODE != B_KMAJ_TR || (int64_t)g.K * g.ldb * ES < (int64_t)1 << 31;
      const int nb = QB || !whole_ok ? 0 : g.K / BKE - NBUF;
      int kt = 0;
      if constexpr (SPLIT)
        for (; kt + UN <= nb; kt += UN)
          static_for<0, UN>([&](auto PH) { step(PH, kt + decltype(PH)::value, IC<0>()); });
      for (; kt + UN <= nk; kt += UN)
        static_for<0, UN>([&](auto PH) { step(PH, kt + decltype(PH)::value, IC<1>()); });
      static_for<0, UN - 1>([&](auto PH) {
        constexpr int P = decltype(PH)::value;
        if (kt + P < nk) step(PH, kt + P, IC<1>());
      });
    }
    // The loads of the stages past the end still write LDS: drain them before
    // the buffers are reused.
    __builtin_amdgcn_s_waitcnt(0 | W_ENC);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    if (coh && tid == 0) fz_done(fz.sync);
  } else if constexpr (FS) {
    // Staged fragments: every MFMA fragment of a stage is read from LDS one
    // step ahead into the second of two register sets, so the MFMAs of a
    // step never wait on LDS and the reads of the next stage overlap them.
    // A stage's LDS buffer is free once its fragments are in registers, so
    // two buffers suffice: step kt writes stage kt + 2 over stage kt.
    constexpr int E_ST = 2;
    constexpr int D_LD = E_ST + RD - 1;
    constexpr int UN = RD % 2 == 0 ? RD : 2 * RD;  // unroll: register sets and fragment sets static
    Frag F[2][SPW];
    auto read_stage = [&](int buf, Frag(&f)[SPW]) {
#pragma unroll
      for (int s2 = 0; s2 < SPW; ++s2) read_frags(buf, s2, f[s2]);
    };
    auto mma_stage = [&](const Frag(&f)[SPW]) {
#pragma unroll
      for (int s2 = 0; s2 < SPW; ++s2) mma_frags(f[s2]);
    };
    // (With a quantized B, stage 0 may be the bf16 LoRA step.)
    auto pro_load = [&](auto SET, int kt) {
      if (QB && is_lora(kt)) {
        load_A(SET, kt);
        load_B(SET, kt);
      } else {
        load_stage(SET, kt);
      }
    };
    auto pro_store = [&](auto SET, int kt, int buf) {
      if (QB && is_lora(kt)) {
        store_A(SET, buf);
        store_B(SET, buf);
      } else {
        store_stage(SET, buf);
      }
    };
    static_for<0, RD>([&](auto SI) {
      constexpr int st = decltype(SI)::value;
      pro_load(IC<st>(), st);
    });
    static_for<0, E_ST>([&](auto SI) {
      constexpr int st = decltype(SI)::value;
      pro_store(IC<st % RD>(), st, st);
      if constexpr (st + RD < D_LD) pro_load(IC<(st + RD) % RD>(), st + RD);
    });
    __syncthreads();
    read_stage(0, F[0]);
    __syncthreads();
    auto step = [&](auto PH, int kt) {
      constexpr int P = decltype(PH)::value;  // kt % UN
      const int cb = P % 2;                    // LDS buffer of stage kt (and kt + 2)
      if constexpr (FS == 2) {
        // Interleaved: the step's memory instructions are spread between its
        // MFMAs (which depend only on registers read in the previous step), so
        // the load, LDS and matrix pipes work side by side instead of in turn.
        load_stage(IC<(P + D_LD) % RD>(), kt + D_LD);
        store_stage(IC<(P + E_ST) % RD>(), cb);
        read_stage(1 - cb, F[(P + 1) % 2]);
        mma_stage(F[P % 2]);
        constexpr int NM = SPW * FM * FN;
        constexpr int NV = A_PER + (QB ? 3 : BMODE == B_KMAJ_REG ? KB_PER * VEC : B_PER);
        constexpr int NW = A_PER + (QB ? 2 : BMODE == B_KMAJ_REG ? KB_PER * VEC : B_PER);
        constexpr int NR = SPW * (FM + FN * (BMODE == B_KMAJ_TR ? 2 : 1));
        static_for<0, NM>([&](auto MI) {
          constexpr int m = decltype(MI)::value;
          constexpr int v = (m + 1) * NV / NM - m * NV / NM;
          constexpr int w = (m + 1) * NW / NM - m * NW / NM;
          constexpr int r = (m + 1) * NR / NM - m * NR / NM;
          if constexpr (v > 0) __builtin_amdgcn_sched_group_barrier(0x020, v, 0);  // VMEM read
          if constexpr (w > 0) __builtin_amdgcn_sched_group_barrier(0x200, w, 0);  // DS write
          if constexpr (r > 0) __builtin_amdgcn_sched_group_barrier(0x100, r, 0);  // DS read
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                       // MFMA
        });
      } else {
        load_stage(IC<(P + D_LD) % RD>(), kt + D_LD);
        __builtin_amdgcn_sched_barrier(0);
        store_stage(IC<(P + E_ST) % RD>(), cb);
        __builtin_amdgcn_sched_barrier(0);
        read_stage(1 - cb, F[(P + 1) % 2]);
        __builtin_amdgcn_sched_barrier(0);
        mma_stage(F[P % 2]);
      }
      // Keep the MFMAs ahead of the barrier: the scheduler would otherwise
      // hoist the barrier (and its wait for every outstanding LDS read) above
      // them, so they would stall on the reads of the next stage.
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
    };
    // Whole groups of UN steps without branches (a step skipped on some path
    // would make the compiler wait for every load in flight where the paths
    // merge), then the remaining steps.
    int kt = 0;
    for (; kt + UN <= nk; kt += UN) static_for<0, UN>([&](auto PH) { step(PH, kt + decltype(PH)::value); });
    static_for<0, UN - 1>([&](auto PH) {
      constexpr int P = decltype(PH)::value;
      if (kt + P < nk) step(PH, kt + P);
    });
  } else {
    constexpr int E_ST = NBUF == 3 ? 2 : 1;
    constexpr int D_LD = E_ST + RD - 1;
    Frag f0;
    {
      // prologue: stages 0 .. D_LD - 1 loaded, 0 .. E_ST - 1 stored
      static_for<0, RD>([&](auto SI) {
        constexpr int st = decltype(SI)::value;
        load_stage(IC<st>(), st);
      });
      static_for<0, E_ST>([&](auto SI) {
        constexpr int st = decltype(SI)::value;
        store_stage(IC<st % RD>(), st);
        if constexpr (st + RD < D_LD) load_stage(IC<(st + RD) % RD>(), st + RD);
      });
      __syncthreads();
      if constexpr (NBUF == 3) read_frags(0, 0, f0);
    }
    int cb = 0;  // LDS buffer of stage kt
    auto step = [&](auto PH, int kt) {
      constexpr int P = decltype(PH)::value;  // kt % RD
      const int nb1 = cb + 1 == NBUF ? 0 : cb + 1;
      const int nbe = NBUF == 3 ? (nb1 + 1 == NBUF ? 0 : nb1 + 1) : nb1;
      load_stage(IC<(P + D_LD) % RD>(), kt + D_LD);
      // Keep the loads at the top of the step: left alone, the scheduler sinks
      // them to the end of the step, exposing the full memory latency.
      __builtin_amdgcn_sched_barrier(0);
      store_stage(IC<(P + E_ST) % RD>(), nbe);
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (NBUF == 3) {
        compute(cb, f0);
        read_frags(nb1, 0, f0);
      } else {
        read_frags(cb, 0, f0);
        compute(cb, f0);
      }
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
      cb = nb1;
    };
    // Whole groups of RD steps without branches (a step skipped on some path
    // would make the compiler wait for every load in flight where the paths
    // merge), then the remaining steps.
    int kt = 0;
    for (; kt + RD <= nk; kt += RD) static_for<0, RD>([&](auto PH) { step(PH, kt + decltype(PH)::value); });
    static_for<0, RD - 1>([&](auto PH) {
      constexpr int P = decltype(PH)::value;
      if (kt + P < nk) step(PH, kt + P);
    });
  }
  // ---- cross-wave reduction over the WK k-split (fixed order) ----------------
  // Block b = i*FN + j of the wave tile is owned by wave wk == b % WK.  In phase
  // r the wave hands block b to owner (wk + r) % WK through LDS.
  if constexpr (WK > 1) {
    char *slot_base = smem + (wm * WN + wn) * WK * OWN * 4096;
#pragma unroll
    for (int r = 1; r < WK; ++r) {
      const int to = (wk + r) % WK;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        if (b % WK == to) {
          char *p = slot_base + (to * OWN + b / WK) * 4096 + lane * 16;
#pragma unroll
          for (int q = 0; q < 4; ++q)
            *(f32x4 *)(p + q * 1024) = f32x4{acc[b / FN][b % FN][4 * q + 0], acc[b / FN][b % FN][4 * q + 1],
                                             acc[b / FN][b % FN][4 * q + 2], acc[b / FN][b % FN][4 * q + 3]};
        }
      }
      __syncthreads();
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        if (b % WK == wk) {
          const char *p = slot_base + (wk * OWN + b / WK) * 4096 + lane * 16;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const f32x4 v = *(const f32x4 *)(p + q * 1024);
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[b / FN][b % FN][4 * q + e] += v[e];
          }
        }
      }
      __syncthreads();
    }
  }

  // ---- sum of partial rank-r products: store (loads issued before the loop) --
  if (BMODE == B_ROW && g.usum_out) {
    if (us_idx >= 0) {
      if constexpr (!US_EARLY) us_load();
      float v = us_part[0];
#pragma unroll
      for (int q = 1; q < MAX_SPLIT; ++q)
        if (q < g.usum_parts) v += us_part[q];
      g.usum_out[us_idx] = v;
    }
    // elements beyond one per thread (large r with few tile columns)
    for (int e = us_first + NT; e < us_last; e += NT) {
      const int64_t o = (int64_t)(m0 + e / g.usum_r) * g.usum_r + e % g.usum_r;
      float v = g.usum_src[o];
      for (int q = 1; q < g.usum_parts; ++q) v += g.usum_src[q * (int64_t)g.M * g.usum_r + o];
      g.usum_out[o] = v;
    }
  }

  // ---- epilogue: lane holds D[n][m] at m = lane % 32, n = 8q + 4(lane / 32) + e
  if constexpr (EPI == EPI_CE_STATS) {
    // Row statistics of this tile of logits: max and sum of exp over its valid
    // columns, and the target's logit when the target column lies in the tile.
    // The fp32 tile goes through LDS; four threads share a row and combine
    // their partial max and sum in a fixed order.
    __syncthreads();
    float *zt = (float *)smem;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if (WK > 1 && b % WK != wk) continue;
      const int i = b / FN, j = b % FN;
      const int row = wm * WTM + i * 32 + lrow;
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          zt[row * (BN + 1) + wn * WTN + j * 32 + 8 * q + 4 * (lane >> 5) + e] = acc[i][j][4 * q + e];
    }
    __syncthreads();
    const int row = tid >> 2, sub = tid & 3;
    constexpr int CPT = BN / 4;  // columns per thread
    const int ncol = min(BN, g.N - n0);
    const float *zr = zt + row * (BN + 1);
    float mx = -INFINITY;
#pragma unroll
    for (int c = sub * CPT; c < (sub + 1) * CPT; ++c) mx = c < ncol ? fmaxf(mx, zr[c]) : mx;
    mx = fmaxf(mx, __shfl_xor(mx, 1));
    mx = fmaxf(mx, __shfl_xor(mx, 2));
    float sm = 0.0f;
#pragma unroll
    for (int c = sub * CPT; c < (sub + 1) * CPT; ++c) sm += c < ncol ? __expf(zr[c] - mx) : 0.0f;
    sm += __shfl_xor(sm, 1);
    sm += __shfl_xor(sm, 2);
    const int m = m0 + row;
    if (sub == 0 && m < g.M) {
      g.ce_max[(int64_t)nt * g.M + m] = mx;
      g.ce_sum[(int64_t)nt * g.M + m] = sm;
      const int tp = g.tpos[m] - g.col0 - n0;
      if (tp >= 0 && tp < ncol) g.ce_tgt[m] = zr[tp];
    }
    return;
  }
  if constexpr (EPI == EPI_TOPK) {
    // Cosines c = z * rn_a[m] * rn_b[n] of this tile; every one above the
    // row's threshold is appended to the row's candidate list.  Four threads
    // share a row, each a block of BN / 4 columns: their counts give each its
    // place after one atomic add on the row's count (the list's order is
    // irrelevant, its content is not).  The tile's rn_b sits in LDS.
    __syncthreads();
    float *zt = (float *)smem;
    float *rbs = zt + BM * (BN + 1);
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if (WK > 1 && b % WK != wk) continue;
      const int i = b / FN, j = b % FN;
      const int row = wm * WTM + i * 32 + lrow;
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          zt[row * (BN + 1) + wn * WTN + j * 32 + 8 * q + 4 * (lane >> 5) + e] = acc[i][j][4 * q + e];
    }
    if (tid < BN) rbs[tid] = n0 + tid < g.N ? g.rn_b[n0 + tid] : 0.0f;
    __syncthreads();
    const int row = tid >> 2, sub = tid & 3;
    constexpr int CPT = BN / 4;
    const int m = m0 + row;
    if (m >= g.M) return;  // all four threads of the row leave together
    const int ncol = min(BN, g.N - n0);
    const int c_lo = sub * CPT;
    const float *zr = zt + row * (BN + 1);
    const float ra = g.rn_a[m], th = g.tk_thr[m];
    int mine = 0;
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      const int cc = c_lo + c;
      mine += (cc < ncol) & (zr[cc] * ra * rbs[cc] > th);
    }
    const int l0 = lane & ~3;
    const int n0c = __shfl(mine, l0), n1c = __shfl(mine, l0 + 1), n2c = __shfl(mine, l0 + 2),
              n3c = __shfl(mine, l0 + 3);
    const int total = n0c + n1c + n2c + n3c;
    const int before = (sub > 0 ? n0c : 0) + (sub > 1 ? n1c : 0) + (sub > 2 ? n2c : 0);
    int base = 0;
    if (sub == 0 && total > 0) base = atomicAdd(g.tk_cnt + m, total);
    base = __shfl(base, l0);
    if (mine == 0) return;
    int slot = base + before;
    float *vr = g.tk_val + (int64_t)m * g.tk_cap;
    int32_t *ir = g.tk_idx + (int64_t)m * g.tk_cap;
    for (int c = 0; c < CPT; ++c) {
      const int cc = c_lo + c;
      const float v = zr[cc] * ra * rbs[cc];
      if (cc < ncol && v > th) {
        if (slot < g.tk_cap) {  // never past the list (the sizes rule it out)
          vr[slot] = v;
          ir[slot] = g.col0 + n0 + cc;
        }
        ++slot;
      }
    }
    return;
  }
  if constexpr (EPI == EPI_CE_DZ) {
    // dz = dscale * (exp(z - lse[m]) - [column is the target]), bf16; columns
    // from N up to the padded row length ldc are written as zeros.
    T *C = (T *)g.C;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if (WK > 1 && b % WK != wk) continue;
      const int i = b / FN, j = b % FN;
      const int m = m0 + wm * WTM + i * 32 + lrow;
      if (m >= g.M) continue;
      const float l = g.lse[m];
      const int tp = g.tpos[m] - g.col0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = n0 + wn * WTN + j * 32 + 8 * q + 4 * (lane >> 5);
        if (n < g.ldc) {
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e)
            v[e] = n + e < g.N ? g.dscale * (__expf(acc[i][j][4 * q + e] - l) - (n + e == tp ? 1.0f : 0.0f))
                               : 0.0f;
          const uint32_t lo = (uint32_t)E::from_float(v[0]) | ((uint32_t)E::from_float(v[1]) << 16);
          const uint32_t hi = (uint32_t)E::from_float(v[2]) | ((uint32_t)E::from_float(v[3]) << 16);
          *(uint2 *)((T *)g.C + (int64_t)m * g.ldc + n) = make_uint2(lo, hi);
        }
      }
    }
    (void)C;
    return;
  }
  if constexpr (EPI == EPI_F32) {
    // fp32 output, overwritten or (c_accumulate) added to.
    float *C = (float *)g.C;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if (WK > 1 && b % WK != wk) continue;
      const int i = b / FN, j = b % FN;
      const int m = m0 + wm * WTM + i * 32 + lrow;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = n0 + wn * WTN + j * 32 + 8 * q + 4 * (lane >> 5);
        if (m < g.M && n < g.N) {
          f32x4 *dst = (f32x4 *)(C + (int64_t)m * g.ldc + n);
          f32x4 v = f32x4{acc[i][j][4 * q + 0], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                          acc[i][j][4 * q + 3]};
          if (g.c_accumulate) v += *dst;
          *dst = v;
        }
      }
    }
    return;
  }
  T *C = (T *)g.C;
  if constexpr (DMA && WK == 1 && ES == 2) {
    // Stores staged through LDS (free once the ring has drained), 32 rows of
    // the wave's tile at a time: the lanes write their runs of 4 columns into
    // the wave's own LDS rows, then read whole 16-byte pieces back so that
    // each store instruction writes complete 128-byte lines of C.  (Storing
    // the runs directly scatters 16-byte pieces over 32 rows per
    // instruction; the staged form took 8-10 us off every wave of 256-wide
    // tiles.)  Each wave uses its own rows, and a wave's LDS accesses are
    // performed in order, so no barrier is needed.
    constexpr int ROWB = WTN * 2 + 16;        // padded LDS row
    constexpr int LPR = WTN / 8, RPI = 64 / LPR;  // lanes per row, rows per store
    static_assert(NWV * 32 * ROWB <= LDS, "staged epilogue fits the LDS");
    char *rows = smem + wave * 32 * ROWB;
    const int ncol = n0 + wn * WTN + (lane % LPR) * 8;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t lo = (uint32_t)E::from_float(acc[i][j][4 * q + 0]) |
                              ((uint32_t)E::from_float(acc[i][j][4 * q + 1]) << 16);
          const uint32_t hi = (uint32_t)E::from_float(acc[i][j][4 * q + 2]) |
                              ((uint32_t)E::from_float(acc[i][j][4 * q + 3]) << 16);
          *(uint2 *)(rows + lrow * ROWB + (j * 32 + 8 * q + 4 * (lane >> 5)) * 2) = make_uint2(lo, hi);
        }
#pragma unroll
      for (int r0 = 0; r0 < 32; r0 += RPI) {
        const int row = r0 + lane / LPR;
        if (lane < RPI * LPR && row < 32) {
          const u32x4 v = ld16(rows + row * ROWB + (lane % LPR) * 16);
          const int m = m0 + wm * WTM + i * 32 + row;
          if (m < g.M && ncol < g.N) st16(C + (int64_t)m * g.ldc + ncol, v);
        }
      }
    }
    if (coh) fz_report();
    return;
  }
  if constexpr (DMA && WK > 1 && ES == 2) {
    // The same for tiles whose waves split k: after the reduction each wave
    // owns some 32 x 32 blocks of its wave tile, so the whole tile is staged
    // in LDS (the reduction's last barrier has freed it), and after one
    // barrier every thread stores 16-byte pieces of whole rows.
    constexpr int ROWB = BN * 2 + 16;
    constexpr int LPR = BN / 8, RPR = NT / LPR;  // lanes per row, rows per round
    static_assert(BM * ROWB <= LDS, "staged epilogue fits the LDS");
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if (b % WK != wk) continue;
      const int i = b / FN, j = b % FN;
      const int row = wm * WTM + i * 32 + lrow;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t lo = (uint32_t)E::from_float(acc[i][j][4 * q + 0]) |
                            ((uint32_t)E::from_float(acc[i][j][4 * q + 1]) << 16);
        const uint32_t hi = (uint32_t)E::from_float(acc[i][j][4 * q + 2]) |
                            ((uint32_t)E::from_float(acc[i][j][4 * q + 3]) << 16);
        *(uint2 *)(smem + row * ROWB + (wn * WTN + j * 32 + 8 * q + 4 * (lane >> 5)) * 2) = make_uint2(lo, hi);
      }
    }
    __syncthreads();
    const int ncol = n0 + (tid % LPR) * 8;
#pragma unroll
    for (int r0 = 0; r0 < BM; r0 += RPR) {
      const int row = r0 + tid / LPR;
      const u32x4 v = ld16(smem + row * ROWB + (tid % LPR) * 16);
      const int m = m0 + row;
      if (m < g.M && ncol < g.N) st16(C + (int64_t)m * g.ldc + ncol, v);
    }
    if (coh) fz_report();
    return;
  }
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    if (WK > 1 && b % WK != wk) continue;
    const int i = b / FN, j = b % FN;
    const int m = m0 + wm * WTM + i * 32 + lrow;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int n = n0 + wn * WTN + j * 32 + 8 * q + 4 * (lane >> 5);
      if (m < g.M && n < g.N) {
        T *dst = C + (int64_t)m * g.ldc + n;
        if constexpr (ES == 2) {
          uint32_t lo = (uint32_t)E::from_float(acc[i][j][4 * q + 0]) |
                        ((uint32_t)E::from_float(acc[i][j][4 * q + 1]) << 16);
          uint32_t hi = (uint32_t)E::from_float(acc[i][j][4 * q + 2]) |
                        ((uint32_t)E::from_float(acc[i][j][4 * q + 3]) << 16);
          *(uint2 *)dst = make_uint2(lo, hi);
        } else {
          *(f32x4 *)dst = f32x4{acc[i][j][4 * q + 0], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                acc[i][j][4 * q + 3]};
        }
      }
    }
  }
  // A fused tile wave whose wait gave up is counted once its stores are out.
  if (coh) fz_report();
}

// Tile rows per XCD group: each XCD's ~ntiles/8 consecutive tiles form a block
// of about sqrt(c * BN / BM) tile rows, which minimises the A rows plus B
// columns it streams.
static inline int pick_group_m(int tiles_m, int tiles_n, int BM, int BN) {
  const double c = (double)tiles_m * tiles_n / 8.0;
  int gmv = (int)(__builtin_sqrt(c * BN / BM) + 0.5);
  if (gmv < 1) gmv = 1;
  if (gmv > tiles_m) gmv = tiles_m;
  return gmv;
}

template <class E, int BM, int BN, int WM, int WN, int WK, int BMODE, int BKB, int NBUF, int RD, int FS,
          int QB = 0, int EPI = EPI_STORE, int DMA = 0>
static hipError_t launch_cfg(const GemmArgs &g, const SideArgs *side, hipStream_t st, FuseArgs *fz = nullptr) {
  const int tm = g.M > 0 ? (g.M + BM - 1) / BM : 0, tn = (g.N + BN - 1) / BN;
  // Direct-to-LDS tiles address a k-major B2 with B's per-lane offsets.
  if (DMA && BMODE == B_KMAJ_TR && g.r > 0 && g.ldb2 != g.ldb) return hipErrorInvalidValue;
  SideArgs sa{};
  int nside = 0;
  if (side) {
    sa = *side;
    nside = side_workgroups(&sa, std::is_same<E, BF16>::value ? DT_BF16 : DT_F32);
  }
  FuseArgs fa{};
  if (fz && fz->nprod > 0) {
    // Side items of a fused launch run on the producer workgroups.
    nside = 0;
    // 16 rows per producer while they fit beside the tiles on the 256 CUs (a
    // tile needs the producers' rows only in its last steps), else 32, else
    // (256 x 256 tiles) 64.
    const int free = 256 - tm * tn;
    const int64_t T = fz->row.M;
    const int mb = ((T + 15) / 16 + 7) / 8 * 8 <= free ? 1 : ((T + 31) / 32 + 7) / 8 * 8 <= free || BM * BN != 65536 ? 2 : 4;
    fz->row.mb = mb;
    fz->nprod = (int)((T + 16 * mb - 1) / (16 * mb));
    fz->ncons = fz->hold ? 0 : tm * tn;  // consumers: the tiles (0: every wait gives up)
    fz->nwg = (fz->nprod + 7) / 8 * 8;
    fa = *fz;
  }
  if (BMODE == B_ROW && nside > 0) return hipErrorInvalidValue;  // side items run in k-major launches only
  const int grid = tm * tn + nside + fa.nwg;
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_kernel<E, BM, BN, WM, WN, WK, BMODE, BKB, NBUF, RD, FS, QB, EPI, DMA>), dim3(grid),
                     dim3(64 * WM * WN * WK), 0, st, g, tm > 0 ? pick_group_m(tm, tn, BM, BN) : 1,
                     sa, nside, fa);
  return hipGetLastError();
}

// Tile shape per problem: an estimate of the time of each candidate -- full
// waves of tiles over the 256 CUs times the per-tile cost.  Relative per-CU
// throughput measured on MI355X at T = 2048 and 4096 over the shapes of the
// Llama and Qwen layers, for 128x128, 256x128 (8 waves, 64-deep stages) and
// 256x256 (4 waves of 128x128, 32-deep stages), all direct-to-LDS: row-major
// B 0.84 : 0.99 : 1.02; k-major B (the transposed reads cost the small tile
// more) 0.76 : 1.04 : 1.11.  128x64 (0.56 row-major, 0.47 k-major) only where
// 128x128 tiles would leave most CUs idle (the Qwen k/v forward, 2048 -> 256).
// 256x192 (4 waves of 128x96, 32-deep stages; 0.88 row-major, 0.91 k-major)
// where it alone fills the 256 CUs in one wave: a 4096 x 3072 output, 5-8 %
// faster there than three waves of 128x128 or 192 tiles of 256x256.  Not for
// launches with token-reduction side items: with every CU holding a tile,
// those run after the tiles instead of beside them (+7 % on such launches).
// Returns 0: 128x128, 1: 256x128, 2: 256x256, 3: 128x64, 4: 256x192.
static inline int pick_shape(int M, int N, bool b_kmajor, bool with_side) {
  auto cost = [&](int bm, int bn, double eff) {
    const long tiles = (long)((M + bm - 1) / bm) * ((N + bn - 1) / bn);
    return (double)((tiles + 255) / 256) * bm * bn / eff;
  };
  const double c0 = cost(128, 128, b_kmajor ? 0.76 : 0.84), c1 = cost(256, 128, b_kmajor ? 1.04 : 0.99),
               c2 = cost(256, 256, b_kmajor ? 1.11 : 1.02), c3 = cost(128, 64, b_kmajor ? 0.47 : 0.56),
               c4 = cost(256, 192, b_kmajor ? 0.91 : 0.88);
  if (!with_side && c4 < c0 && c4 < c1 && c4 < c2 && c4 < c3) return 4;
  if (c3 < c0 && c3 < c1 && c3 < c2) return 3;
  if (c2 <= c1 && c2 <= c0) return 2;
  return c1 < c0 ? 1 : 0;
}

}  // namespace lora
