// The bf16 MFMA grouped GEMM of the expert layer and the helpers that the
// forward (grouped_ffn.hip) and the backward (grouped_ffn_bwd.hip) share:
// C[m][n] = sum_k A[m][k] B_e[n][k] over a tile list of one device's groups.
//
// bf16 path: one persistent workgroup per CU walks a tile list built on the
// device from the group table (no host round trip); a tile never spans two
// groups. Tiles are handed out so that the workgroups resident on one XCD
// (the hardware deals workgroup ids round-robin over the 8 XCDs) work on
// neighbouring tiles, which share operand panels in that XCD's L2. Each tile
// is 256 x BN, eight waves (two per SIMD) with v_mfma_f32_32x32x16_bf16 and
// fp32 accumulators in registers; operands stream global -> LDS by DMA
// through a ring of 32-deep k-slices, and MFMA fragments are double-buffered
// in registers. The same kernel serves the backward's GEMMs (see the
// epilogues below).
//
// Packed weights (llep_pack_weights) keep the contraction dimension last, so
// both GEMMs read 16-byte runs along K for A and B alike. In the gate/up
// matrix, gate columns 32j..32j+31 are followed by the matching up columns,
// so one wave holds gate and up values of the same output element in the
// same accumulator register slot and applies SwiGLU without data exchange.
#pragma once

#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace llep {

constexpr int kTileM = 256;  // rows per GEMM tile (one m-tile never spans two groups)
#ifndef LLEP_GEMM_WAVES
#define LLEP_GEMM_WAVES 8
#endif
// wave layout of a 256 x 256 tile (and of the 256 x 192 down-projection tile)
#ifndef LLEP_GEMM2_WAVES
#define LLEP_GEMM2_WAVES LLEP_GEMM_WAVES
#endif
// waves along M of the 256 x 256 tile: 2 x 4 (128 x 64 per wave); 4 x 2
// (64 x 128) measured within 1% of it
#ifndef LLEP_WAVES_M256
#define LLEP_WAVES_M256 2
#endif
constexpr int kWavesM = LLEP_WAVES_M256, kWavesN = LLEP_GEMM_WAVES / LLEP_WAVES_M256;
constexpr int kWavesM192 = LLEP_GEMM2_WAVES / 2, kWavesN192 = 2;
#ifndef LLEP_GROUP_M
#define LLEP_GROUP_M 8
#endif
constexpr int kGroupM = LLEP_GROUP_M;  // m-tiles per super-row of the tile order

// ---------------------------------------------------------------------------
// bf16 MFMA grouped GEMM: C[m][n] = sum_k A[m][k] B_e[n][k]
// ---------------------------------------------------------------------------

// Epilogues: the forward projections (plain bf16 C, or SwiGLU of gate/up
// column pairs; a training forward also stores the gate / up values), the
// SwiGLU backward (C = d act; reads the gate / up values, writes their
// gradients and the activation), and the backward's
// multi-problem launch: the input-gradient tiles (plain bf16 C) together with
// the tiles of the two weight gradients (fp32, per expert; gate/up columns
// de-interleaved), handed out through a work counter.
enum Epilogue : int { kEpiPlain = 0, kEpiSwiglu = 1, kEpiSwigluBwd = 2, kEpiBwdMulti = 3 };

// A weight-gradient problem: per expert e, C_e[m][n] = sum over the k-segment
// of e of A[m][k] B[n][k], both operands blocked over the whole k range.
struct WgProblem {
  const uint16_t *A, *B;  // blocked [M][kmax], [N][kmax]
  int64_t blk_stride;     // bytes per 16-row block of A and B (kmax / 32 KB)
  float *C, *C2;          // C [E][M][N] fp32; gate/up problem: gate into C, up into C2,
                          // each [E][M][N / 2]
  int64_t expert_stride;  // elements per expert of C (and C2)
  int32_t M, N, gate_up;
};

struct GemmArgs {
  const uint16_t *A;
  int64_t lda;           // row-major A: elements per row
  int64_t a_blk_stride;  // blocked A: bytes per 16-row block across all of K
  const uint16_t *B;
  int64_t b_expert_stride;  // elements between experts' packed B
  int64_t b_blk_stride;     // bytes per 16-row block of B across all of K
  uint16_t *C;
  int64_t ldc;
  const int32_t *groups;
  const int4 *tiles;        // forward: (group, m-tile, padded first row, 0)
  const int32_t *n_mtiles;
  int32_t N, Kdim;
  // forward SwiGLU, training: the raw gate / up values, row-major by x_perm
  // row (ld = N, gate / up interleaved per 32 as in the packed weights);
  // null: not written
  uint16_t *gu_save;
  // SwiGLU backward: reads the gate / up values (row-major by x_perm row,
  // ld 2F, interleaved per 32); writes [d g | d u] blocked over padded rows
  // (C) and [d g | d u] and the activation transposed into the
  // weight-gradient layout: blocks of 16 columns x 32 rows over
  // [columns][kmax], the rows of group g starting at kbase[g]
  const uint16_t *GU;
  uint16_t *dgu_t, *act_t;
  const int32_t *kbase;
  int64_t kmax;
  // multi-problem backward launch: weight-gradient tiles of the experts in
  // wg_experts (longest k-segment first), problem wp[0] then wp[1] per
  // expert, and the tiles of the main problem, handed out longest first
  // (LaunchSched::decode); tiles past the first gridDim come from the
  // counter *queue (zero before the launch)
  WgProblem wp[2];
  const int4 *wg_experts;  // (expert, first k-slice, k-slices, 0)
  const int32_t *n_wg;
  const int32_t *n_wg_long;  // the first of them whose tiles are at least as long as a main tile
  int32_t *queue;
};


// ---------------------------------------------------------------------------
// bf16 MFMA grouped GEMM, 256 x BN tiles, eight waves of WM x WN.
//
// Operand tiles move global -> LDS directly (global_load_lds_dwordx4: no VGPR
// staging) in k-slices of 32, through a ring of kStages LDS stages with
// kAhead slices requested ahead of the one being read. Waits count
// outstanding DMA instructions (they complete in issue order), one barrier
// per slice.
//
// LDS stage layout: rows of 32 bf16 (64 B = 4 chunks of 16 B); chunk index
// XORed with (row / 4) % 4. A ds_read_b128 serves 16 lanes per cycle from 64
// four-byte banks; the fragment reads put 16 consecutive rows (4 rows per
// 256-B bank line) in one group, and the XOR spreads them over all banks.
// One DMA instruction fills 1 KB = 16 rows: lane l writes row l / 4, chunk
// slot l % 4, so it loads logical chunk (l % 4) ^ ((l / 16) % 4).
// ---------------------------------------------------------------------------

typedef __attribute__((address_space(3))) void *lds_void_ptr;
typedef __attribute__((address_space(1))) void *gbl_void_ptr;

constexpr int kSK = 32;      // k-slice per LDS stage
constexpr int kAhead = 4;    // slices requested ahead of the one being read
// One stage more than the look-ahead: slice kt+kAhead goes into the buffer
// of slice kt-1 (free since the previous barrier), requested half before the
// barrier that releases slice kt+1 and half after it, so after a barrier the
// MFMAs restart at once.
constexpr int kStages = kAhead + 1;

// The DMA is issued through asm so the compiler does not treat it as a
// pending LDS write: it would otherwise wait for every DMA in flight before
// each LDS read. The kernel orders DMA and reads itself (wait_cnt + barrier);
// DMA completions are in issue order, so the compiler's own vmcnt waits for
// other loads stay correct (they can only wait longer). The global address
// is a wave-uniform 64-bit base in SGPRs plus a per-lane 32-bit byte offset
// (the instruction's saddr form), so no lane computes a 64-bit address; the
// LDS destination (1 KB, 16 bytes per lane) starts at m0.
__device__ __forceinline__ void dma16(const char *base_in, int32_t voff, uint32_t lds) {
  // the base is wave-uniform by construction; readfirstlane states it (the
  // builtin returns int: both halves are widened as unsigned)
  const uint64_t bv = reinterpret_cast<uint64_t>(base_in);
  const uint32_t lo = uint32_t(__builtin_amdgcn_readfirstlane(uint32_t(bv)));
  const uint32_t hi = uint32_t(__builtin_amdgcn_readfirstlane(uint32_t(bv >> 32)));
  const uint64_t base = (uint64_t(hi) << 32) | uint64_t(lo);
  // the LDS address is wave-uniform too (free when it already sits in a
  // scalar register)
  const uint32_t lds_u = uint32_t(__builtin_amdgcn_readfirstlane(lds));
  // m0 is reserved to the compiler: saved and restored inside the asm
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, %3\n\t"
      "s_nop 0\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds_u), "v"(voff), "s"(base)
      : "memory");
}

// LDS byte address of a shared-memory object (wave-uniform; once per kernel)
__device__ __forceinline__ uint32_t lds_addr(const void *p) {
  return __builtin_amdgcn_readfirstlane(
      static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void_ptr)(p))));
}

// s_waitcnt vmcnt(n) (expcnt / lgkmcnt not waited on)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

// s_waitcnt vmcnt(VM) lgkmcnt(LGKM)
template <int VM, int LGKM>
__device__ __forceinline__ void wait_cnt() {
  static_assert(VM >= 0 && VM < 64 && LGKM >= 0 && LGKM < 16, "waitcnt");
  __builtin_amdgcn_s_waitcnt((VM & 15) | ((VM >> 4) << 14) | 0x70 | (LGKM << 8));
}

// Wait until at most VM of this wave's DMA instructions are in flight and
// its LDS reads are done, then meet the other waves. The compiler-level
// fences keep LDS reads from being moved across the barrier (s_barrier alone
// does not order them, and no hardware wait is emitted for DMA targets).
template <int VM>
__device__ __forceinline__ void wait_and_sync() {
  asm volatile("" ::: "memory");
  wait_cnt<VM, 0>();
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ int lds_swz32(int row, int kc) {
  return row * kSK + ((kc ^ ((row >> 2) & 3)) << 3);
}

// v_permlane32_swap: lanes 32..63 of `lo` trade places with lanes 0..31 of
// `hi`. Lanes l and l + 32 of an accumulator block hold four columns each of
// the same row, 4 apart; one swap per register pair turns them into eight
// consecutive columns per lane, so a row's values move as 16-byte runs.
__device__ __forceinline__ void swap_halves(uint32_t &lo, uint32_t &hi) {
  const auto r = __builtin_amdgcn_permlane32_swap(lo, hi, false, false);
  lo = r[0];
  hi = r[1];
}

struct TileCoord {
  int e, row0, prow0, m0, rows_valid, n0, cols_valid, k0, nk, grp;
  int p, N;  // problem (0: the main one, 1 / 2: wp[0] / wp[1]) and its columns
  int mt;    // entry of the tile list (the forward's single-launch form)
};

template <int BM, int BN>
__device__ __forceinline__ bool decode_tile(const GemmArgs &g, int u, int n_mt, int n_nt,
                                            TileCoord &t) {
  if (u >= n_mt * n_nt) return false;
  const int sr = u / (kGroupM * n_nt);
  const int rem = u - sr * (kGroupM * n_nt);
  const int gm = min(kGroupM, n_mt - sr * kGroupM);
  const int nt = rem / gm;
  const int4 te = g.tiles[sr * kGroupM + rem % gm];
  const int32_t *gr = g.groups + 4 * te.x;
  t.grp = te.x;
  t.e = gr[1];
  t.row0 = gr[2];
  t.prow0 = te.z;
  t.m0 = te.y * BM;
  t.rows_valid = min(BM, gr[3] - t.m0);
  t.n0 = nt * BN;
  t.cols_valid = min(BN, g.N - t.n0);
  t.k0 = 0;
  t.nk = g.Kdim / kSK;
  t.p = 0;
  t.N = g.N;
  return true;
}

// weight-gradient tile u < n_exp * (tiles of wp[0] + tiles of wp[1]):
// expert-major, then problem, then m-tile, then n-tile; the contraction runs
// over the expert's k-segment
template <int BM, int BN>
__device__ __forceinline__ void decode_tile_wg(const GemmArgs &g, int u, int per0, int per1,
                                               TileCoord &t) {
  const int i = u / (per0 + per1);
  int rem = u - i * (per0 + per1);
  const bool second = rem >= per0;
  rem -= second ? per0 : 0;
  const int M = second ? g.wp[1].M : g.wp[0].M;
  const int N = second ? g.wp[1].N : g.wp[0].N;
  const int n_nt = (N + BN - 1) / BN;
  const int4 we = g.wg_experts[i];
  t.grp = 0;
  t.e = we.x;
  t.row0 = 0;
  t.prow0 = 0;
  t.m0 = (rem / n_nt) * BM;
  t.rows_valid = min(BM, M - t.m0);
  t.n0 = (rem % n_nt) * BN;
  t.cols_valid = min(BN, N - t.n0);
  t.k0 = we.y;
  t.nk = we.z;
  t.p = second ? 2 : 1;
  t.N = N;
}

// Byte size of the LDS ring of a 256 x BN tile (kStages stages of A and B
// slices).
template <int BN>
constexpr uint32_t ring_bytes() {
  return uint32_t(kStages) * (256 * kSK * 2 + BN * kSK * 2);
}

// Tile hand-out of a persistent launch, as the tile loop below sees it:
//   request()  thread 0, at the start of every tile: ask for the next tile
//              (e.g. from a counter) while the current one computes;
//   next(t)    all threads, after the tile's main loop and its closing
//              barrier: true with t the next tile of this loop (its first
//              slices are requested during the epilogue), false when this
//              loop ends after the current tile;
//   done(c, more)  all threads, after tile c's epilogue (its stores issued;
//              more: another tile of this loop follows);
//   kCoherentC whether C is stored device-coherent (read by other tiles of
//              the same launch).
//
// LaunchSched serves a launch of one problem: tiles (it * G + slot) of the
// tile order, or, in the backward's multi-problem launch, the weight-gradient
// tiles and then the main problem's tiles from the work counter g.queue (the
// first G implicitly: tile blockIdx-derived slot).
template <int BM, int BN, bool kMulti>
struct LaunchSched {
  static constexpr bool kCoherentC = false;  // C is read only by later launches
  GemmArgs g;  // a copy (no reference to the kernel argument: its fields
               // then stay in registers)
  int n_mt, n_nt, per0, per1, n_wgt, n_long, G, slot, it;
  int32_t *s_next;  // LDS: the next tile from the counter (multi-problem launch)

  __device__ __forceinline__ LaunchSched(const GemmArgs g_, int32_t *s_next_) : g(g_), s_next(s_next_) {
    n_mt = *g.n_mtiles;
    n_nt = (g.N + BN - 1) / BN;
    per0 = per1 = n_wgt = n_long = 0;
    if constexpr (kMulti) {
      per0 = ((g.wp[0].M + BM - 1) / BM) * ((g.wp[0].N + BN - 1) / BN);
      per1 = ((g.wp[1].M + BM - 1) / BM) * ((g.wp[1].N + BN - 1) / BN);
      n_wgt = *g.n_wg * (per0 + per1);
      n_long = *g.n_wg_long * (per0 + per1);
    }
    G = gridDim.x;  // a multiple of 8
    // the hardware deals workgroups round-robin over the 8 XCDs: slot gives
    // each XCD a contiguous block of G / 8 tiles of every round
    slot = (blockIdx.x % 8) * (G / 8) + blockIdx.x / 8;
    it = 0;
  }
  // The multi-problem launch hands its tiles out longest first, so that the
  // last ones to start are short and the workgroups finish together: the
  // weight-gradient tiles of the experts whose k-segment is at least as long
  // as a main tile's, then the main tiles, then the other weight-gradient
  // tiles.
  __device__ __forceinline__ bool decode(int u, TileCoord &c) const {
    if constexpr (kMulti) {
      const int n_main = n_mt * n_nt;
      if (u < n_long || (u >= n_long + n_main && u < n_wgt + n_main)) {
        decode_tile_wg<BM, BN>(g, u < n_long ? u : u - n_main, per0, per1, c);
        return true;
      }
      return decode_tile<BM, BN>(g, u - n_long, n_mt, n_nt, c);
    }
    return decode_tile<BM, BN>(g, u, n_mt, n_nt, c);
  }
  __device__ __forceinline__ bool first(TileCoord &t) { return decode(slot, t); }
  __device__ __forceinline__ void request() {
    if (kMulti && threadIdx.x == 0) *s_next = atomicAdd(g.queue, 1) + G;
  }
  __device__ __forceinline__ bool next(TileCoord &t) {
    ++it;
    // (the value every thread reads from LDS is the same: stated, so the
    // tile's coordinates stay in scalar registers)
    return decode(kMulti ? __builtin_amdgcn_readfirstlane(*s_next) : it * G + slot, t);
  }
  __device__ __forceinline__ void done(const TileCoord &, bool) {}
};

// A is row-major (lda) or, with kABlocked, in 16 x 32 blocks over padded
// rows; C likewise with kCBlocked. B is always in 16 x 32 blocks.
//
// The tile loop of one workgroup: tiles from `sched`, starting with t (none
// of whose slices has been requested yet), through the LDS ring at `smem`
// (ring_bytes<BN>() bytes, 1 KB aligned).
template <int BN, int WAVES_M, int WAVES_N, int kEpi, bool kABlocked, bool kCBlocked,
          class Sched>
__device__ __forceinline__ void gemm_tiles(const GemmArgs g, char *smem, TileCoord t,
                                           Sched &sched) {
  constexpr int BM = 256;
  constexpr int NW = WAVES_M * WAVES_N;
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr bool kSwiglu = kEpi == kEpiSwiglu;
  constexpr bool kMulti = kEpi == kEpiBwdMulti;
  // DMA blocks (16 rows each) per stage, dealt round-robin over the waves:
  // every wave has A_PER_WAVE A blocks and B_FULL B blocks, the first B_REM
  // waves one B block more. Waits count the PER_STAGE instructions every
  // wave issues per slice (conservative for the waves with one more).
  constexpr int A_BLOCKS = BM / 16, B_BLOCKS = BN / 16;
  // Half the waves (one per SIMD) issue all the DMA: a DMA instruction that
  // waits for room in the memory pipeline then holds up only that wave,
  // while the other wave on the SIMD keeps issuing MFMAs (+4% measured).
  constexpr int NWD = NW / 2;
  constexpr int A_PER_WAVE = A_BLOCKS / NWD;
  constexpr int B_FULL = B_BLOCKS / NWD, B_REM = B_BLOCKS % NWD;
  constexpr int B_SLOTS = B_FULL + (B_REM ? 1 : 0);
  constexpr int PER_STAGE = A_PER_WAVE + B_FULL;
  constexpr uint32_t A_STAGE_BYTES = BM * kSK * 2, B_STAGE_BYTES = BN * kSK * 2;
  static_assert(A_BLOCKS % NWD == 0 && PER_STAGE > 0 && NWD <= NW, "DMA split");
  static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile");
  static_assert(kAhead == 4, "waits below are written for four slices ahead");
  static_assert(!kSwiglu || (WN % 64) == 0, "SwiGLU needs gate/up column pairs per wave");
  // stage s: A rows at s * STAGE_BYTES, then B rows; the last two stages are
  // also the epilogue's staging area
  constexpr uint32_t STAGE_BYTES = A_STAGE_BYTES + B_STAGE_BYTES;
  static_assert(kStages * STAGE_BYTES == ring_bytes<BN>(), "ring size");
  auto stageA = [&](int st) { return reinterpret_cast<const uint16_t *>(smem + st * STAGE_BYTES); };
  auto stageB = [&](int st) {
    return reinterpret_cast<const uint16_t *>(smem + st * STAGE_BYTES + A_STAGE_BYTES);
  };

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
  const int64_t lda_b = g.lda * 2;
  const uint32_t sA0 = lds_addr(smem), sB0 = sA0 + A_STAGE_BYTES;

  const char *Ab, *Bb;
  int32_t offA[A_PER_WAVE], offB[B_SLOTS];
  auto setup = [&](const TileCoord &c) {
    // The lane-derived parts are recomputed for every tile from a lane index
    // the compiler cannot hoist out of the tile loop, so they occupy no
    // register across it. A 16 x 32 block is 1 KB; lane l fills LDS bytes
    // 16l .. 16l+15 = row l / 4, chunk slot l % 4, which holds logical
    // chunk kc_load of that row.
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int kc_load = (ln & 3) ^ ((ln >> 4) & 3);
    const int32_t blk_lane = (ln >> 2) * 64 + kc_load * 16;
    const uint16_t *Ap = g.A, *Bp = g.B;
    int64_t a_bs = g.a_blk_stride, b_es = g.b_expert_stride, b_bs = g.b_blk_stride;
    if (kMulti && c.p != 0) {
      const bool second = c.p == 2;
      Ap = second ? g.wp[1].A : g.wp[0].A;
      Bp = second ? g.wp[1].B : g.wp[0].B;
      a_bs = b_bs = second ? g.wp[1].blk_stride : g.wp[0].blk_stride;
      b_es = 0;
    }
    // rows (columns) past the tile's valid ones re-read its last valid row
    // (block), so every address stays in bounds
    if (kABlocked) {
      // padded rows of the group; weight gradients: rows of the expert's
      // M x K operand (prow0 = 0), from its k-segment on
      const int64_t rb0 = (c.prow0 + c.m0) >> 4;
      Ab = reinterpret_cast<const char *>(Ap) + rb0 * a_bs + int64_t(c.k0) * 1024;
#pragma unroll
      for (int j = 0; j < A_PER_WAVE; ++j) {
        const int rb = min(wave + NWD * j, (c.rows_valid - 1) >> 4);
        offA[j] = int32_t(rb * a_bs + blk_lane);
      }
    } else {
      Ab = reinterpret_cast<const char *>(g.A) + int64_t(c.row0 + c.m0) * lda_b;
      // 24-bit operands (r < 256, lda_b <= 2 * LLEP_MAX_FFN_DIM bytes): one
      // multiply-add with a 32-bit addend per offset
      const uint32_t lda_b32 = uint32_t(lda_b);
#pragma unroll
      for (int j = 0; j < A_PER_WAVE; ++j) {
        const int r = min((wave + NWD * j) * 16 + (ln >> 2), c.rows_valid - 1);
        offA[j] = int32_t(__umul24(uint32_t(r), lda_b32) + uint32_t(kc_load * 16));
      }
    }
    Bb = reinterpret_cast<const char *>(Bp) + int64_t(c.e) * b_es * 2 + (c.n0 >> 4) * b_bs +
         int64_t(c.k0) * 1024;
#pragma unroll
    for (int j = 0; j < B_SLOTS; ++j) {
      const int nb = min(wave + NWD * j, (c.cols_valid - 1) >> 4);
      offB[j] = int32_t(nb * b_bs + blk_lane);
    }
  };
  // request slice kt into stage st: 64 B per row along K for a row-major A,
  // the next 1 KB block for blocked operands
  auto issue = [&](int st, int kt) {
    const uint32_t a_st = sA0 + st * STAGE_BYTES, b_st = sB0 + st * STAGE_BYTES;
    const int kba = kABlocked ? kt * 1024 : kt * kSK * 2;
    const int kbb = kt * 1024;
#pragma unroll
    for (int j = 0; j < A_PER_WAVE; ++j)
      if (wave < NWD) dma16(Ab + kba, offA[j], a_st + (wave + NWD * j) * 1024);
#pragma unroll
    for (int j = 0; j < B_FULL; ++j)
      if (wave < NWD) dma16(Bb + kbb, offB[j], b_st + (wave + NWD * j) * 1024);
    if (B_REM != 0 && wave < B_REM)
      dma16(Bb + kbb, offB[B_SLOTS - 1], b_st + (wave + NWD * B_FULL) * 1024);
  };
  auto prologue = [&]() {
#pragma unroll
    for (int k = 0; k < kAhead; ++k)
      if (k < t.nk) issue(k, k);
  };
  setup(t);
  prologue();

  // MFMA operands of one 16-deep k-step: TM (A) and TN (B) 16-byte
  // fragments per lane. Two sets alternate: the set for the next k-step is
  // read from LDS while the current one feeds the MFMAs, so LDS latency hides
  // behind the MFMAs.
  static_assert(kSK == 32, "two k-steps per slice");
  auto read_frags = [&](int st, int ks, bf16x8 (&fa)[TM], bf16x8 (&fb)[TN]) {
    const uint16_t *a_s = stageA(st);
    const uint16_t *b_s = stageB(st);
    const int kc = ks * 2 + (lane >> 5);
#pragma unroll
    for (int i = 0; i < TM; ++i)
      fa[i] = *reinterpret_cast<const bf16x8 *>(&a_s[lds_swz32(wm * WM + i * 32 + (lane & 31), kc)]);
#pragma unroll
    for (int j = 0; j < TN; ++j)
      fb[j] = *reinterpret_cast<const bf16x8 *>(&b_s[lds_swz32(wn * WN + j * 32 + (lane & 31), kc)]);
  };
  auto mfma_step = [&](f32x16 (&acc)[TM][TN], const bf16x8 (&fa)[TM], const bf16x8 (&fb)[TN]) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[j], fa[i], acc[i][j], 0, 0, 0);
  };
  auto next_stage = [](int st) { return st + 1 == kStages ? 0 : st + 1; };

  // One k-step of MFMAs with the side work of the loop spread between them
  // in a fixed order: after MFMA s come side operations [s NS / NM,
  // (s+1) NS / NM), where side operation q < NR reads fragment q of k-step
  // ks_next of stage st_next and q >= NR issues DMA q - NR of slice kt_dma.
  // The scheduling barriers keep that order, so the memory instructions issue
  // while the MFMAs execute instead of in bursts between them.
  constexpr int NM = TM * TN, NR = TM + TN, ND = A_PER_WAVE + B_SLOTS;
  // DMA side operations of a slice in its first k-step (the rest in the
  // second); every DMA-issuing wave issues at least D0 per slice
  constexpr int D0 = PER_STAGE / 2;
  static_assert(D0 <= PER_STAGE && (kAhead - 2) * PER_STAGE + D0 < 64, "wait count");
  // dma_wave: std::true_type for the waves that issue the DMA, else
  // std::false_type (their DMA side operations are empty)
  auto side_op = [&](auto dma_wave, int q, int dma_lo, int st_next, int ks_next,
                     bf16x8 (&fa)[TM], bf16x8 (&fb)[TN], int st_dma, int kt_dma) {
    constexpr bool kDmaWave = decltype(dma_wave)::value;
    if (q < TM) {
      const uint16_t *a_s = stageA(st_next);
      fa[q] = *reinterpret_cast<const bf16x8 *>(
          &a_s[lds_swz32(wm * WM + q * 32 + (lane & 31), ks_next * 2 + (lane >> 5))]);
    } else if (q < NR) {
      const uint16_t *b_s = stageB(st_next);
      fb[q - TM] = *reinterpret_cast<const bf16x8 *>(
          &b_s[lds_swz32(wn * WN + (q - TM) * 32 + (lane & 31), ks_next * 2 + (lane >> 5))]);
    } else if constexpr (kDmaWave) {
      const int d = dma_lo + q - NR;
      const uint32_t a_st = sA0 + st_dma * STAGE_BYTES, b_st = sB0 + st_dma * STAGE_BYTES;
      const int kba = kABlocked ? kt_dma * 1024 : kt_dma * kSK * 2;
      const int kbb = kt_dma * 1024;
      if (d < A_PER_WAVE)
        dma16(Ab + kba, offA[d], a_st + (wave + NWD * d) * 1024);
      else if (d < A_PER_WAVE + B_FULL)
        dma16(Bb + kbb, offB[d - A_PER_WAVE], b_st + (wave + NWD * (d - A_PER_WAVE)) * 1024);
      else if (wave < B_REM)
        dma16(Bb + kbb, offB[B_SLOTS - 1], b_st + (wave + NWD * B_FULL) * 1024);
    }
  };
  auto interleaved_step = [&](auto dma_wave, f32x16 (&acc)[TM][TN], const bf16x8 (&fa)[TM],
                              const bf16x8 (&fb)[TN], bf16x8 (&fa_next)[TM],
                              bf16x8 (&fb_next)[TN], int st_next, int ks_next, int dma_lo,
                              int dma_hi, int st_dma, int kt_dma) {
    const int NS = NR + (dma_hi - dma_lo);
#pragma unroll
    for (int s = 0; s < NM; ++s) {
      acc[s / TN][s % TN] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
          fb[s % TN], fa[s / TN], acc[s / TN][s % TN], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int q = 0; q < NR + ND; ++q) {
        if (q < NS && q * NM >= s * NS && q * NM < (s + 1) * NS) {
          side_op(dma_wave, q, dma_lo, st_next, ks_next, fa_next, fb_next, st_dma, kt_dma);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  };

  for (;;) {
    const int nk = t.nk;
    // ask for the tile after this one (read after the barrier that ends the
    // loop; rewritten only after the barrier that ends the epilogue)
    sched.request();
    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.0f;
    // A wave whose 32 x 32 blocks all lie past the tile's last valid row or
    // column (a group's last, partly filled m-tile; the last n-tile) has no
    // MFMA work: it runs the same slice loop with the same DMA requests and
    // barriers, without LDS reads or MFMAs (its accumulators stay zero and
    // the epilogue stores none of its rows or columns).
    // (wave-uniform in a scalar register, so both sides hold their barriers
    // as a uniform branch)
    const int active =
        __builtin_amdgcn_readfirstlane(int(t.rows_valid > wm * WM && t.cols_valid > wn * WN));
    if (active) {
      bf16x8 fa0[TM], fb0[TN], fa1[TM], fb1[TN];
      // slice kt sits in stage kt % kStages; st tracks the slice being read,
      // st_req the stage of slice kt + kAhead
      int st = 0, st_req = kAhead % kStages, kt_req = kAhead;
      // slices 0 .. min(kAhead, nk) - 1 were requested; wait for slice 0
      if (nk >= kAhead)
        wait_and_sync<(kAhead - 1) * PER_STAGE>();
      else
        wait_and_sync<0>();
      read_frags(st, 0, fa0, fb0);
      int kt = 0;
      // steady state: request slice kt + kAhead, two and a half slices stay
      // in flight past slice kt + 1 (compile-time wait count). The last slice is peeled
      // so no branch joins around the LDS reads (the wait inserted at such a
      // join would drain the fresh reads).
      // (one copy of the loop for the DMA-issuing waves and one for the
      // others, so the DMA needs no per-instruction branch)
      auto steady = [&](auto dma_wave) {
        for (; kt < nk - kAhead; ++kt) {
          // k-step 0 of slice kt; reads of its k-step 1; the first D0 DMA of
          // slice kt + kAhead
          interleaved_step(dma_wave, acc, fa0, fb0, fa1, fb1, st, 1, 0, D0, st_req, kt_req);
          // slice kt + 1 has landed when at most the D0 of slice kt + kAhead
          // and all of slices kt + 2 .. kt + kAhead - 1 are in flight
          wait_and_sync<(kAhead - 2) * PER_STAGE + D0>();
          st = next_stage(st);
          // k-step 1 of slice kt; reads of k-step 0 of slice kt + 1; the rest
          // of the DMA of slice kt + kAhead (its stage, that of slice kt - 1,
          // has been free since the previous barrier)
          interleaved_step(dma_wave, acc, fa1, fb1, fa0, fb0, st, 0, D0, ND, st_req, kt_req);
          st_req = next_stage(st_req);
          ++kt_req;
        }
      };
      if (wave < NWD)
        steady(std::true_type{});
      else
        steady(std::false_type{});
      // tail: everything is requested; nk - 2 - kt slices remain past kt + 1
      for (; kt < nk - 1; ++kt) {
        read_frags(st, 1, fa1, fb1);
        mfma_step(acc, fa0, fb0);
        const int left = nk - 2 - kt;
        if (left >= 2)
          wait_and_sync<2 * PER_STAGE>();
        else if (left == 1)
          wait_and_sync<PER_STAGE>();
        else
          wait_and_sync<0>();
        st = next_stage(st);
        read_frags(st, 0, fa0, fb0);
        mfma_step(acc, fa1, fb1);
      }
      read_frags(st, 1, fa1, fb1);
      mfma_step(acc, fa0, fb0);
      mfma_step(acc, fa1, fb1);
    } else {
      int st_req = kAhead % kStages, kt_req = kAhead;
      if (nk >= kAhead)
        wait_and_sync<(kAhead - 1) * PER_STAGE>();
      else
        wait_and_sync<0>();
      int kt = 0;
      for (; kt < nk - kAhead; ++kt) {
        issue(st_req, kt_req);
        st_req = next_stage(st_req);
        ++kt_req;
        wait_and_sync<(kAhead - 1) * PER_STAGE>();
      }
      for (; kt < nk - 1; ++kt) {
        const int left = nk - 2 - kt;
        if (left >= 2)
          wait_and_sync<2 * PER_STAGE>();
        else if (left == 1)
          wait_and_sync<PER_STAGE>();
        else
          wait_and_sync<0>();
      }
    }
    // every wave is done with the ring before the next tile's slices land
    __syncthreads();
    const TileCoord c = t;
    const bool more = sched.next(t);
    // the next tile's first kAhead - 1 slices load during the epilogue; the
    // last stages hold the epilogue's staging area until the barrier below
    static_assert(kStages - (kAhead - 1) >= 2, "two stages free for staging");
    if (more) {
      setup(t);
#pragma unroll
      for (int k = 0; k < kAhead - 1; ++k)
        if (k < t.nk) issue(k, k);
    }

    // Epilogue. The MFMAs take the weight fragment as their first operand,
    // so a 32x32 accumulator block is the transposed output block: lane l
    // holds output row l % 32 and, in slots 4g .. 4g+3, the four consecutive
    // columns 8g + 4 (l / 32) + 0..3. Each wave writes its results to its own
    // part of the staging area, then reads them back in store order, so the
    // global stores are contiguous runs: whole 1 KB blocks for a blocked C,
    // WN-column row segments for a row-major C.
    constexpr uint32_t STAGING = 2 * STAGE_BYTES / NW;  // bytes per wave
    char *stg = smem + (kStages - 2) * STAGE_BYTES + wave * STAGING;
    const int rows_w = c.rows_valid - wm * WM;  // valid rows of this wave's tile part
    const int h = lane >> 5;
    auto pack2 = [](float lo, float hi) { return pack_bf16x2(lo, hi); };
    if constexpr (kSwiglu) {
      // gate columns 64p .. 64p+31 and the matching up columns 64p+32 ..
      // 64p+63 of the tile give activation columns f = 32 (pc / 64) + 0..31.
      // One activation block (16 rows x 32 columns, 1 KB) per 16 rows.
      static_assert(kCBlocked && TN % 2 == 0, "SwiGLU needs gate/up block pairs");
      static_assert((TN / 2) * (WM / 16) * 1024 <= STAGING, "staging");
      const int64_t rb0 = (c.prow0 + c.m0 + wm * WM) >> 4;
#pragma unroll
      for (int p = 0; p < TN / 2; ++p) {
        const int pc = c.n0 + wn * WN + p * 64;
        if (pc >= g.N) continue;
        char *sp = stg + p * (WM / 16) * 1024;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          char *blk = sp + (2 * i + ((lane & 31) >> 4)) * 1024 + (lane & 15) * 64;
#pragma unroll
          for (int gq = 0; gq < 4; ++gq) {
            float hv[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float gv = acc[i][2 * p][4 * gq + e], uv = acc[i][2 * p + 1][4 * gq + e];
              hv[e] = gv * __builtin_amdgcn_rcpf(1.0f + __expf(-gv)) * uv;
            }
            // 16-byte chunk gq of the row, XOR-swizzled by (row / 4) % 4 so
            // the 16 rows of a block spread over the banks
            *reinterpret_cast<uint2 *>(blk + ((gq ^ ((lane >> 2) & 3)) << 4) + 8 * h) =
                make_uint2(pack2(hv[0], hv[1]), pack2(hv[2], hv[3]));
          }
        }
        if (g.gu_save) {
          // raw gate and up values of this wave's rows: after the half-wave
          // swaps lane l stores columns 16 q + 0..7 of its row and lane
          // l + 32 columns 16 q + 8..15
#pragma unroll
          for (int i = 0; i < TM; ++i) {
            const bool row_ok = i * 32 + (lane & 31) < rows_w;
            uint16_t *gr = g.gu_save +
                           int64_t(c.row0 + c.m0 + wm * WM + i * 32 + (lane & 31)) * g.N + pc;
            const f32x16 &ga = acc[i][2 * p], &ua = acc[i][2 * p + 1];
#pragma unroll
            for (int q = 0; q < 2; ++q) {
              uint32_t g0 = pack2(ga[8 * q], ga[8 * q + 1]), g1 = pack2(ga[8 * q + 2], ga[8 * q + 3]);
              uint32_t g2 = pack2(ga[8 * q + 4], ga[8 * q + 5]), g3 = pack2(ga[8 * q + 6], ga[8 * q + 7]);
              uint32_t u0 = pack2(ua[8 * q], ua[8 * q + 1]), u1 = pack2(ua[8 * q + 2], ua[8 * q + 3]);
              uint32_t u2 = pack2(ua[8 * q + 4], ua[8 * q + 5]), u3 = pack2(ua[8 * q + 6], ua[8 * q + 7]);
              swap_halves(g0, g2);
              swap_halves(g1, g3);
              swap_halves(u0, u2);
              swap_halves(u1, u3);
              if (row_ok) {
                *reinterpret_cast<uint4 *>(gr + 16 * q + 8 * h) = make_uint4(g0, g1, g2, g3);
                *reinterpret_cast<uint4 *>(gr + 32 + 16 * q + 8 * h) = make_uint4(u0, u1, u2, u3);
              }
            }
          }
        }
        // block rb of this wave = activation row block (prow0 + m0 + wm WM) / 16 + rb
        char *dst = reinterpret_cast<char *>(g.C) + (rb0 * (g.ldc >> 5) + (pc >> 6)) * 1024 +
                    lane * 16;
#pragma unroll
        for (int rb = 0; rb < WM / 16; ++rb) {
          if (rb * 16 >= rows_w) break;  // the group's padded rows end here
          char *d = dst + int64_t(rb) * (g.ldc >> 5) * 1024;
          if constexpr (Sched::kCoherentC) {
            // device-coherent stores (written through the XCD's L2), so a
            // reader on another XCD in the same launch finds them in memory
            // once they have completed: 8 bytes per lane, lane l at bytes
            // 8 l of each half of the block, so each store instruction
            // writes 512 contiguous bytes (whole lines)
            char *blk0 = reinterpret_cast<char *>(d - lane * 16);
#pragma unroll
            for (int half = 0; half < 2; ++half) {
              const int o = half * 512 + lane * 8;  // byte of the block
              const int row = o >> 6, chunk = (o >> 4) & 3;
              const uint2 v = *reinterpret_cast<const uint2 *>(
                  sp + rb * 1024 + row * 64 + ((chunk ^ ((row >> 2) & 3)) << 4) + (o & 8));
              __hip_atomic_store(reinterpret_cast<uint64_t *>(blk0 + o),
                                 uint64_t(v.x) | (uint64_t(v.y) << 32), __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_AGENT);
            }
          } else {
            *reinterpret_cast<i32x4 *>(d) = *reinterpret_cast<const i32x4 *>(
                sp + rb * 1024 + (lane >> 2) * 64 + (((lane & 3) ^ ((lane >> 4) & 3)) << 4));
          }
        }
      }
    } else if constexpr (kEpi == kEpiSwigluBwd) {
      // C = d act for activation columns f. With g = gate, u = up (saved by
      // the forward or recomputed; row-major by x_perm row, gate f at column
      // 64 (f / 32) + f % 32, up 32 further): d gate = d act u silu'(g) and
      // d up = d act silu(g) go to C in the same layout (for dX), and d gate,
      // d up and act = silu(g) u go transposed to the weight-gradient layout:
      // a 32-row piece of the group is one 32-deep k-block there, staged in
      // LDS as [column][row] (2 KB per 32 x 32 output) and stored as two
      // 1 KB blocks. Rows past the group's end are written as zeros.
      static_assert(kCBlocked, "gate/up gradients are blocked over padded rows");
      static_assert(3 * 2048 <= STAGING, "staging");
      const int F = int(g.ldc);
      const int gu_blocks = (2 * F) >> 5;
      const int64_t kblocks = g.kmax >> 5;
      const int kb_grp = g.kbase[c.grp];
      uint16_t *st16 = reinterpret_cast<uint16_t *>(stg);
      // The 32 x 32 blocks go in order b = i TN + j; block b + 1's gate / up
      // values are requested before block b is computed and stored, so their
      // latency hides behind that work (the loads would otherwise wait for
      // the stores before them, which the compiler cannot reorder).
      auto block_ok = [&](int i, int j) {
        return i * 32 < rows_w && c.n0 + wn * WN + j * 32 < g.N;
      };
      auto gu_index = [&](int i, int j) {  // gate column 2 col0 of the lane's row
        const int row = c.row0 + c.m0 + wm * WM + i * 32 + (lane & 31);
        const int col0 = c.n0 + wn * WN + j * 32;
        return int64_t(row) * (2 * F) + 2 * col0;
      };
      auto dgu_index = [&](int i, int j) {  // blocked [padded rows][2F]
        const int pr = c.prow0 + c.m0 + wm * WM + i * 32 + (lane & 31);
        const int col0 = c.n0 + wn * WN + j * 32;
        return (int64_t(pr >> 4) * gu_blocks + (col0 >> 5) * 2) * 512 + (pr & 15) * 32;
      };
      // 16-byte loads (lane l: columns 16 q + 0..7, lane l + 32: 16 q + 8..15),
      // then half-wave swaps give each lane its accumulator columns
      // 8 gq + 4 h + 0..3
      auto load_block = [&](int i, int j, uint2 (&gw)[4], uint2 (&uw)[4]) {
        const bool ok = block_ok(i, j) && i * 32 + (lane & 31) < rows_w;
        const int64_t gb = ok ? gu_index(i, j) : 0;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const int cc = 16 * q + 8 * h;
          uint4 x = ok ? *reinterpret_cast<const uint4 *>(g.GU + gb + cc) : make_uint4(0u, 0u, 0u, 0u);
          uint4 y = ok ? *reinterpret_cast<const uint4 *>(g.GU + gb + 32 + cc)
                       : make_uint4(0u, 0u, 0u, 0u);
          swap_halves(x.x, x.z);
          swap_halves(x.y, x.w);
          swap_halves(y.x, y.z);
          swap_halves(y.y, y.w);
          gw[2 * q] = make_uint2(x.x, x.y);
          gw[2 * q + 1] = make_uint2(x.z, x.w);
          uw[2 * q] = make_uint2(y.x, y.y);
          uw[2 * q + 1] = make_uint2(y.z, y.w);
        }
      };
      uint2 gcur[4], ucur[4], gnxt[4], unxt[4];
      load_block(0, 0, gcur, ucur);
#pragma unroll
      for (int b = 0; b < TM * TN; ++b) {
        const int i = b / TN, j = b % TN;
        if (b + 1 < TM * TN) load_block((b + 1) / TN, (b + 1) % TN, gnxt, unxt);
        if (block_ok(i, j)) {
          const int rr = c.m0 + wm * WM + i * 32;  // first row of the piece in its group
          const bool row_ok = i * 32 + (lane & 31) < rows_w;
          const int64_t kb = (kb_grp + rr) >> 5;
          const int col0 = c.n0 + wn * WN + j * 32;  // first activation column f
          const int64_t gblk = dgu_index(i, j);
          // two column groups gq = 2 q, 2 q + 1 at a time (columns
          // 8 gq + 4 h + e of the 32-block; rows past the group's end 0)
          uint16_t *dgu = g.C;
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            float dg[2][4], du[2][4], av[2][4];
#pragma unroll
            for (int s = 0; s < 2; ++s) {
              const uint2 gw = gcur[2 * q + s], uw = ucur[2 * q + s];
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                dg[s][e] = du[s][e] = av[s][e] = 0.0f;
                if (row_ok) {
                  const uint32_t gbits = (e < 2 ? gw.x : gw.y) >> (16 * (e & 1));
                  const uint32_t ubits = (e < 2 ? uw.x : uw.y) >> (16 * (e & 1));
                  const float gv = __uint_as_float(gbits << 16), uv = __uint_as_float(ubits << 16);
                  const float sg = __builtin_amdgcn_rcpf(1.0f + __expf(-gv));
                  const float da = acc[i][j][4 * (2 * q + s) + e];
                  dg[s][e] = da * uv * (sg * (1.0f + gv * (1.0f - sg)));
                  du[s][e] = da * (gv * sg);
                  av[s][e] = gv * sg * uv;
                }
              }
            }
            // transposed staging: output o at o * 1024 elements, [column][row]
#pragma unroll
            for (int s = 0; s < 2; ++s)
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const int n = (8 * (2 * q + s) + 4 * h + e) * 32 + (lane & 31);
                st16[n] = f32_to_bf16(dg[s][e]);
                st16[1024 + n] = f32_to_bf16(du[s][e]);
                st16[2048 + n] = f32_to_bf16(av[s][e]);
              }
            // [d g | d u] blocked, as 16-byte runs after the half-wave swaps
            // (lane l: columns 16 q + 0..7, lane l + 32: 16 q + 8..15)
            uint32_t a0 = pack2(dg[0][0], dg[0][1]), a1 = pack2(dg[0][2], dg[0][3]);
            uint32_t a2 = pack2(dg[1][0], dg[1][1]), a3 = pack2(dg[1][2], dg[1][3]);
            uint32_t b0 = pack2(du[0][0], du[0][1]), b1 = pack2(du[0][2], du[0][3]);
            uint32_t b2 = pack2(du[1][0], du[1][1]), b3 = pack2(du[1][2], du[1][3]);
            swap_halves(a0, a2);
            swap_halves(a1, a3);
            swap_halves(b0, b2);
            swap_halves(b1, b3);
            if (row_ok) {
              *reinterpret_cast<uint4 *>(dgu + gblk + 16 * q + 8 * h) = make_uint4(a0, a1, a2, a3);
              *reinterpret_cast<uint4 *>(dgu + gblk + 512 + 16 * q + 8 * h) =
                  make_uint4(b0, b1, b2, b3);
            }
          }
          // d gate rows 64 (f / 32) + 0..31 and d up rows + 32 of [2F][kmax];
          // act rows f of [F][kmax]; 16 rows per 1 KB block. Non-temporal
          // stores: these blocks are read only by the next launch, and kept
          // out of the L2 they leave the operands of this GEMM there (0.5-1.2%
          // faster backward; the same for the blocked [d g | d u] above,
          // which the dX GEMM reads soon after, was 1-3% slower).
          const int64_t ngate = 2 * col0;  // = 64 * (col0 / 32)
#pragma unroll
          for (int bb = 0; bb < 2; ++bb) {
            const i32x4 vg = *reinterpret_cast<const i32x4 *>(stg + bb * 1024 + lane * 16);
            const i32x4 vu = *reinterpret_cast<const i32x4 *>(stg + 2048 + bb * 1024 + lane * 16);
            const i32x4 va = *reinterpret_cast<const i32x4 *>(stg + 4096 + bb * 1024 + lane * 16);
            __builtin_nontemporal_store(
                vg, reinterpret_cast<i32x4 *>(g.dgu_t + (((ngate >> 4) + bb) * kblocks + kb) * 512 +
                                              lane * 8));
            __builtin_nontemporal_store(
                vu, reinterpret_cast<i32x4 *>(
                        g.dgu_t + ((((ngate + 32) >> 4) + bb) * kblocks + kb) * 512 + lane * 8));
            __builtin_nontemporal_store(
                va, reinterpret_cast<i32x4 *>(g.act_t + (((col0 >> 4) + bb) * kblocks + kb) * 512 +
                                              lane * 8));
          }
        }
        if (b + 1 < TM * TN) {
#pragma unroll
          for (int gq = 0; gq < 4; ++gq) {
            gcur[gq] = gnxt[gq];
            ucur[gq] = unxt[gq];
          }
        }
      }
    } else {
      // fp32 weight gradient of expert c.e (problem c.p): C[m][n], rows
      // m < M, written as 16-byte runs of 4 columns. Gate/up problem: column
      // n = 64 q + cc is gate column 32 q + cc (cc < 32) or up column
      // 32 q + cc - 32.
      auto wgrad_epilogue = [&]() {
        const bool second = c.p == 2;
        float *C = second ? g.wp[1].C : g.wp[0].C;
        float *C2 = g.wp[0].C2;
        const bool gate_up = !second && g.wp[0].gate_up;
        const int64_t es = second ? g.wp[1].expert_stride : g.wp[0].expert_stride;
        // The fp32 gradients leave as whole 128-byte row pieces: each 32 x 32
        // block is written to the wave's staging area (rows RSF bytes apart,
        // so the 32 rows of a write spread over the banks) and read back so
        // that store k covers rows 8k .. 8k+7 of the block, lane l row
        // 8k + l / 8 and columns 4 (l % 8) .. 4 (l % 8) + 3. (Stored straight
        // from the accumulators, every store instruction wrote 32-byte pieces
        // of 32 rows, and the many short tiles of the small experts were
        // bound by those partial-line writes.) The stores are non-temporal:
        // nothing in the call reads the gradients back.
        constexpr int RSF = 32 * 4 + 16;
        static_assert(32 * RSF <= STAGING, "staging");
        const int ld = gate_up ? (c.N >> 1) : c.N;  // fp32 elements per gradient row
        const int rr = lane >> 3, rc = (lane & 7) * 4;  // read-back row / column of the lane
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          if (i * 32 >= rows_w) break;
          const int m0 = c.m0 + wm * WM + i * 32;  // first gradient row of the block
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const int col0 = c.n0 + wn * WN + j * 32;
            if (col0 >= c.N) continue;
            // gate / up columns are interleaved per 32 in the tile: the block
            // belongs to one of the two gradients, at column 32 (col0 / 64)
            float *base;
            if (gate_up)
              base = ((col0 & 32) ? C2 : C) + int64_t(c.e) * es + 32 * (col0 >> 6);
            else
              base = C + int64_t(c.e) * es + col0;
#pragma unroll
            for (int gq = 0; gq < 4; ++gq)
              *reinterpret_cast<f32x4 *>(stg + (lane & 31) * RSF + (8 * gq + 4 * h) * 4) =
                  f32x4{acc[i][j][4 * gq], acc[i][j][4 * gq + 1], acc[i][j][4 * gq + 2],
                        acc[i][j][4 * gq + 3]};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              const int r = 8 * k + rr;
              const f32x4 v = *reinterpret_cast<const f32x4 *>(stg + r * RSF + rc * 4);
              if (i * 32 + r < rows_w)
                __builtin_nontemporal_store(
                    v, reinterpret_cast<f32x4 *>(base + int64_t(m0 + r) * ld + rc));
            }
          }
        }
      };
      // row-major C: 32 rows x WN columns per piece, rows RS bytes apart
      auto rowmajor_epilogue = [&]() {
        static_assert(!kCBlocked, "blocked C: other epilogues");
        // row stride padded by 16 bytes: the 32 rows of a piece then fall
        // into different banks
        constexpr int RS = WN * 2 + 16;
        constexpr int CH = WN / 8;  // 16-byte chunks per row segment
        static_assert(32 * RS <= STAGING, "staging");
        const int ncol0 = c.n0 + wn * WN;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          if (i * 32 >= rows_w) break;
#pragma unroll
          for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int gq = 0; gq < 4; ++gq)
              *reinterpret_cast<uint2 *>(stg + (lane & 31) * RS + (j * 32 + 8 * gq + 4 * h) * 2) =
                  make_uint2(pack2(acc[i][j][4 * gq], acc[i][j][4 * gq + 1]),
                             pack2(acc[i][j][4 * gq + 2], acc[i][j][4 * gq + 3]));
          char *crow = reinterpret_cast<char *>(
              g.C + int64_t(c.row0 + c.m0 + wm * WM + i * 32) * g.ldc + ncol0);
#pragma unroll
          for (int r0 = 0; r0 < 32 * CH; r0 += kWave) {
            const int q = r0 + lane;
            const int row = q / CH, ch = q % CH;
            if (q < 32 * CH && i * 32 + row < rows_w && ncol0 + ch * 8 < g.N)
              *reinterpret_cast<i32x4 *>(crow + int64_t(row) * g.ldc * 2 + ch * 16) =
                  *reinterpret_cast<const i32x4 *>(stg + row * RS + ch * 16);
          }
        }
      };
      if constexpr (kMulti) {
        if (c.p != 0)
          wgrad_epilogue();
        else
          rowmajor_epilogue();
      } else {
        rowmajor_epilogue();
      }
    }
    sched.done(c, more);
    if (more) {
      // the staging area is the last stages of the ring again: every wave's
      // staging reads are done (lgkmcnt) before slice kAhead - 1 may land
      // there; the DMAs and stores in flight are not waited for
      wait_and_sync<63>();
      if (kAhead - 1 < t.nk) issue(kAhead - 1, kAhead - 1);
    }
    if (!more) break;
  }
}

// One persistent launch of one problem (forward projections, backward
// GEMMs): one workgroup per CU walks its tiles (LaunchSched).
template <int BN, int WAVES_M, int WAVES_N, int kEpi, bool kABlocked, bool kCBlocked>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N)
__attribute__((amdgpu_waves_per_eu(WAVES_M * WAVES_N / 4, WAVES_M * WAVES_N / 4)))
void gemm256_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(1024))) char smem[ring_bytes<BN>()];
  __shared__ int32_t s_next;  // multi-problem launch: the next tile from the counter
  LaunchSched<256, BN, kEpi == kEpiBwdMulti> sched(g, &s_next);
  TileCoord t;
  if (!sched.first(t)) return;
  gemm_tiles<BN, WAVES_M, WAVES_N, kEpi, kABlocked, kCBlocked>(g, smem, t, sched);
}

// ---------------------------------------------------------------------------
// Packed weights: each expert's matrix W[n][k] (n = output column of the
// GEMM, k = contraction index; K a multiple of 32) is stored in blocks of
// 16 rows x 32 k, block (n / 16, k / 32) at position (n / 16) * (K / 32) +
// k / 32, row-major inside the block. A slice of 32 k of 16 rows is one
// contiguous 1 KB (bf16) that one DMA instruction moves.
// ---------------------------------------------------------------------------

__host__ __device__ __forceinline__ int64_t packed_index(int n, int k, int K) {
  return (int64_t(n >> 4) * (K >> 5) + (k >> 5)) * 512 + (n & 15) * 32 + (k & 31);
}

// ---------------------------------------------------------------------------
// float32 path helpers: the rows and groups of a launch's device range
// ---------------------------------------------------------------------------

__device__ __forceinline__ void device_range(const int32_t *groups, const int32_t *group_begin,
                                             int device, int P, int &lo, int &hi, int &row_first,
                                             int &rows) {
  lo = device < 0 ? group_begin[0] : group_begin[device];
  hi = device < 0 ? group_begin[P] : group_begin[device + 1];
  row_first = lo < hi ? groups[4 * lo + 2] : 0;
  rows = lo < hi ? groups[4 * (hi - 1) + 2] + groups[4 * (hi - 1) + 3] - row_first : 0;
}

__device__ __forceinline__ int group_of_row(const int32_t *groups, int lo, int hi, int row) {
  // last group g in [lo, hi) with row_start <= row
  int a = lo, b = hi - 1;
  while (a < b) {
    const int mid = (a + b + 1) >> 1;
    if (groups[4 * mid + 2] <= row) a = mid;
    else b = mid - 1;
  }
  return a;
}

// number of compute units of the current device (256 if it cannot be read)
inline int cu_count() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 256;
  return n > 0 ? n : 256;
}

// Tile list of the groups of `device` (all devices with -1), in the order
// the GEMM hands tiles out; *n_tiles receives the entry count. cap: rows of
// the group table (2E + P), all of which may be read.
hipError_t launch_tile_table(const int32_t *groups, const int32_t *group_begin, int32_t cap,
                             int32_t device, int32_t P, int4 *tiles, int32_t *n_tiles,
                             hipStream_t stream);

}  // namespace llep
