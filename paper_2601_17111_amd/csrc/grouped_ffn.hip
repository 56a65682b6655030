// Step 4 of the LLEP hot path: grouped SwiGLU expert GEMMs over one device's
// groups (Alg. 4 grouped GEMMs for native and foreign experts; the
// three-matrix SwiGLU expert of Sec. 5.1).
//
// For a group (device, e, row_start, n) with X = x_perm[row_start, +n):
//   act = silu(X Wg_e) * (X Wu_e)      GEMM 1, SwiGLU fused in the epilogue
//   out = act Wd_e                      GEMM 2
//
// This file: the tile list, the forward launcher, the float32 forward (one
// thread per output element, reference precision, no matrix cores) and the
// weight packing. The GEMM kernel itself is in gemm.h.
#include <algorithm>
#include <mutex>

#include "gemm.h"

namespace llep {

struct WsLayout {
  size_t seq_off, tiles_off, done_off, act_off, total;
  int64_t max_mtiles;
};

// Workspace: the tile count (int at 0), the single launch's [2][8] queue
// counters (at 64), the tile list, its per-m-tile counters, then the
// activation.
static WsLayout ws_layout(int64_t R, int32_t E, int32_t P, int32_t F, llep_dtype dtype) {
  WsLayout L;
  const int64_t max_groups = 2 * int64_t(E) + P;
  L.max_mtiles = R / kTileM + max_groups + 1;
  L.seq_off = 64;
  L.tiles_off = 256;
  const size_t tiles_bytes = (size_t(L.max_mtiles) * 16 + 255) / 256 * 256;
  L.done_off = L.tiles_off + tiles_bytes;
  const size_t done_bytes = (size_t(L.max_mtiles) * 4 + 255) / 256 * 256;
  L.act_off = L.done_off + done_bytes;
  const size_t eb = dtype == LLEP_BF16 ? 2 : 4;
  // each group's activation rows start on a 16-row block boundary
  L.total = L.act_off + size_t(R + 16 * max_groups) * size_t(F) * eb;
  return L;
}

size_t ffn_workspace_bytes(int64_t R, int32_t E, int32_t P, int32_t F, llep_dtype dtype) {
  return ws_layout(R, E, P, F, dtype).total;
}

// ---------------------------------------------------------------------------
// tile list: one entry (group, m-tile, padded first row of the group) per BM
// rows of each group of the range. Padded rows: the groups' rows laid end to
// end with each group rounded up to a multiple of 16 (the row blocks of the
// activation matrix). Also zeroes the single launch's counters (seq [2][8]
// and done [tiles]) when given: a kernel, not a memset, so the call can be
// captured in a graph.
// ---------------------------------------------------------------------------

// Thread t holds the entries 5t .. 5t+4 of the group table (up to its
// capacity of at most kMaxChunks groups); their row counts are requested
// together with the range's bounds (no load waits for another), and the
// tile and padded-row bases are one exclusive scan: per thread, then over
// the wave's lanes, then over the four waves.
constexpr int kTileTableThreads = 256;
constexpr int kTileTablePer = (kMaxChunks + kTileTableThreads - 1) / kTileTableThreads;

__global__ __launch_bounds__(kTileTableThreads) void tile_table_kernel(
    const int32_t *__restrict__ groups, const int32_t *__restrict__ group_begin, int32_t cap,
    int32_t device, int32_t P, int32_t BM, int4 *__restrict__ tiles, int32_t *__restrict__ n_tiles,
    int32_t *__restrict__ seq, int32_t *__restrict__ done) {
  __shared__ int32_t wsum[kTileTableThreads / kWave][2];
  const int tid = threadIdx.x;
  const int lane = tid % kWave, wave = tid / kWave;
  const int lo = device < 0 ? group_begin[0] : group_begin[device];
  const int hi = device < 0 ? group_begin[P] : group_begin[device + 1];
  int32_t n[kTileTablePer];
#pragma unroll
  for (int j = 0; j < kTileTablePer; ++j)
    n[j] = groups[4 * min(kTileTablePer * tid + j, cap - 1) + 3];
  int32_t mt[kTileTablePer], pr[kTileTablePer];
  int32_t smt = 0, spr = 0;
#pragma unroll
  for (int j = 0; j < kTileTablePer; ++j) {
    const int g = kTileTablePer * tid + j;
    const bool in = g >= lo && g < hi && g < cap;
    mt[j] = in ? (n[j] + BM - 1) / BM : 0;
    pr[j] = in ? (n[j] + 15) / 16 * 16 : 0;
    smt += mt[j];
    spr += pr[j];
  }
  // inclusive scan over the wave, then the waves' totals
  int32_t imt = smt, ipr = spr;
  for (int off = 1; off < kWave; off <<= 1) {
    const int32_t a = __shfl_up(imt, off), b = __shfl_up(ipr, off);
    if (lane >= off) {
      imt += a;
      ipr += b;
    }
  }
  if (lane == kWave - 1) {
    wsum[wave][0] = imt;
    wsum[wave][1] = ipr;
  }
  __syncthreads();
  int32_t base = imt - smt, pbase = ipr - spr, total = 0;
  for (int w = 0; w < kTileTableThreads / kWave; ++w) {
    if (w < wave) {
      base += wsum[w][0];
      pbase += wsum[w][1];
    }
    total += wsum[w][0];
  }
#pragma unroll
  for (int j = 0; j < kTileTablePer; ++j) {
    const int g = kTileTablePer * tid + j;
    for (int i = 0; i < mt[j]; ++i) tiles[base + i] = make_int4(g, i, pbase, 0);
    base += mt[j];
    pbase += pr[j];
  }
  if (tid == 0) *n_tiles = total;
  if (seq != nullptr && tid < 16) seq[tid] = 0;
  if (done != nullptr)
    for (int i = tid; i < total; i += kTileTableThreads) done[i] = 0;
}

hipError_t launch_tile_table(const int32_t *groups, const int32_t *group_begin, int32_t cap,
                             int32_t device, int32_t P, int4 *tiles, int32_t *n_tiles,
                             hipStream_t stream) {
  hipLaunchKernelGGL(tile_table_kernel, dim3(1), dim3(kTileTableThreads), 0, stream, groups,
                     group_begin, cap, device, P, kTileM, tiles, n_tiles, nullptr, nullptr);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// float32 forward
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void ffn_f32_gate_up_kernel(
    const float *__restrict__ x_perm, const float *__restrict__ wgu, float *__restrict__ act,
    float *__restrict__ gu_save, const int32_t *__restrict__ groups,
    const int32_t *__restrict__ group_begin, int32_t device, int32_t P, int32_t D, int32_t F) {
  int lo, hi, row_first, rows;
  device_range(groups, group_begin, device, P, lo, hi, row_first, rows);
  const int64_t total = int64_t(rows) * F;
  for (int64_t u = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; u < total;
       u += int64_t(gridDim.x) * blockDim.x) {
    const int row = row_first + int(u / F), f = int(u % F);
    const int e = groups[4 * group_of_row(groups, lo, hi, row) + 1];
    const float *xr = x_perm + int64_t(row) * D;
    const int pg = 64 * (f / 32) + (f % 32);
    const float *we = wgu + int64_t(e) * 2 * F * D;
    float gs = 0.0f, us = 0.0f;
    for (int d = 0; d < D; ++d) {
      gs = fmaf(xr[d], we[packed_index(pg, d, D)], gs);
      us = fmaf(xr[d], we[packed_index(pg + 32, d, D)], us);
    }
    act[int64_t(row) * F + f] = gs / (1.0f + expf(-gs)) * us;
    if (gu_save) {
      gu_save[int64_t(row) * 2 * F + pg] = gs;
      gu_save[int64_t(row) * 2 * F + pg + 32] = us;
    }
  }
}

__global__ __launch_bounds__(256) void ffn_f32_down_kernel(
    const float *__restrict__ act, const float *__restrict__ wd, float *__restrict__ out,
    const int32_t *__restrict__ groups, const int32_t *__restrict__ group_begin, int32_t device,
    int32_t P, int32_t D, int32_t F) {
  int lo, hi, row_first, rows;
  device_range(groups, group_begin, device, P, lo, hi, row_first, rows);
  const int64_t total = int64_t(rows) * D;
  for (int64_t u = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; u < total;
       u += int64_t(gridDim.x) * blockDim.x) {
    const int row = row_first + int(u / D), c = int(u % D);
    const int e = groups[4 * group_of_row(groups, lo, hi, row) + 1];
    const float *ar = act + int64_t(row) * F;
    const float *we = wd + int64_t(e) * D * F;
    float s = 0.0f;
    for (int f = 0; f < F; ++f) s = fmaf(ar[f], we[packed_index(c, f, F)], s);
    out[int64_t(row) * D + c] = s;
  }
}

// ---------------------------------------------------------------------------
// One persistent launch for both projections (bf16).
//
// Work items: per m-tile of the tile list (256 rows of one group), n1
// gate/up tiles (phase 0, 256 columns of [Wg | Wu] each, SwiGLU epilogue)
// and n2 down-projection tiles (phase 1, BN2 columns of Wd each), each phase
// in super-rows of kGroupM m-tiles (phase 0 m-tile fastest, as in the
// two-launch form; phase 1 n-tile fastest). Every round of G tiles (G
// workgroups) is dealt in blocks of G / 8 consecutive tiles, one block per
// XCD, so that the
// tiles that run together on an XCD share operand panels in its L2 and the
// XCDs work on neighbouring tiles; here each XCD takes the tiles of its
// blocks from a counter, one at a time, and once its own are taken, those
// of the other XCDs (x+1, x+2, ... mod 8). A workgroup takes phase-0 tiles
// until every phase-0 queue is empty, then phase-1 tiles the same way: the
// last tiles of a phase even out over the XCDs, and the CUs left idle by the
// last round of gate/up tiles start down-projection tiles.
//
// A phase-1 tile of m-tile m reads the activations of all n1 phase-0 tiles
// of m, which may have run on other XCDs (each XCD has its own L2): phase-0
// tiles store the activations device-coherent (through the L2 to memory,
// whole 512-byte runs per store instruction), and each adds 1 to done[m]
// once its stores have completed; the phase-1 tile starts once
// done[m] == n1, then invalidates its caches (agent-scope acquire) before
// it reads them. Deadlock-free whatever number of workgroups is
// resident: a workgroup takes a phase-1 tile only after it has found every
// phase-0 queue empty, so every tile it may wait for has been taken by a
// running workgroup, and phase-0 tiles wait for nothing. The wait is
// bounded all the same: past about a second it sets LLEP_STATUS_FFN_WAIT in
// the plan's status word and goes on (the call's outputs are then
// undefined).
//
// Every output element is the same sum in the same k order as in the
// two-launch form, so the results are bit-identical to it, and do not depend
// on which device's groups a launch covers.
// ---------------------------------------------------------------------------

struct FusedFfnArgs {
  int32_t *seq;     // [2][8] tiles taken from each queue (phase 0: beyond the
                    // first G / 8, which go to the XCD's workgroups directly)
  int32_t *done;    // [m-tiles] finished phase-0 tiles per m-tile
  int32_t *status;  // the plan's status word
  int32_t n1, n2;   // n-tiles of the two phases
};

constexpr int kFfnWaitSpins = 1 << 22;  // x s_sleep 8 (512 clocks): about a second
// the wave that claims tiles: one of the waves that issue no DMA (the
// second half of the 8)
constexpr int kClaimWave = 4;
// an item is (queue << kQueueShift) | position in the queue; bit 30 marks
// a claimed item whose m-tile was seen complete at claim time
constexpr int kQueueShift = 27;
constexpr int kReadyFlag = 1 << 30;
static_assert(kClaimWave >= kWavesM * kWavesN / 2 && kClaimWave < kWavesM * kWavesN,
              "the claiming wave requests no slices");

// The tile hand-out of one phase (kPhase 0: gate/up tiles of width BN1,
// 1: down-projection tiles of width BN2) of the single launch.
template <int kPhase, int BN1, int BN2>
struct FusedSched {
  static constexpr int BN = kPhase == 0 ? BN1 : BN2;
  static constexpr bool kCoherentC = kPhase == 0;  // the activations
  const int4 *tiles;
  const int32_t *groups;
  FusedFfnArgs f;
  int n_mt, xcd, G, per_xcd;
  int nn, N, nk, total;  // n-tiles, columns, k-slices and tiles of the phase
  int cur;        // claiming wave: queues of this phase found empty so far
  int claimed;    // claiming wave: the tile claimed for after the running one
  int4 pre_te;    // claiming wave: the claimed tile's list entry
  int pre_e, pre_row0, pre_n;  // claiming wave: its group's expert, first row, rows
  int pending;    // phase 0: m-tile of the previous tile, not yet counted (or -1)
  int32_t *mailbox;  // LDS words that broadcast the claiming wave's claim

  __device__ __forceinline__ FusedSched(const GemmArgs &g, const FusedFfnArgs f_, char *smem)
      : f(f_) {
    tiles = g.tiles;
    groups = g.groups;
    n_mt = __builtin_amdgcn_readfirstlane(*g.n_mtiles);
    xcd = blockIdx.x % 8;
    G = gridDim.x;  // a multiple of 8
    per_xcd = G / 8;
    nn = kPhase == 0 ? f.n1 : f.n2;
    total = n_mt * nn;
    N = g.N;
    nk = g.Kdim / kSK;
    cur = 0;
    claimed = -1;
    pending = -1;
    mailbox = reinterpret_cast<int32_t *>(smem);
  }
  // tiles of the phase in XCD y's blocks
  __device__ __forceinline__ int length(int y) const {
    const int rounds = total / G, rem = total - rounds * G;
    return rounds * per_xcd + min(per_xcd, max(0, rem - y * per_xcd));
  }
  // the claiming wave (uniformly; its lane 0 does the atomics): the next
  // tile of this phase as an item, or -1 when every queue of the phase is
  // empty
  __device__ __forceinline__ int claim() {
    const int first = kPhase == 0 ? per_xcd : 0;  // phase 0: the first round is dealt
    while (cur < 8) {
      const int y = (xcd + cur) & 7;
      int j = 0;
      if (threadIdx.x == 64 * kClaimWave) j = atomicAdd(f.seq + 8 * kPhase + y, 1);
      j = __builtin_amdgcn_readfirstlane(j) + first;
      if (j < length(y)) return (y << kQueueShift) | j;
      ++cur;
    }
    return -1;
  }
  // all threads: the claiming wave's value (the mailbox is the first words
  // of the ring: no slice may be in flight into them, and everyone has read
  // them before the next barrier)
  __device__ __forceinline__ int broadcast(int v) {
    if (threadIdx.x == 64 * kClaimWave) *mailbox = v;
    __syncthreads();
    return __builtin_amdgcn_readfirstlane(*mailbox);
  }
  // the first tile of the phase
  __device__ __forceinline__ int first() {
    const int j0 = blockIdx.x / 8;
    if (kPhase == 0 && j0 < length(xcd)) return (xcd << kQueueShift) | j0;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int it = broadcast(wave == kClaimWave ? claim() : 0);
    __syncthreads();
    return it;
  }
  // position j of XCD y's queue = tile u of the phase's order: its n-tile
  // and its entry of the tile list
  __device__ __forceinline__ void locate(int it, int &nt, int &mt) const {
    const int y = it >> kQueueShift;
    const int j = it & ((1 << kQueueShift) - 1);
    const int u = (j / per_xcd) * G + y * per_xcd + j % per_xcd;
    const int sr = u / (kGroupM * nn);
    const int rem = u - sr * (kGroupM * nn);
    const int gm = min(kGroupM, n_mt - sr * kGroupM);
    if (kPhase == 1) {
      // down-projection tiles n-tile fastest: consecutive claims share an
      // m-tile's activation panel (fewer L2 misses: -7% fetched bytes, same
      // time)
      nt = rem % nn;
      mt = sr * kGroupM + rem / nn;
    } else {
      nt = rem / gm;
      mt = sr * kGroupM + rem % gm;
    }
  }
  __device__ __forceinline__ int mt_of(int it) const {
    int nt, mt;
    locate(it, nt, mt);
    return mt;
  }
  __device__ __forceinline__ void decode(int it, TileCoord &c) const {
    int nt, mt;
    locate(it, nt, mt);
    const int4 te = tiles[mt];
    const int32_t *gr = groups + 4 * te.x;
    fill(it, te, gr[1], gr[2], gr[3], c);
  }
  __device__ __forceinline__ void fill(int it, int4 te, int e, int row0, int n,
                                       TileCoord &c) const {
    int nt, mt;
    locate(it, nt, mt);
    c.grp = te.x;
    c.e = e;
    c.row0 = row0;
    c.prow0 = te.z;
    c.m0 = te.y * kTileM;
    c.rows_valid = min(kTileM, n - c.m0);
    c.N = N;
    c.n0 = nt * BN;
    c.cols_valid = min(BN, N - c.n0);
    c.k0 = 0;
    c.nk = nk;
    c.p = 0;
    c.mt = mt;
  }
  // thread 0: wait until every phase-0 tile of m-tile mt has stored its
  // activations (bounded; not polled when seen complete already), then
  // acquire them at agent scope
  __device__ __forceinline__ void wait_ready(int mt, bool seen = false) {
    if (threadIdx.x == 0) {
      int spins = 0;
      while (!seen &&
             __hip_atomic_load(f.done + mt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < f.n1) {
        if (++spins > kFfnWaitSpins) {
          atomicOr(f.status, LLEP_STATUS_FFN_WAIT);
          break;
        }
        __builtin_amdgcn_s_sleep(8);
      }
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      // the cache invalidation has completed before the other waves, past
      // the barrier that follows, request the activations
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
  }
  // The tile after this one is claimed at the start of this one by a wave
  // that requests no slices (the first wave past the DMA-issuing half): it
  // waits only for the atomic, while every wave waits for the tile's first
  // slice, and keeps the answer in a scalar register until the main loop
  // ends. It also reads the claimed tile's list entry and its group's
  // expert, first row and row count, which next() hands to every wave
  // through LDS: no global load then sits between this tile's main loop and
  // the next tile's first requests (about 1% on the gpt-oss-120b shapes).
  // Phase 1: the same wave also reads the claimed tile's count of finished
  // gate/up tiles; when it is complete already, the tile need not poll it
  // after the main loop.
  __device__ __forceinline__ void request() {
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (wave == kClaimWave) {
      claimed = claim();
      if (claimed >= 0) {
        pre_te = tiles[mt_of(claimed)];
        const int32_t *gr = groups + 4 * pre_te.x;
        pre_e = gr[1];
        pre_row0 = gr[2];
        pre_n = gr[3];
      }
      if (kPhase == 1 && claimed >= 0) {
        int v = 0;
        if (threadIdx.x == 64 * kClaimWave)
          v = __hip_atomic_load(f.done + mt_of(claimed), __ATOMIC_RELAXED,
                                __HIP_MEMORY_SCOPE_AGENT);
        if (__builtin_amdgcn_readfirstlane(v) >= f.n1) claimed |= kReadyFlag;
      }
    }
  }
  __device__ __forceinline__ bool next(TileCoord &t) {
    // the previous tile's activation stores completed in every wave before
    // the barrier that closed this tile's main loop (its last wait is for
    // all memory operations): count that tile now
    if (kPhase == 0 && pending >= 0) {
      if (threadIdx.x == 0)
        __hip_atomic_fetch_add(f.done + pending, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      pending = -1;
    }
    if (threadIdx.x == 64 * kClaimWave) {
      mailbox[1] = pre_te.x;
      mailbox[2] = pre_te.y;
      mailbox[3] = pre_te.z;
      mailbox[4] = pre_e;
      mailbox[5] = pre_row0;
      mailbox[6] = pre_n;
    }
    const int mine = claimed;
    const int v = broadcast(mine);
    const int it = v < 0 ? -1 : (v & ~kReadyFlag);
    if (it >= 0) {
      const int4 te = {__builtin_amdgcn_readfirstlane(mailbox[1]),
                       __builtin_amdgcn_readfirstlane(mailbox[2]),
                       __builtin_amdgcn_readfirstlane(mailbox[3]), 0};
      fill(it, te, __builtin_amdgcn_readfirstlane(mailbox[4]),
           __builtin_amdgcn_readfirstlane(mailbox[5]), __builtin_amdgcn_readfirstlane(mailbox[6]),
           t);
      if (kPhase == 1) wait_ready(t.mt, (v & kReadyFlag) != 0);
    }
    __syncthreads();  // mailbox read (and the wait done) before the ring fills
    return it >= 0;
  }
  // phase 0: the tile's activations are stored; count it for its m-tile.
  // They were stored device-coherent (written through the L2), so once every
  // wave's stores have completed they are in memory for readers on any XCD:
  // no L2 writeback is needed before the count is raised (a writeback of the
  // whole L2, even one not waited for, cost 5-7% of the call). When another
  // phase-0 tile follows, the count waits for the end of that tile's main
  // loop (next()), so the stores drain behind its first slices instead of
  // holding every wave here; the workgroup's last phase-0 tile is counted
  // at once, before any phase-1 tile is claimed or waited for.
  __device__ __forceinline__ void done(const TileCoord &c, bool more) {
    if (kPhase != 0) return;
    if (more) {
      pending = c.mt;
      return;
    }
    wait_and_sync<0>();  // every wave's stores have completed
    if (threadIdx.x == 0)
      __hip_atomic_fetch_add(f.done + c.mt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
};

template <int BN2, int WM2, int WN2>
__global__ __launch_bounds__(64 * kWavesM * kWavesN)
__attribute__((amdgpu_waves_per_eu(kWavesM * kWavesN / 4, kWavesM * kWavesN / 4)))
void ffn_fused_kernel(GemmArgs g1, GemmArgs g2, FusedFfnArgs f) {
  static_assert(WM2 * WN2 == kWavesM * kWavesN, "both phases run the same waves");
  static_assert(ring_bytes<BN2>() <= ring_bytes<256>(), "one ring serves both phases");
  __shared__ __attribute__((aligned(1024))) char smem[ring_bytes<256>()];
  TileCoord t;
  {
    FusedSched<0, 256, BN2> s0(g1, f, smem);
    const int it = s0.first();
    if (it >= 0) {
      s0.decode(it, t);
      gemm_tiles<256, kWavesM, kWavesN, kEpiSwiglu, false, true>(g1, smem, t, s0);
      // the last epilogue's staging reads are done before the ring fills again
      wait_and_sync<63>();
    }
  }
  FusedSched<1, 256, BN2> s1(g2, f, smem);
  const int it = s1.first();
  if (it >= 0) {
    s1.decode(it, t);
    s1.wait_ready(t.mt);
    __syncthreads();
    gemm_tiles<BN2, WM2, WN2, kEpiPlain, true, false>(g2, smem, t, s1);
  }
}

// ---------------------------------------------------------------------------
// launch
// ---------------------------------------------------------------------------

hipError_t launch_grouped_ffn(const FfnArgs &a, hipStream_t stream) {
  const WsLayout L = ws_layout(a.R, a.E, a.P, a.F, a.dtype);
  char *ws = static_cast<char *>(a.ws);
  int32_t *n_mtiles = reinterpret_cast<int32_t *>(ws);
  int32_t *seq = reinterpret_cast<int32_t *>(ws + L.seq_off);
  int4 *tiles = reinterpret_cast<int4 *>(ws + L.tiles_off);
  int32_t *done = reinterpret_cast<int32_t *>(ws + L.done_off);
  void *act = ws + L.act_off;
  if (a.dtype == LLEP_BF16) {
    const int grid = (cu_count() + 7) / 8 * 8;  // one workgroup per CU, XCD-balanced
    hipLaunchKernelGGL(tile_table_kernel, dim3(1), dim3(kTileTableThreads), 0, stream, a.groups,
                       a.group_begin, 2 * a.E + a.P, a.device, a.P, kTileM, tiles, n_mtiles, seq,
                       done);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    GemmArgs g1 = {};
    g1.A = static_cast<const uint16_t *>(a.x_perm);
    g1.lda = a.D;
    g1.B = static_cast<const uint16_t *>(a.w_gate_up);
    g1.b_expert_stride = int64_t(2) * a.F * a.D;
    g1.b_blk_stride = int64_t(a.D / kSK) * 1024;
    g1.C = static_cast<uint16_t *>(act);
    g1.ldc = a.F;
    g1.groups = a.groups;
    g1.tiles = tiles;
    g1.n_mtiles = n_mtiles;
    g1.N = 2 * a.F;
    g1.Kdim = a.D;
    g1.gu_save = static_cast<uint16_t *>(a.gate_up_out);
    GemmArgs g2 = g1;
    g2.gu_save = nullptr;
    g2.A = static_cast<const uint16_t *>(act);
    g2.lda = a.F;
    g2.a_blk_stride = int64_t(a.F / kSK) * 1024;
    g2.B = static_cast<const uint16_t *>(a.w_down);
    g2.b_expert_stride = int64_t(a.D) * a.F;
    g2.b_blk_stride = int64_t(a.F / kSK) * 1024;
    g2.C = static_cast<uint16_t *>(a.out_perm);
    g2.ldc = a.D;
    g2.N = a.D;
    g2.Kdim = a.F;
    // the down projection's N is D: 192-wide tiles divide D = 2880 exactly
    const bool d192 = a.D % 256 != 0 && a.D % 192 == 0;
    FusedFfnArgs f = {};
    f.seq = seq;
    f.done = done;
    f.status = a.status;
    f.n1 = (2 * a.F + 255) / 256;
    f.n2 = d192 ? a.D / 192 : (a.D + 255) / 256;
    // one launch for both projections while every tile index of a phase
    // fits the item encoding (below 2^27 tiles per phase: at D = F = 65536,
    // about 6.7 * 10^7 pairs; two launches beyond)
    if (a.status != nullptr && L.max_mtiles * std::max(f.n1, f.n2) < (int64_t(1) << kQueueShift)) {
      if (d192)
        hipLaunchKernelGGL((ffn_fused_kernel<192, kWavesM192, kWavesN192>), dim3(grid),
                           dim3(64 * kWavesM * kWavesN), 0, stream, g1, g2, f);
      else
        hipLaunchKernelGGL((ffn_fused_kernel<256, kWavesM, kWavesN>), dim3(grid),
                           dim3(64 * kWavesM * kWavesN), 0, stream, g1, g2, f);
      return hipGetLastError();
    }
    constexpr int NT = 64 * kWavesM * kWavesN;
    hipLaunchKernelGGL((gemm256_kernel<256, kWavesM, kWavesN, kEpiSwiglu, false, true>),
                       dim3(grid), dim3(NT), 0, stream, g1);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    if (d192)
      hipLaunchKernelGGL((gemm256_kernel<192, kWavesM192, kWavesN192, kEpiPlain, true, false>),
                         dim3(grid), dim3(64 * kWavesM192 * kWavesN192), 0, stream, g2);
    else
      hipLaunchKernelGGL((gemm256_kernel<256, kWavesM, kWavesN, kEpiPlain, true, false>),
                         dim3(grid), dim3(NT), 0, stream, g2);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(ffn_f32_gate_up_kernel, dim3(1024), dim3(256), 0, stream,
                     static_cast<const float *>(a.x_perm), static_cast<const float *>(a.w_gate_up),
                     static_cast<float *>(act), static_cast<float *>(a.gate_up_out), a.groups,
                     a.group_begin, a.device, a.P, a.D, a.F);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(ffn_f32_down_kernel, dim3(1024), dim3(256), 0, stream,
                     static_cast<const float *>(act), static_cast<const float *>(a.w_down),
                     static_cast<float *>(a.out_perm), a.groups, a.group_begin, a.device, a.P,
                     a.D, a.F);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// The library's own workspace for callers that cannot allocate
// (llep_grouped_ffn_noalloc): one array per GPU, held until the process ends.
// On the host `scratch` names a stand-in, not a device address: its address
// on a GPU comes from hipGetSymbolAddress with that GPU current, looked up
// once per GPU and kept; the kernels get that address, never the name.
// ---------------------------------------------------------------------------

static __device__ __align__(256) char scratch[LLEP_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxGpus = 64;

hipError_t ffn_scratch_address(void **ptr) {
  static std::mutex mu;
  static void *addr[kMaxGpus] = {};
  int dev = -1;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  if (dev < 0 || dev >= kMaxGpus) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    void *p = nullptr;
    err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (err != hipSuccess) return err;
    if (p == nullptr) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

// ---------------------------------------------------------------------------
// weight packing: tiled transposes (setup, not on the timed path)
// ---------------------------------------------------------------------------

// dst[b] at packed_index(map(c), r) = src[b][r][c]; map: 0 identity, 1 gate
// slot, 2 up slot of the interleaved gate/up layout; the contraction index r
// runs over the `rows` of src.
template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const T *__restrict__ src, T *__restrict__ dst,
                                                        int32_t rows, int32_t cols, int64_t sbs,
                                                        int64_t dbs, int32_t mode) {
  __shared__ T tile[64][65];
  const int b = blockIdx.z, r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int r = r0 + i, c = c0 + tx;
    if (r < rows && c < cols) tile[i][tx] = src[b * sbs + int64_t(r) * cols + c];
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int c = c0 + i, r = r0 + tx;
    if (c < cols && r < rows) {
      const int drow = mode == 0 ? c : 64 * (c / 32) + (c % 32) + (mode == 2 ? 32 : 0);
      dst[b * dbs + packed_index(drow, r, rows)] = tile[tx][i];
    }
  }
}

template <typename T>
static hipError_t pack_typed(int32_t E, int32_t D, int32_t F, const void *wg, const void *wu,
                             const void *wd, void *gu, void *dn, hipStream_t stream) {
  const dim3 blk(256);
  const dim3 g_gu((F + 63) / 64, (D + 63) / 64, E);
  const int64_t sbs = int64_t(D) * F, dbs_gu = int64_t(2) * F * D;
  hipLaunchKernelGGL(transpose_kernel<T>, g_gu, blk, 0, stream, static_cast<const T *>(wg),
                     static_cast<T *>(gu), D, F, sbs, dbs_gu, 1);
  hipLaunchKernelGGL(transpose_kernel<T>, g_gu, blk, 0, stream, static_cast<const T *>(wu),
                     static_cast<T *>(gu), D, F, sbs, dbs_gu, 2);
  const dim3 g_dn((D + 63) / 64, (F + 63) / 64, E);
  hipLaunchKernelGGL(transpose_kernel<T>, g_dn, blk, 0, stream, static_cast<const T *>(wd),
                     static_cast<T *>(dn), F, D, sbs, sbs, 0);
  return hipGetLastError();
}

hipError_t launch_pack(int32_t E, int32_t D, int32_t F, llep_dtype dtype, const void *w_gate,
                       const void *w_up, const void *w_down, void *gu, void *dn,
                       hipStream_t stream) {
  if (dtype == LLEP_BF16) return pack_typed<uint16_t>(E, D, F, w_gate, w_up, w_down, gu, dn, stream);
  return pack_typed<float>(E, D, F, w_gate, w_up, w_down, gu, dn, stream);
}

}  // namespace llep
