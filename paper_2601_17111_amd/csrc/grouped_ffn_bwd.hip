// Backward of step 4 of the LLEP hot path (the grouped SwiGLU expert GEMMs):
// input gradients of the range's rows and per-expert weight gradients with
// the gradient return of spilled chunks (Sec. 1 and Sec. 4: LLEP stays exact
// in training, the spilled chunks' weight gradients go back to the expert's
// native device and are added there). The GEMMs are gemm.h's kernel with its
// backward epilogues.
#include "gemm.h"

namespace llep {

// ---------------------------------------------------------------------------
// Backward of the grouped SwiGLU FFN (bf16), for the groups of one device or
// of all devices. Given d out for the groups' rows (from the combine's
// backward):
//   1. g, u = X [Wg | Wu] (row-major by x_perm row), unless the training
//      forward kept them
//   2. d act = d out Wd^T; epilogue: d g, d u and act = silu(g) u
//   3. dX = [d g | d u] [Wg | Wu]^T               (x_perm rows)
//   4. weight gradients, in fp32 per expert: the rows of an expert's groups
//      are laid end to end in gradient-return order (the group on the
//      expert's native device first, then the other devices in increasing
//      order; each group padded with zero rows to a multiple of 32), and
//      dWg | dWu = X^T [d g | d u], dWd = act^T d out contract over that
//      segment, so an expert's gradient sums its native partial and then the
//      returned partials, in a fixed order.
// ---------------------------------------------------------------------------

struct BwdLayout {
  size_t tiles_off, wge_off, kbase_off, chunk_off;
  size_t gu_off, dgu_off, xt_off, dot_off, actt_off, dgut_off, total;
  int64_t max_groups, max_mtiles, prow_max, kmax;
};

static size_t round256(size_t v) { return (v + 255) / 256 * 256; }

static BwdLayout bwd_layout(int64_t R, int32_t E, int32_t P, int32_t D, int32_t F) {
  BwdLayout L;
  L.max_groups = 2 * int64_t(E) + P;
  L.max_mtiles = R / kTileM + L.max_groups + 1;
  L.prow_max = R + 16 * L.max_groups;
  L.kmax = (R + 32 * L.max_groups + 31) / 32 * 32;
  size_t o = 256;  // counters: n_mtiles, n_wg, k-slices in use, work counter, long n_wg,
                   // copy counter
  L.tiles_off = o;  o = round256(o + size_t(L.max_mtiles) * 16);
  L.wge_off = o;    o = round256(o + size_t(E) * 16);
  L.kbase_off = o;  o = round256(o + size_t(L.max_groups) * 4);
  L.chunk_off = o;  o = round256(o + size_t(L.kmax / 32) * 4);
  L.gu_off = o;     o = round256(o + size_t(R) * 2 * F * 2);  // by x_perm row
  L.dgu_off = o;    o = round256(o + size_t(L.prow_max) * 2 * F * 2);
  L.xt_off = o;     o = round256(o + size_t(D) * L.kmax * 2);
  L.dot_off = o;    o = round256(o + size_t(D) * L.kmax * 2);
  L.actt_off = o;   o = round256(o + size_t(F) * L.kmax * 2);
  L.dgut_off = o;   o = round256(o + size_t(2 * F) * L.kmax * 2);
  L.total = o;
  return L;
}

// float32 path: [d g | d u] (gate / up interleaved per 32 like the packed
// [Wg | Wu]) and the activation, per x_perm row
static size_t f32_bwd_bytes(int64_t R, int32_t F) {
  return 256 + round256(size_t(R) * 3 * F * 4);
}

bool ffn_backward_rows_ok(int64_t R, int32_t E, int32_t P) {
  // a DMA lane's byte offset reaches 16 blocks of kmax / 32 KB each
  return bwd_layout(R, E, P, 64, 64).kmax * 512 <= int64_t(INT32_MAX);
}

size_t ffn_backward_workspace_bytes(int64_t R, int32_t E, int32_t P, int32_t D, int32_t F,
                                    llep_dtype dtype) {
  if (dtype == LLEP_F32) return f32_bwd_bytes(R, F);
  return bwd_layout(R, E, P, D, F).total;
}

// One workgroup. For the groups [lo, hi) of the range: each group's first
// weight-gradient row (kbase[group], a multiple of 32) in gradient-return
// order, the owner group of every 32-row chunk, and the
// experts present with their segment (first 32-row slice, slices), longest
// segment first (ties: lower expert id), and how many of them have at least
// long_slices slices (those tiles are handed out before the input-gradient
// tiles, the shorter ones after them). Zeroes the work counters of the
// multi-problem launch and of the d act launch's copies.
__global__ __launch_bounds__(1024) void wgrad_table_kernel(
    const int32_t *__restrict__ groups, const int32_t *__restrict__ group_begin, int32_t device,
    int32_t P, int32_t E, int32_t M, int32_t *__restrict__ kbase,
    int32_t *__restrict__ chunk_group, int4 *__restrict__ wg_experts, int32_t *__restrict__ n_wg,
    int32_t long_slices, int32_t *__restrict__ n_wg_long, int32_t *__restrict__ kslices,
    int32_t *__restrict__ queue, int32_t *__restrict__ copy_counter) {
  __shared__ int32_t se[kMaxChunks], skey[kMaxChunks], ssl[kMaxChunks], skb[kMaxChunks];
  __shared__ int32_t esl[LLEP_MAX_EXPERTS];
  const int tid = threadIdx.x;
  const int lo = device < 0 ? group_begin[0] : group_begin[device];
  const int hi = device < 0 ? group_begin[P] : group_begin[device + 1];
  const int G = min(hi - lo, kMaxChunks);
  for (int i = tid; i < G; i += blockDim.x) {
    const int32_t *gr = groups + 4 * (lo + i);
    const int d = gr[0], e = gr[1], n = gr[3];
    se[i] = e;
    skey[i] = d == e / M ? -1 : d;  // native device first
    ssl[i] = (n + 31) / 32;
  }
  __syncthreads();
  // (the loops over groups and experts below are unrolled so that their
  // LDS reads, which do not depend on one another, are in flight together)
  for (int i = tid; i < G; i += blockDim.x) {
    int32_t kb = 0;
#pragma unroll 8
    for (int j = 0; j < G; ++j)
      if (se[j] < se[i] || (se[j] == se[i] && skey[j] < skey[i])) kb += ssl[j];
    kbase[lo + i] = kb * 32;
    skb[i] = kb;
  }
  for (int e = tid; e < E; e += blockDim.x) {
    int32_t sl = 0;
#pragma unroll 8
    for (int j = 0; j < G; ++j) sl += se[j] == e ? ssl[j] : 0;
    esl[e] = sl;
  }
  __syncthreads();
  // owner group of every 32-row slice: one wave per group, its lanes
  // striding over the group's slices
  for (int i = tid / kWave; i < G; i += blockDim.x / kWave)
    for (int c = skb[i] + tid % kWave; c < skb[i] + ssl[i]; c += kWave) chunk_group[c] = lo + i;
  for (int e = tid; e < E; e += blockDim.x) {
    const int32_t sl = esl[e];
    if (sl == 0) continue;
    int32_t idx = 0, start = 0;
#pragma unroll 8
    for (int f = 0; f < E; ++f) idx += esl[f] > sl || (esl[f] == sl && f < e);
#pragma unroll 8
    for (int j = 0; j < G; ++j) start += se[j] < e ? ssl[j] : 0;
    wg_experts[idx] = make_int4(e, start, sl, 0);
  }
  // counts over the experts and groups: one wave, lanes striding, then a
  // wave sum
  if (tid < kWave) {
    int32_t n = 0, nl = 0, tot = 0;
    for (int e = tid; e < E; e += kWave) {
      n += esl[e] > 0;
      nl += esl[e] > 0 && esl[e] >= long_slices;
    }
    for (int j = tid; j < G; j += kWave) tot += ssl[j];
    for (int off = kWave / 2; off > 0; off >>= 1) {
      n += __shfl_xor(n, off);
      nl += __shfl_xor(nl, off);
      tot += __shfl_xor(tot, off);
    }
    if (tid == 0) {
      *n_wg = n;
      *n_wg_long = nl;
      *kslices = tot;
      *queue = 0;
      *copy_counter = 0;
    }
  }
}

// The other weight-gradient operands: C columns of the range's rows
// (row-major by x_perm row, ld elements) copied into the weight-gradient
// layout, blocks of 16 columns x 32 rows over [C][kmax], row kbase[g] + r of
// the layout = row r of group g (zero for the padding r >= n_g). Item i of a
// source is its 32-row slice c = i / (C / 64) and its 64-column group
// i % (C / 64); the two sources (X, d out) follow one another.
struct WgradCopy {
  const uint16_t *src[2];
  uint16_t *dst[2];
  int64_t ld;
  int32_t C;  // a multiple of 64
  int64_t kmax;
  const int32_t *groups, *kbase, *chunk_group, *kslices;
  int32_t *counter;  // items taken; zeroed by the table kernel
};

constexpr int kCopyBatch = 8;             // items per counter claim
constexpr int kCopyTileBytes = 64 * 32 * 2;  // LDS staging tile of one wave

// One wavefront copies items taken kCopyBatch at a time from w.counter until
// none is left, with no barrier: each wave stages through its own LDS tile
// (`tile`, kCopyTileBytes) of 64 columns x 32 rows, column-major, the four
// 8-row chunks of column col in slots chunk ^ ((col / 8) % 4) so that a
// write instruction spreads over the banks. The loads of a batch are all
// issued before its first item is staged.
__device__ __forceinline__ void wgrad_copy_items(const WgradCopy &w, uint16_t *tile) {
  const int lane = threadIdx.x & 63;
  const int cgroups = w.C / 64;
  const int per_src = __builtin_amdgcn_readfirstlane(*w.kslices) * cgroups;
  const int n_items = 2 * per_src;
  // load layout: lane l holds row 8 q + l / 8 of the slice, columns
  // 8 (l % 8) .. + 7 of the item's 64 (each load instruction covers 8 whole
  // rows of 128 bytes)
  const int a = lane & 7, b = lane >> 3;
  const bool odd = b & 1;
  for (;;) {
    int b0 = 0;
    if (lane == 0) b0 = atomicAdd(w.counter, kCopyBatch);
    b0 = __builtin_amdgcn_readfirstlane(b0);
    if (b0 >= n_items) break;
    i32x4 v[kCopyBatch][4];
#pragma unroll
    for (int j = 0; j < kCopyBatch; ++j) {
      const int i = min(b0 + j, n_items - 1);  // past the end: the last item again (not stored)
      const int s = i >= per_src, rem = i - s * per_src;
      const int c = rem / cgroups, cc = rem - c * cgroups;
      const int gi = w.chunk_group[c];
      const int n = w.groups[4 * gi + 3];
      const int r0 = c * 32 - w.kbase[gi];
      const uint16_t *src = w.src[s] + int64_t(w.groups[4 * gi + 2]) * w.ld + cc * 64 + a * 8;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int row = r0 + 8 * q + b;
        v[j][q] = i32x4{0, 0, 0, 0};
        if (row < n) v[j][q] = *reinterpret_cast<const i32x4 *>(src + int64_t(row) * w.ld);
      }
    }
#pragma unroll
    for (int j = 0; j < kCopyBatch; ++j) {
      const int i = b0 + j;
      if (i >= n_items) break;
      const int s = i >= per_src, rem = i - s * per_src;
      const int c = rem / cgroups, cc = rem - c * cgroups;
      // the previous item's reads of the tile are done before it is rewritten
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      // Lanes l and l ^ 8 hold rows r and r ^ 1 of the same columns: each
      // writes one 32-bit word of two rows, the even-row lane for the even
      // column of a pair, the odd-row lane for the odd one.
#pragma unroll
      for (int q = 0; q < 4; ++q) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t mine = uint32_t(v[j][q][e]);
          const uint32_t other = uint32_t(__shfl_xor(int(mine), 8));
          const uint32_t word = odd ? ((other >> 16) | (mine & 0xffff0000u))
                                    : ((mine & 0xffffu) | (other << 16));
          const int col = 8 * a + 2 * e + int(odd);
          *reinterpret_cast<uint32_t *>(tile + col * 32 + ((q ^ (a & 3)) << 3) + (b & 6)) = word;
        }
      }
      // the tile is written before any lane reads it back
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      // block bb: columns 16 bb .. 16 bb + 15; lane l column l / 4, rows
      // 8 (l % 4) .. + 7
      uint16_t *dst = w.dst[s] + int64_t(c) * 512 + (lane >> 2) * 32 + (lane & 3) * 8;
#pragma unroll
      for (int bb = 0; bb < 4; ++bb) {
        const int col = bb * 16 + (lane >> 2);
        *reinterpret_cast<i32x4 *>(dst + int64_t(cc * 4 + bb) * (w.kmax / 32) * 512) =
            *reinterpret_cast<const i32x4 *>(tile + col * 32 + (((lane & 3) ^ ((col >> 3) & 3)) << 3));
      }
    }
  }
}

// Step 2 of the backward (d act GEMM with the SwiGLU backward epilogue) and
// the copies of X and d out into the weight-gradient layout in one launch:
// the GEMM deals its tiles in rounds, so the workgroups without a tile in the
// last, partly filled round start on the copies while the others finish
// their tiles, and everyone takes copy items once its tiles are done.
template <int BN, int WAVES_M, int WAVES_N>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N)
__attribute__((amdgpu_waves_per_eu(WAVES_M * WAVES_N / 4, WAVES_M * WAVES_N / 4)))
void dact_kernel(GemmArgs g, WgradCopy w) {
  static_assert(WAVES_M * WAVES_N * kCopyTileBytes <= ring_bytes<BN>(), "copy tiles fit the ring");
  __shared__ __attribute__((aligned(1024))) char smem[ring_bytes<BN>()];
  __shared__ int32_t s_next;
  {
    LaunchSched<256, BN, false> sched(g, &s_next);
    TileCoord t;
    if (sched.first(t)) gemm_tiles<BN, WAVES_M, WAVES_N, kEpiSwigluBwd, false, true>(g, smem, t, sched);
  }
  // every wave is done with the ring (its last epilogue's staging reads)
  // before the copies reuse it
  __syncthreads();
  wgrad_copy_items(w, reinterpret_cast<uint16_t *>(smem + (threadIdx.x >> 6) * kCopyTileBytes));
}

// Packed weights for the backward GEMMs, in the forward's block layout:
// [Wg | Wu] rows d with the gate/up columns interleaved per 32 (K = 2F), and
// Wd rows f (K = D).
template <typename T>
__global__ __launch_bounds__(256) void pack_bwd_kernel(const T *__restrict__ wg,
                                                       const T *__restrict__ wu,
                                                       const T *__restrict__ wd, T *__restrict__ gut,
                                                       T *__restrict__ dnt, int32_t E, int32_t D,
                                                       int32_t F) {
  const int64_t per = int64_t(D) * F, total = int64_t(E) * per;
  for (int64_t u = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; u < total;
       u += int64_t(gridDim.x) * blockDim.x) {
    const int64_t e = u / per, r = u % per;
    // Wg, Wu [E][D][F]: element (d, f)
    const int d = int(r / F), f = int(r % F);
    const int j = 64 * (f / 32) + (f % 32);
    gut[e * 2 * per + packed_index(d, j, 2 * F)] = wg[u];
    gut[e * 2 * per + packed_index(d, j + 32, 2 * F)] = wu[u];
    // Wd [E][F][D]: element (f2, d2) = row f2 of the (K = D) packing
    const int f2 = int(r / D), d2 = int(r % D);
    dnt[e * per + packed_index(f2, d2, D)] = wd[u];
  }
}

hipError_t launch_pack_backward(int32_t E, int32_t D, int32_t F, llep_dtype dtype, const void *w_gate,
                                const void *w_up, const void *w_down, void *gut, void *dnt,
                                hipStream_t stream) {
  if (dtype == LLEP_F32)
    hipLaunchKernelGGL(pack_bwd_kernel<float>, dim3(4096), dim3(256), 0, stream,
                       static_cast<const float *>(w_gate), static_cast<const float *>(w_up),
                       static_cast<const float *>(w_down), static_cast<float *>(gut),
                       static_cast<float *>(dnt), E, D, F);
  else
    hipLaunchKernelGGL(pack_bwd_kernel<uint16_t>, dim3(4096), dim3(256), 0, stream,
                       static_cast<const uint16_t *>(w_gate), static_cast<const uint16_t *>(w_up),
                       static_cast<const uint16_t *>(w_down), static_cast<uint16_t *>(gut),
                       static_cast<uint16_t *>(dnt), E, D, F);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// float32 backward: one thread per output element (small layers; reference
// precision, no matrix cores). Same operations and the same gradient-return
// order as the bf16 path, without the bf16 roundings of the intermediates.
// ---------------------------------------------------------------------------

// per (row, f) of the range: g, u (saved by the training forward, else
// recomputed), d act = d out . Wd[f], then
// d g, d u (into [row][2F], gate at 64 (f / 32) + f % 32, up 32 further) and
// act = silu(g) u (into [row][F])
__global__ __launch_bounds__(256) void ffn_f32_bwd_act_kernel(
    const float *__restrict__ x_perm, const float *__restrict__ d_out_perm,
    const float *__restrict__ gu_saved, const float *__restrict__ wgu,
    const float *__restrict__ wdt, float *__restrict__ dgu,
    float *__restrict__ act, const int32_t *__restrict__ groups,
    const int32_t *__restrict__ group_begin, int32_t device, int32_t P, int32_t D, int32_t F) {
  int lo, hi, row_first, rows;
  device_range(groups, group_begin, device, P, lo, hi, row_first, rows);
  const int64_t total = int64_t(rows) * F;
  for (int64_t u = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; u < total;
       u += int64_t(gridDim.x) * blockDim.x) {
    const int row = row_first + int(u / F), f = int(u % F);
    const int e = groups[4 * group_of_row(groups, lo, hi, row) + 1];
    const float *xr = x_perm + int64_t(row) * D;
    const float *dor = d_out_perm + int64_t(row) * D;
    const int pg = 64 * (f / 32) + (f % 32);
    const float *we = wgu + int64_t(e) * 2 * F * D;
    const float *wd = wdt + int64_t(e) * F * D;
    float gs = 0.0f, us = 0.0f, da = 0.0f;
    for (int d = 0; d < D; ++d) {
      if (!gu_saved) {
        gs = fmaf(xr[d], we[packed_index(pg, d, D)], gs);
        us = fmaf(xr[d], we[packed_index(pg + 32, d, D)], us);
      }
      da = fmaf(dor[d], wd[packed_index(f, d, D)], da);
    }
    if (gu_saved) {
      gs = gu_saved[int64_t(row) * 2 * F + pg];
      us = gu_saved[int64_t(row) * 2 * F + pg + 32];
    }
    const float sg = 1.0f / (1.0f + expf(-gs));
    dgu[int64_t(row) * 2 * F + pg] = da * us * (sg * (1.0f + gs * (1.0f - sg)));
    dgu[int64_t(row) * 2 * F + pg + 32] = da * gs * sg;
    act[int64_t(row) * F + f] = gs * sg * us;
  }
}

// per (row, d) of the range: dX = [d g | d u] . [Wg | Wu] row d
__global__ __launch_bounds__(256) void ffn_f32_bwd_dx_kernel(
    const float *__restrict__ dgu, const float *__restrict__ wgut, float *__restrict__ dx,
    const int32_t *__restrict__ groups, const int32_t *__restrict__ group_begin, int32_t device,
    int32_t P, int32_t D, int32_t F) {
  int lo, hi, row_first, rows;
  device_range(groups, group_begin, device, P, lo, hi, row_first, rows);
  const int64_t total = int64_t(rows) * D;
  for (int64_t u = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; u < total;
       u += int64_t(gridDim.x) * blockDim.x) {
    const int row = row_first + int(u / D), c = int(u % D);
    const int e = groups[4 * group_of_row(groups, lo, hi, row) + 1];
    const float *gr = dgu + int64_t(row) * 2 * F;
    const float *we = wgut + int64_t(e) * 2 * F * D;
    float s = 0.0f;
    for (int j = 0; j < 2 * F; ++j) s = fmaf(gr[j], we[packed_index(c, j, 2 * F)], s);
    dx[int64_t(row) * D + c] = s;
  }
}

// per (expert, m, n) of the three weight gradients: the sum over the
// expert's groups of the range in gradient-return order (the group on the
// expert's native device first, then the others by increasing device), rows
// in order. Which = 0: dWg[e][d][f] (X^T d g), 1: dWu, 2: dWd[e][f][d]
// (act^T d out). Experts without a group in the range are not written.
__global__ __launch_bounds__(256) void ffn_f32_bwd_wgrad_kernel(
    const float *__restrict__ x_perm, const float *__restrict__ d_out_perm,
    const float *__restrict__ dgu, const float *__restrict__ act, float *__restrict__ dwg,
    float *__restrict__ dwu, float *__restrict__ dwd, const int32_t *__restrict__ groups,
    const int32_t *__restrict__ group_begin, int32_t device, int32_t P, int32_t E, int32_t M,
    int32_t D, int32_t F) {
  const int lo = device < 0 ? group_begin[0] : group_begin[device];
  const int hi = device < 0 ? group_begin[P] : group_begin[device + 1];
  const int64_t per = int64_t(D) * F, total = 3 * int64_t(E) * per;
  for (int64_t u = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; u < total;
       u += int64_t(gridDim.x) * blockDim.x) {
    const int which = int(u / (int64_t(E) * per));
    const int64_t rem = u % (int64_t(E) * per);
    const int e = int(rem / per);
    const int64_t o = rem % per;
    // dWg, dWu: element (d, f); dWd: element (f, d)
    const int a = which < 2 ? int(o / F) : int(o / D);  // d, or f for dWd
    const int b = which < 2 ? int(o % F) : int(o % D);  // f, or d for dWd
    float s = 0.0f;
    bool any = false;
    for (int pass = 0; pass < 2; ++pass) {
      for (int gi = lo; gi < hi; ++gi) {
        const int32_t *gr = groups + 4 * gi;
        if (gr[1] != e || (gr[0] == e / M) != (pass == 0)) continue;
        any = true;
        for (int r = gr[2]; r < gr[2] + gr[3]; ++r) {
          if (which == 0)
            s = fmaf(x_perm[int64_t(r) * D + a], dgu[int64_t(r) * 2 * F + 64 * (b / 32) + b % 32], s);
          else if (which == 1)
            s = fmaf(x_perm[int64_t(r) * D + a],
                     dgu[int64_t(r) * 2 * F + 64 * (b / 32) + b % 32 + 32], s);
          else
            s = fmaf(act[int64_t(r) * F + a], d_out_perm[int64_t(r) * D + b], s);
        }
      }
    }
    if (!any) continue;
    float *dst = which == 0 ? dwg : which == 1 ? dwu : dwd;
    dst[int64_t(e) * per + o] = s;
  }
}

static hipError_t launch_grouped_ffn_backward_f32(const FfnBwdArgs &a, hipStream_t stream) {
  float *dgu = reinterpret_cast<float *>(static_cast<char *>(a.ws) + 256);
  float *act = dgu + size_t(a.R) * 2 * a.F;
  const int grid = 4096;
  hipLaunchKernelGGL(ffn_f32_bwd_act_kernel, dim3(grid), dim3(256), 0, stream,
                     static_cast<const float *>(a.x_perm), static_cast<const float *>(a.d_out_perm),
                     static_cast<const float *>(a.gate_up), static_cast<const float *>(a.w_gate_up),
                     static_cast<const float *>(a.w_down_t), dgu, act, a.groups, a.group_begin,
                     a.device, a.P, a.D, a.F);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(ffn_f32_bwd_dx_kernel, dim3(grid), dim3(256), 0, stream, dgu,
                     static_cast<const float *>(a.w_gate_up_t), static_cast<float *>(a.dx_perm),
                     a.groups, a.group_begin, a.device, a.P, a.D, a.F);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  hipLaunchKernelGGL(ffn_f32_bwd_wgrad_kernel, dim3(grid), dim3(256), 0, stream,
                     static_cast<const float *>(a.x_perm), static_cast<const float *>(a.d_out_perm),
                     dgu, act, a.dw_gate, a.dw_up, a.dw_down, a.groups, a.group_begin, a.device,
                     a.P, a.E, a.E / a.P, a.D, a.F);
  return hipGetLastError();
}

hipError_t launch_grouped_ffn_backward(const FfnBwdArgs &a, hipStream_t stream) {
  if (a.dtype == LLEP_F32) return launch_grouped_ffn_backward_f32(a, stream);
  const BwdLayout L = bwd_layout(a.R, a.E, a.P, a.D, a.F);
  char *ws = static_cast<char *>(a.ws);
  int32_t *n_mtiles = reinterpret_cast<int32_t *>(ws);
  int32_t *n_wg = n_mtiles + 1;
  int32_t *kslices = n_mtiles + 2;
  int32_t *queue = n_mtiles + 3;
  int32_t *n_wg_long = n_mtiles + 4;
  int32_t *copy_counter = n_mtiles + 5;
  int4 *tiles = reinterpret_cast<int4 *>(ws + L.tiles_off);
  int4 *wge = reinterpret_cast<int4 *>(ws + L.wge_off);
  int32_t *kbase = reinterpret_cast<int32_t *>(ws + L.kbase_off);
  int32_t *chunk = reinterpret_cast<int32_t *>(ws + L.chunk_off);
  uint16_t *gu = reinterpret_cast<uint16_t *>(ws + L.gu_off);
  uint16_t *dgu = reinterpret_cast<uint16_t *>(ws + L.dgu_off);
  uint16_t *xt = reinterpret_cast<uint16_t *>(ws + L.xt_off);
  uint16_t *dot = reinterpret_cast<uint16_t *>(ws + L.dot_off);
  uint16_t *actt = reinterpret_cast<uint16_t *>(ws + L.actt_off);
  uint16_t *dgut = reinterpret_cast<uint16_t *>(ws + L.dgut_off);
  const int grid = (cu_count() + 7) / 8 * 8;
  const int D = a.D, F = a.F;
  hipError_t err;
#define LLEP_CHECK_LAUNCH()            \
  do {                                 \
    err = hipGetLastError();           \
    if (err != hipSuccess) return err; \
  } while (0)
  err = launch_tile_table(a.groups, a.group_begin, 2 * a.E + a.P, a.device, a.P, tiles, n_mtiles,
                          stream);
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(wgrad_table_kernel, dim3(1), dim3(1024), 0, stream, a.groups, a.group_begin,
                     a.device, a.P, a.E, a.E / a.P, kbase, chunk, wge, n_wg, 2 * F / kSK,
                     n_wg_long, kslices, queue, copy_counter);
  LLEP_CHECK_LAUNCH();
  constexpr int NT = 64 * kWavesM * kWavesN;
  constexpr int NT192 = 64 * kWavesM192 * kWavesN192;
  const bool d192 = D % 256 != 0 && D % 192 == 0;
  const bool f192 = F % 256 != 0 && F % 192 == 0;
  // 1. g, u = X [Wg | Wu] (interleaved per 32), row-major by x_perm row,
  // unless the forward saved them
  GemmArgs g = {};
  g.A = static_cast<const uint16_t *>(a.x_perm);
  g.lda = D;
  g.B = static_cast<const uint16_t *>(a.w_gate_up);
  g.b_expert_stride = int64_t(2) * F * D;
  g.b_blk_stride = int64_t(D / kSK) * 1024;
  g.C = gu;
  g.ldc = 2 * F;
  g.groups = a.groups;
  g.tiles = tiles;
  g.n_mtiles = n_mtiles;
  g.N = 2 * F;
  g.Kdim = D;
  if (!a.gate_up) {
    hipLaunchKernelGGL((gemm256_kernel<256, kWavesM, kWavesN, kEpiPlain, false, false>),
                       dim3(grid), dim3(NT), 0, stream, g);
    LLEP_CHECK_LAUNCH();
  }
  // 2. d act = d out Wd^T; the epilogue writes [d g | d u] blocked (for dX)
  // and [d g | d u], act transposed into the weight-gradient layout; in the
  // same launch, the other weight-gradient operands X and d out, with the
  // rows of each expert laid end to end along k (gradient-return order)
  GemmArgs g2 = g;
  g2.A = static_cast<const uint16_t *>(a.d_out_perm);
  g2.lda = D;
  g2.B = static_cast<const uint16_t *>(a.w_down_t);
  g2.b_expert_stride = int64_t(F) * D;
  g2.b_blk_stride = int64_t(D / kSK) * 1024;
  g2.C = dgu;
  g2.ldc = F;
  g2.N = F;
  g2.Kdim = D;
  g2.GU = a.gate_up ? static_cast<const uint16_t *>(a.gate_up) : gu;
  g2.dgu_t = dgut;
  g2.act_t = actt;
  g2.kbase = kbase;
  g2.kmax = L.kmax;
  WgradCopy wc = {};
  wc.src[0] = static_cast<const uint16_t *>(a.x_perm);
  wc.src[1] = static_cast<const uint16_t *>(a.d_out_perm);
  wc.dst[0] = xt;
  wc.dst[1] = dot;
  wc.ld = D;
  wc.C = D;
  wc.kmax = L.kmax;
  wc.groups = a.groups;
  wc.kbase = kbase;
  wc.chunk_group = chunk;
  wc.kslices = kslices;
  wc.counter = copy_counter;
  if (f192)
    hipLaunchKernelGGL((dact_kernel<192, kWavesM192, kWavesN192>), dim3(grid), dim3(NT192), 0,
                       stream, g2, wc);
  else
    hipLaunchKernelGGL((dact_kernel<256, kWavesM, kWavesN>), dim3(grid), dim3(NT), 0, stream, g2,
                       wc);
  LLEP_CHECK_LAUNCH();
  // 3. one launch: dX = [d g | d u] [Wg | Wu]^T into the x_perm rows, and
  // the weight gradients X^T [d g | d u] (de-interleaved into dWg, dWu) and
  // act^T d out, per expert over its k-segment
  GemmArgs g3 = g;
  g3.A = dgu;
  g3.lda = 2 * F;
  g3.a_blk_stride = int64_t(2 * F / kSK) * 1024;
  g3.B = static_cast<const uint16_t *>(a.w_gate_up_t);
  g3.b_expert_stride = int64_t(2) * F * D;
  g3.b_blk_stride = int64_t(2 * F / kSK) * 1024;
  g3.C = static_cast<uint16_t *>(a.dx_perm);
  g3.ldc = D;
  g3.N = D;
  g3.Kdim = 2 * F;
  const int64_t wblk = (L.kmax / 32) * 1024;
  g3.wp[0] = WgProblem{xt, dgut, wblk, a.dw_gate, a.dw_up, int64_t(D) * F, D, 2 * F, 1};
  g3.wp[1] = WgProblem{actt, dot, wblk, a.dw_down, nullptr, int64_t(F) * D, F, D, 0};
  g3.wg_experts = wge;
  g3.n_wg = n_wg;
  g3.n_wg_long = n_wg_long;
  g3.queue = queue;
  // 256 x 192 tiles: the 256 x 256 ring fills the LDS and leaves no room for
  // the work counter's broadcast slot
  hipLaunchKernelGGL((gemm256_kernel<192, kWavesM192, kWavesN192, kEpiBwdMulti, true, false>),
                     dim3(grid), dim3(NT192), 0, stream, g3);
  LLEP_CHECK_LAUNCH();
#undef LLEP_CHECK_LAUNCH
  return hipSuccess;
}

}  // namespace llep
