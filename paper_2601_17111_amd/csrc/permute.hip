// Step 3 of the LLEP hot path: permute token-expert pairs into their rows.
//
// Order (Sec. 2.1 re-indexing; Alg. 4 sorting, gathering, chunk building):
// pair p of expert e has rank r = number of earlier pairs of e. It lies in the
// chunk (d, e, s, t) of the plan with s <= r < t, and goes to row
// chunk_row + (r - s).
//
// rank_kernel    one workgroup per slice of kRankSub pairs (a quarter of a
//                histogram tile). The slice's base rank per expert is its
//                tile's base (the plan's scan of the histogram) plus the
//                histogram's counts of the tile's earlier slices; inside the
//                slice each wave owns 64 consecutive pairs and ranks them
//                with ballot-built match masks, so the order never depends
//                on atomics. The chunk table is copied to LDS first, so
//                finding a pair's chunk reads no memory. Writes pair_row,
//                row_pair and gate_perm.
// gather_kernel  one wavefront per 1 KB piece of a token's row (64 16-byte
//                vectors): reads it once and writes it to the K rows of the
//                token's pairs.
#include "common.h"
#include "kernels.h"

namespace llep {

__global__ __launch_bounds__(256) void rank_kernel(
    const int32_t *__restrict__ ids, const float *__restrict__ gates, int64_t R,
    int32_t E, int32_t max_chunks, int32_t n_tiles, const int32_t *__restrict__ rank_base,
    const int32_t *__restrict__ chunks, const int32_t *__restrict__ chunk_row,
    const int32_t *__restrict__ expert_chunk_begin, int32_t *__restrict__ pair_row,
    int32_t *__restrict__ row_pair, float *__restrict__ gate_perm) {
  // LDS: per-wave bases [kRankWaves][E], then the plan's chunk table
  // (expert_chunk_begin [E+1]; start, end, first row per chunk)
  extern __shared__ int32_t smem[];
  int32_t *wbase = smem;
  int32_t *ecb = wbase + kRankWaves * E;
  int32_t *c_start = ecb + (E + 1);
  int32_t *c_end = c_start + kMaxChunks;
  int32_t *c_row = c_end + kMaxChunks;
  const int tid = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int nb = bits_for(uint32_t(E));
  // slice blockIdx.x = slice `sub` of rank tile `tile`; wave w ranks its 64
  // consecutive pairs
  const int64_t tile = blockIdx.x / kRankWaves;
  const int sub = int(blockIdx.x % kRankWaves);
  const int64_t p = int64_t(blockIdx.x) * kRankSub + w * kWave + lane_id();
  static_assert(kRankSub == kRankWaves * kWave, "a slice is one 64-pair block per wave");
  // Every global load is issued up front, before any is waited for: the
  // pair's id and gate, the slice's base counts (all of the tile's earlier
  // slices' counts, summed afterwards for the ones before this slice), the
  // chunk count and the chunk table (read up to the table's capacity, so no
  // load waits for the count). Indices past the valid range are clamped
  // into it and their values dropped.
  constexpr int kThreads = kRankWaves * kWave;
  const int64_t pc = p < R ? p : R - 1;
  const int32_t id_raw = ids[pc];
  const float gate_raw = gates[pc];
  constexpr int kBaseIter = (LLEP_MAX_EXPERTS + kThreads - 1) / kThreads;
  const int32_t *slice_cnt = rank_base + int64_t(n_tiles) * (E + 1) + tile * kRankWaves * E;
  int32_t tb[kBaseIter], sc[kBaseIter][kRankWaves - 1];
#pragma unroll
  for (int i = 0; i < kBaseIter; ++i) {
    const int ec = min(tid + kThreads * i, E - 1);
    tb[i] = rank_base[tile * E + ec];
#pragma unroll
    for (int v = 0; v < kRankWaves - 1; ++v) sc[i][v] = slice_cnt[v * E + ec];
  }
  const int ncap = min(max_chunks, kMaxChunks);
  const int32_t nc_raw = expert_chunk_begin[E];
  constexpr int kEcbIter = (LLEP_MAX_EXPERTS + 1 + kThreads - 1) / kThreads;
  int32_t ecbv[kEcbIter];
#pragma unroll
  for (int j = 0; j < kEcbIter; ++j) ecbv[j] = expert_chunk_begin[min(tid + kThreads * j, E)];
  constexpr int kChunkIter = (kMaxChunks + kThreads - 1) / kThreads;
  int32_t cs[kChunkIter], ce[kChunkIter], cr[kChunkIter];
#pragma unroll
  for (int k = 0; k < kChunkIter; ++k) {
    const int cc = min(tid + kThreads * k, ncap - 1);
    cs[k] = chunks[4 * cc + 2];
    ce[k] = chunks[4 * cc + 3];
    cr[k] = chunk_row[cc];
  }
  __builtin_amdgcn_sched_barrier(0);  // the loads above issue together
  uint32_t ev = uint32_t(E);  // sentinel: past the end or invalid
  float gv = 0.0f;
  if (p < R) {
    gv = gate_raw;
    if (id_raw >= 0 && id_raw < E) ev = uint32_t(id_raw);
  }
  // base rank of each expert in this slice: the tile's base (the plan's
  // scan of the tile counts) plus the counts of the tile's earlier slices
  int32_t sb[kBaseIter];
#pragma unroll
  for (int i = 0; i < kBaseIter; ++i) {
    int32_t b = tb[i];
#pragma unroll
    for (int v = 0; v < kRankWaves - 1; ++v) b += v < sub ? sc[i][v] : 0;
    sb[i] = tid + kThreads * i < E ? b : 0;
  }
  const int nc = min(max(nc_raw, 0), ncap);
  for (int i = tid; i < kRankWaves * E; i += kThreads) wbase[i] = 0;
#pragma unroll
  for (int j = 0; j < kEcbIter; ++j) {
    const int i = tid + kThreads * j;
    if (i <= E) ecb[i] = min(max(ecbv[j], 0), nc);
  }
#pragma unroll
  for (int k = 0; k < kChunkIter; ++k) {
    const int c = tid + kThreads * k;
    if (c < nc) {
      c_start[c] = cs[k];
      c_end[c] = ce[k];
      c_row[c] = cr[k];
    }
  }
  __syncthreads();
  // per-wave counts of each expert (one leader lane per expert value)
  const uint64_t m = match_any(ev, nb);
  if (ev < uint32_t(E) && (m & lanemask_lt()) == 0) wbase[w * E + ev] = __popcll(m);
  __syncthreads();
  // wave bases = slice base + counts of the slice's earlier waves
#pragma unroll
  for (int i = 0; i < kBaseIter; ++i) {
    const int e = tid + kThreads * i;
    if (e >= E) continue;
    int32_t run = sb[i];
    for (int v = 0; v < kRankWaves; ++v) {
      const int32_t c = wbase[v * E + e];
      wbase[v * E + e] = run;
      run += c;
    }
  }
  __syncthreads();
  // rank, locate the chunk, write the row
  if (ev < uint32_t(E)) {
    const int32_t r = wbase[w * E + ev] + __popcll(m & lanemask_lt());
    int c = ecb[ev];
    const int c1 = max(ecb[ev + 1], c);
    while (c + 1 < c1 && r >= c_end[c]) ++c;
    // a pair outside every chunk of its expert (a plan built from other
    // ids) gets no row
    const bool inside = c < c1 && r >= c_start[c] && r < c_end[c];
    const int32_t row = inside ? c_row[c] + (r - c_start[c]) : -1;
    pair_row[p] = row;
    if (row >= 0 && row < R) {
      row_pair[row] = int32_t(p);
      gate_perm[row] = gv;
    }
  } else if (p < R) {
    pair_row[p] = -1;
  }
}

// Access choices, measured on MI355X with the gpt-oss-120b, deepseek-v3 and
// qwen3-30b layer shapes inside the full step: non-temporal loads of
// out_perm raise the combine from 0.62-0.65 to 0.73-0.79 of HBM peak;
// non-temporal loads in the gather gain nothing and non-temporal stores of
// x_perm lose 10-15%; a persistent gather that requests the next token's row
// before storing the current one measured no faster, and one wave per
// destination row (sequential writes, each token read K times) was 15-40%
// slower (the gather moves its bytes at 5.9 TB/s, four fifths of them
// writes; a plain fill reaches 6.8). One vector per lane (a wave per 1 KB
// piece of a row, so each wave issues K stores) beats a wave per whole row
// (6 vectors per lane, 6 K stores): 2-6% on the gpt-oss shapes, 5% on
// deepseek-v3, 0.5% on qwen3; 2 or 3 vectors per lane fall in between.
// Workgroups of 2 waves (grid capped at 65536, so on the larger shapes a
// wave takes a second piece) beat 4 waves by 1.3-3.4%; 8 waves, 1 wave,
// an uncapped grid and caps of 16384 or 32768 were slower or mixed.
// Four pairs' rows of at most 4 vectors per lane are in flight per combine
// step (1 or 2 pairs measured within 2%; 1 or 2 vectors per lane, a wave
// per 1 or 2 KB of the output row, within 1%: the combine's stream is
// mostly reads).
constexpr bool kGatherNtLoad = false;
constexpr bool kGatherNtStore = false;
constexpr bool kCombineNtLoad = true;
constexpr bool kCombineNtStore = false;
constexpr int kCombinePairs = 4;
constexpr int kCombineMaxVecs = 4;
// Combine backward: non-temporal loads of out_perm and up to 6 vectors per
// lane (one pass over a 2880-wide bf16 row) measured 359 -> 313 us on the
// gpt-oss-120b layer (0.59 -> 0.68 of HBM peak).
constexpr bool kCombineBwdNtLoad = true;
constexpr int kCombineBwdMaxVecs = 6;

template <bool kNT>
__device__ __forceinline__ i32x4 stream_load(const i32x4 *p) {
  if (kNT) return __builtin_nontemporal_load(p);
  return *p;
}
template <bool kNT>
__device__ __forceinline__ void stream_store(i32x4 *p, const i32x4 &v) {
  if (kNT)
    __builtin_nontemporal_store(v, p);
  else
    *p = v;
}

// Vectors per lane per pass for a row of `vecs` 16-byte vectors: the fewest
// passes of at most max_per_lane vectors, split evenly (a row of 2880 bf16 =
// 360 vectors is one pass of 6 per lane, or two of 3).
inline int vecs_per_lane(int32_t vecs, int max_per_lane) {
  const int vpl = (vecs + kWave - 1) / kWave;
  const int passes = (vpl + max_per_lane - 1) / max_per_lane;
  return (vpl + passes - 1) / passes;
}

// One wavefront per (token, slice of kV * 64 vectors of its row; launched
// with kV = 1): the slice is loaded once (all kV vectors per lane in flight)
// and stored to the rows of the token's K pairs. Row indices come in as one vector load per 64 pairs and are read
// back with v_readlane, so the stores need no further memory round trip.
// Workgroups of kGatherWaves waves, at most kGatherGrid of them (each wave
// then takes a second item when there are more than kGatherGrid workgroups'
// worth of items).
constexpr int kGatherWaves = 2;
constexpr int kGatherGrid = 65536;

template <int kV>
__global__ __launch_bounds__(kGatherWaves * kWave) void gather_kernel(const i32x4 *__restrict__ x,
                                                     i32x4 *__restrict__ x_perm,
                                                     const int32_t *__restrict__ pair_row,
                                                     int64_t T, int32_t K, int32_t vecs,
                                                     int64_t R) {
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = lane_id();
  const int nslices = (vecs + kV * kWave - 1) / (kV * kWave);
  for (int64_t wid = int64_t(blockIdx.x) * kGatherWaves + w; wid < T * nslices;
       wid += int64_t(gridDim.x) * kGatherWaves) {
    const int64_t t = wid / nslices;
    const i32x4 *src = x + t * vecs;
    {
      const int v0 = int(wid % nslices) * kV * kWave;
      i32x4 val[kV];
#pragma unroll
      for (int b = 0; b < kV; ++b) {
        const int v = v0 + b * kWave + lane;
        if (v < vecs) val[b] = stream_load<kGatherNtLoad>(src + v);
      }
      for (int kb = 0; kb < K; kb += kWave) {
        const int nk = min(kWave, K - kb);
        const int32_t rv = lane < nk ? pair_row[t * K + kb + lane] : -1;
        for (int k = 0; k < nk; ++k) {
          const int32_t row = __builtin_amdgcn_readlane(rv, k);
          if (row < 0 || row >= R) continue;
          i32x4 *dst = x_perm + int64_t(row) * vecs;
#pragma unroll
          for (int b = 0; b < kV; ++b) {
            const int v = v0 + b * kWave + lane;
            if (v < vecs) stream_store<kGatherNtStore>(dst + v, val[b]);
          }
        }
      }
    }
  }
}

template <int kV>
void launch_gather_v(int grid, hipStream_t stream, const PermuteArgs &a, int32_t vecs) {
  hipLaunchKernelGGL(gather_kernel<kV>, dim3(grid), dim3(kGatherWaves * kWave), 0, stream,
                     static_cast<const i32x4 *>(a.x), static_cast<i32x4 *>(a.x_perm),
                     a.pair_row, a.T, a.K, vecs, a.R);
}

hipError_t launch_permute(const PermuteArgs &a, hipStream_t stream) {
  if (a.R == 0) return hipSuccess;
  const size_t lds = (size_t(kRankWaves + 1) * a.E + 1 + 3 * size_t(kMaxChunks)) * sizeof(int32_t);
  const int64_t slices = (a.R + kRankSub - 1) / kRankSub;
  hipLaunchKernelGGL(rank_kernel, dim3(slices), dim3(256), lds, stream, a.ids, a.gates,
                     a.R, a.E, a.max_chunks, a.n_tiles, a.plan.rank_base, a.plan.chunks,
                     a.plan.chunk_row, a.plan.expert_chunk_begin, a.pair_row, a.row_pair,
                     a.gate_perm);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const int32_t vecs = int32_t((int64_t(a.D) * a.elem_bytes) / 16);
  const int64_t blocks = (a.T * ((vecs + kWave - 1) / kWave) + kGatherWaves - 1) / kGatherWaves;
  const int grid = int(blocks < kGatherGrid ? blocks : kGatherGrid);
  launch_gather_v<1>(grid, stream, a, vecs);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Step 5: combine. y[t] = sum_k gates[t, k] * out_perm[pair_row[t*K + k]],
// k ascending, float32 accumulation, one rounding to the output type.
// ---------------------------------------------------------------------------

// One wavefront per (token, slice of kV * 64 vectors of the output row);
// the pairs' rows are read kCombinePairs at a time with all their loads in
// flight before they are summed (in k order, so the result does not depend
// on the slicing).
template <bool kBf16, int kV>
__global__ __launch_bounds__(256) void combine_kernel(const i32x4 *__restrict__ out_perm,
                                                      const int32_t *__restrict__ pair_row,
                                                      const float *__restrict__ gates,
                                                      i32x4 *__restrict__ y, int64_t T,
                                                      int32_t K, int32_t vecs) {
  const int64_t R = T * K;
  constexpr int kElems = kBf16 ? 8 : 4;
  constexpr int kPairs = kCombinePairs;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = lane_id();
  const int nslices = (vecs + kV * kWave - 1) / (kV * kWave);
  for (int64_t wid = int64_t(blockIdx.x) * 4 + w; wid < T * nslices;
       wid += int64_t(gridDim.x) * 4) {
    const int64_t t = wid / nslices;
    {
      const int v0 = int(wid % nslices) * kV * kWave;
      float acc[kV][kElems];
#pragma unroll
      for (int b = 0; b < kV; ++b)
#pragma unroll
        for (int i = 0; i < kElems; ++i) acc[b][i] = 0.0f;
      for (int kb = 0; kb < K; kb += kWave) {
        const int nk = min(kWave, K - kb);
        int32_t rv = lane < nk ? pair_row[t * K + kb + lane] : -1;
        if (rv >= R) rv = -1;
        const float gv = lane < nk ? (gates ? gates[t * K + kb + lane] : 1.0f) : 0.0f;
        for (int k0 = 0; k0 < nk; k0 += kPairs) {
          int32_t row[kPairs];
          float g[kPairs];
          i32x4 q[kPairs][kV];
#pragma unroll
          for (int j = 0; j < kPairs; ++j) {
            row[j] = k0 + j < nk ? __builtin_amdgcn_readlane(rv, k0 + j) : -1;
            g[j] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(gv), k0 + j < nk ? k0 + j : 0));
          }
#pragma unroll
          for (int j = 0; j < kPairs; ++j) {
            if (row[j] < 0) continue;
            const i32x4 *src = out_perm + int64_t(row[j]) * vecs;
#pragma unroll
            for (int b = 0; b < kV; ++b) {
              const int v = v0 + b * kWave + lane;
              if (v < vecs) q[j][b] = stream_load<kCombineNtLoad>(src + v);
            }
          }
#pragma unroll
          for (int j = 0; j < kPairs; ++j) {
            if (row[j] < 0) continue;
#pragma unroll
            for (int b = 0; b < kV; ++b) {
              const int v = v0 + b * kWave + lane;
              if (v >= vecs) continue;
              if (kBf16) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                  const uint32_t u = uint32_t(q[j][b][i]);
                  acc[b][2 * i] = fmaf(g[j], __uint_as_float(u << 16), acc[b][2 * i]);
                  acc[b][2 * i + 1] = fmaf(g[j], __uint_as_float(u & 0xffff0000u), acc[b][2 * i + 1]);
                }
              } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[b][i] = fmaf(g[j], __int_as_float(q[j][b][i]), acc[b][i]);
              }
            }
          }
        }
      }
      i32x4 *dst = y + t * vecs;
#pragma unroll
      for (int b = 0; b < kV; ++b) {
        const int v = v0 + b * kWave + lane;
        if (v < vecs) {
          i32x4 q;
          if (kBf16) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
              q[i] = int32_t(pack_bf16x2(acc[b][2 * i], acc[b][2 * i + 1]));
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) q[i] = __float_as_int(acc[b][i]);
          }
          stream_store<kCombineNtStore>(dst + v, q);
        }
      }
    }
  }
}

template <bool kBf16, int kV>
void launch_combine_v(int grid, hipStream_t stream, const CombineArgs &a, int32_t vecs) {
  hipLaunchKernelGGL((combine_kernel<kBf16, kV>), dim3(grid), dim3(256), 0, stream,
                     static_cast<const i32x4 *>(a.out_perm), a.pair_row, a.gates,
                     static_cast<i32x4 *>(a.y), a.T, a.K, vecs);
}

template <bool kBf16>
void launch_combine_t(hipStream_t stream, const CombineArgs &a, int32_t vecs) {
  const int kv = vecs_per_lane(vecs, kCombineMaxVecs);
  const int64_t blocks = (a.T * ((vecs + kv * kWave - 1) / (kv * kWave)) + 3) / 4;
  const int grid = int(blocks < 65536 ? blocks : 65536);
  switch (kv) {
    case 1: launch_combine_v<kBf16, 1>(grid, stream, a, vecs); break;
    case 2: launch_combine_v<kBf16, 2>(grid, stream, a, vecs); break;
    case 3: launch_combine_v<kBf16, 3>(grid, stream, a, vecs); break;
    default: launch_combine_v<kBf16, 4>(grid, stream, a, vecs); break;
  }
}

hipError_t launch_combine(const CombineArgs &a, hipStream_t stream) {
  if (a.T == 0) return hipSuccess;
  const int eb = a.dtype == LLEP_BF16 ? 2 : 4;
  const int32_t vecs = int32_t((int64_t(a.D) * eb) / 16);
  if (a.dtype == LLEP_BF16)
    launch_combine_t<true>(stream, a, vecs);
  else
    launch_combine_t<false>(stream, a, vecs);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Backward of the combine (Eq. 1). For every valid pair (t, k) with row
// r = pair_row[t*K + k]:
//   d_out_perm[r] = gates[t, k] * dy[t]              (one rounding to bf16)
//   d_gates[t, k] = sum_i dy[t, i] * out_perm[r, i]  (float32)
// and d_gates = 0 for pairs without a row. One wavefront per token; the
// token's dy slice is held in registers while the pairs' rows stream past.
// ---------------------------------------------------------------------------

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

template <bool kBf16, int kV>
__global__ __launch_bounds__(256) void combine_bwd_kernel(
    const i32x4 *__restrict__ out_perm, const int32_t *__restrict__ pair_row,
    const float *__restrict__ gates, const i32x4 *__restrict__ dy, i32x4 *__restrict__ d_out_perm,
    float *__restrict__ d_gates, int64_t T, int32_t K, int32_t vecs) {
  const int64_t R = T * K;
  constexpr int kPairs = kCombinePairs;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = lane_id();
  for (int64_t t = int64_t(blockIdx.x) * 4 + w; t < T; t += int64_t(gridDim.x) * 4) {
    for (int kb = 0; kb < K; kb += kWave) {
      const int nk = min(kWave, K - kb);
      int32_t rv = lane < nk ? pair_row[t * K + kb + lane] : -1;
      if (rv >= R) rv = -1;
      const float gv = lane < nk ? gates[t * K + kb + lane] : 0.0f;
      float dg = 0.0f;  // lane j: d gate of pair kb + j
      for (int v0 = 0; v0 < vecs; v0 += kV * kWave) {
        i32x4 dv[kV];
#pragma unroll
        for (int b = 0; b < kV; ++b) {
          const int v = v0 + b * kWave + lane;
          dv[b] = v < vecs ? dy[t * vecs + v] : i32x4{0, 0, 0, 0};
        }
        for (int k0 = 0; k0 < nk; k0 += kPairs) {
          int32_t row[kPairs];
          float g[kPairs];
          i32x4 q[kPairs][kV];
#pragma unroll
          for (int j = 0; j < kPairs; ++j) {
            row[j] = k0 + j < nk ? __builtin_amdgcn_readlane(rv, k0 + j) : -1;
            g[j] = __int_as_float(
                __builtin_amdgcn_readlane(__float_as_int(gv), k0 + j < nk ? k0 + j : 0));
          }
#pragma unroll
          for (int j = 0; j < kPairs; ++j) {
            if (row[j] < 0) continue;
#pragma unroll
            for (int b = 0; b < kV; ++b) {
              const int v = v0 + b * kWave + lane;
              q[j][b] = v < vecs ? stream_load<kCombineBwdNtLoad>(out_perm + int64_t(row[j]) * vecs + v)
                                 : i32x4{0, 0, 0, 0};
            }
          }
#pragma unroll
          for (int j = 0; j < kPairs; ++j) {
            if (row[j] < 0) continue;
            float part = 0.0f;
#pragma unroll
            for (int b = 0; b < kV; ++b) {
              const int v = v0 + b * kWave + lane;
              i32x4 o;
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                if (kBf16) {
                  const uint32_t du = uint32_t(dv[b][i]), qu = uint32_t(q[j][b][i]);
                  const float d0 = __uint_as_float(du << 16), d1 = __uint_as_float(du & 0xffff0000u);
                  part = fmaf(d0, __uint_as_float(qu << 16), part);
                  part = fmaf(d1, __uint_as_float(qu & 0xffff0000u), part);
                  o[i] = int32_t(pack_bf16x2(g[j] * d0, g[j] * d1));
                } else {
                  const float d0 = __int_as_float(dv[b][i]);
                  part = fmaf(d0, __int_as_float(q[j][b][i]), part);
                  o[i] = __float_as_int(g[j] * d0);
                }
              }
              if (v < vecs) d_out_perm[int64_t(row[j]) * vecs + v] = o;
            }
            const float s = wave_sum(part);
            if (lane == k0 + j) dg += s;
          }
        }
      }
      if (lane < nk) d_gates[t * K + kb + lane] = rv >= 0 ? dg : 0.0f;
    }
  }
}

template <bool kBf16, int kV>
void launch_combine_bwd_v(int grid, hipStream_t stream, const CombineBwdArgs &a, int32_t vecs) {
  hipLaunchKernelGGL((combine_bwd_kernel<kBf16, kV>), dim3(grid), dim3(256), 0, stream,
                     static_cast<const i32x4 *>(a.out_perm), a.pair_row, a.gates,
                     static_cast<const i32x4 *>(a.dy), static_cast<i32x4 *>(a.d_out_perm),
                     a.d_gates, a.T, a.K, vecs);
}

template <bool kBf16>
void launch_combine_bwd_t(int grid, hipStream_t stream, const CombineBwdArgs &a, int32_t vecs) {
  switch (vecs_per_lane(vecs, kCombineBwdMaxVecs)) {
    case 1: launch_combine_bwd_v<kBf16, 1>(grid, stream, a, vecs); break;
    case 2: launch_combine_bwd_v<kBf16, 2>(grid, stream, a, vecs); break;
    case 3: launch_combine_bwd_v<kBf16, 3>(grid, stream, a, vecs); break;
    case 4: launch_combine_bwd_v<kBf16, 4>(grid, stream, a, vecs); break;
    case 5: launch_combine_bwd_v<kBf16, 5>(grid, stream, a, vecs); break;
    default: launch_combine_bwd_v<kBf16, 6>(grid, stream, a, vecs); break;
  }
}

hipError_t launch_combine_backward(const CombineBwdArgs &a, hipStream_t stream) {
  if (a.T == 0) return hipSuccess;
  const bool bf16 = a.dtype == LLEP_BF16;
  const int32_t vecs = bf16 ? a.D / 8 : a.D / 4;  // 16-byte vectors per row
  const int64_t blocks = (a.T + 3) / 4;
  const int grid = int(blocks < 65536 ? blocks : 65536);
  if (bf16)
    launch_combine_bwd_t<true>(grid, stream, a, vecs);
  else
    launch_combine_bwd_t<false>(grid, stream, a, vecs);
  return hipGetLastError();
}

}  // namespace llep
