// Step 3 of the LLEP hot path: permute token-expert pairs into their rows.
//
// Order (Sec. 2.1 re-indexing; Alg. 4 sort / index_select / build chunks):
// pair p of expert e has rank r = number of earlier pairs of e. It lies in the
// chunk (d, e, s, t) of the plan with s <= r < t, and goes to row
// chunk_row + (r - s).
//
// rank_kernel    one workgroup per rank tile of kRankTile pairs. The tile's
//                base rank per expert comes from the plan's scan of the
//                histogram; inside the tile each wave owns a contiguous slice
//                and ranks its pairs with ballot-built match masks, so the
//                order never depends on atomics. The chunk table is copied
//                to LDS first, so finding a pair's chunk reads no memory.
//                Writes pair_row, row_pair and gate_perm.
// gather_kernel  one wavefront per token: reads x[t] once (16-byte vectors)
//                and writes it to the K rows of the token's pairs.
#include "common.h"
#include "kernels.h"

namespace llep {

__global__ __launch_bounds__(256) void rank_kernel(
    const int32_t *__restrict__ ids, const float *__restrict__ gates, int64_t R,
    int32_t E, int32_t max_chunks, const int32_t *__restrict__ rank_base,
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
  const int64_t tile0 = int64_t(blockIdx.x) * kRankTile;
  const int64_t s0 = tile0 + int64_t(w) * kRankSub;
  const int nc = min(max(expert_chunk_begin[E], 0), min(max_chunks, kMaxChunks));
  for (int i = tid; i < kRankWaves * E; i += blockDim.x) wbase[i] = 0;
  for (int i = tid; i <= E; i += blockDim.x) ecb[i] = min(max(expert_chunk_begin[i], 0), nc);
  for (int c = tid; c < nc; c += blockDim.x) {
    c_start[c] = chunks[4 * c + 2];
    c_end[c] = chunks[4 * c + 3];
    c_row[c] = chunk_row[c];
  }
  __syncthreads();

  // pass A: per-wave counts of each expert in the wave's slice
  for (int j = 0; j < kRankSub; j += kWave) {
    if (s0 + j >= R) break;
    const int64_t p = s0 + j + lane_id();
    uint32_t e = uint32_t(E);
    if (p < R) {
      const int32_t v = ids[p];
      if (v >= 0 && v < E) e = uint32_t(v);
    }
    const uint64_t m = match_any(e, nb);
    if (e < uint32_t(E) && (m & lanemask_lt()) == 0) wbase[w * E + e] += __popcll(m);
  }
  __syncthreads();
  // wave bases = tile base + counts of the earlier waves of the tile
  for (int e = tid; e < E; e += blockDim.x) {
    int32_t run = rank_base[int64_t(blockIdx.x) * E + e];
    for (int v = 0; v < kRankWaves; ++v) {
      const int32_t c = wbase[v * E + e];
      wbase[v * E + e] = run;
      run += c;
    }
  }
  __syncthreads();

  // pass B: rank, locate the chunk, write the row
  for (int j = 0; j < kRankSub; j += kWave) {
    if (s0 + j >= R) break;
    const int64_t p = s0 + j + lane_id();
    uint32_t e = uint32_t(E);
    if (p < R) {
      const int32_t v = ids[p];
      if (v >= 0 && v < E) e = uint32_t(v);
    }
    const uint64_t m = match_any(e, nb);
    int32_t r = 0;
    if (e < uint32_t(E)) r = wbase[w * E + e] + __popcll(m & lanemask_lt());
    __builtin_amdgcn_wave_barrier();
    if (e < uint32_t(E) && (m & lanemask_lt()) == 0) wbase[w * E + e] += __popcll(m);
    if (e < uint32_t(E)) {
      int c = ecb[e];
      const int c1 = max(ecb[e + 1], c);
      while (c + 1 < c1 && r >= c_end[c]) ++c;
      // a pair outside every chunk of its expert (a plan built from other
      // ids) gets no row
      const bool inside = c < c1 && r >= c_start[c] && r < c_end[c];
      const int32_t row = inside ? c_row[c] + (r - c_start[c]) : -1;
      pair_row[p] = row;
      if (row >= 0 && row < R) {
        row_pair[row] = int32_t(p);
        gate_perm[row] = gates[p];
      }
    } else if (p < R) {
      pair_row[p] = -1;
    }
  }
}

// One wavefront per token; each lane moves 16-byte vectors. kBatch vectors
// per lane are loaded before they are stored, to keep loads in flight.
constexpr int kBatch = 4;

__global__ __launch_bounds__(256) void gather_kernel(const i32x4 *__restrict__ x,
                                                     i32x4 *__restrict__ x_perm,
                                                     const int32_t *__restrict__ pair_row,
                                                     int64_t T, int32_t K, int32_t vecs,
                                                     int64_t R) {
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = lane_id();
  for (int64_t t = int64_t(blockIdx.x) * 4 + w; t < T; t += int64_t(gridDim.x) * 4) {
    const i32x4 *src = x + t * vecs;
    for (int v0 = 0; v0 < vecs; v0 += kBatch * kWave) {
      i32x4 val[kBatch];
#pragma unroll
      for (int b = 0; b < kBatch; ++b) {
        const int v = v0 + b * kWave + lane;
        if (v < vecs) val[b] = src[v];
      }
      for (int k = 0; k < K; ++k) {
        const int32_t row = pair_row[t * K + k];
        if (row < 0 || row >= R) continue;
        i32x4 *dst = x_perm + int64_t(row) * vecs;
#pragma unroll
        for (int b = 0; b < kBatch; ++b) {
          const int v = v0 + b * kWave + lane;
          if (v < vecs) dst[v] = val[b];
        }
      }
    }
  }
}

hipError_t launch_permute(const PermuteArgs &a, hipStream_t stream) {
  if (a.R == 0) return hipSuccess;
  const size_t lds = (size_t(kRankWaves + 1) * a.E + 1 + 3 * size_t(kMaxChunks)) * sizeof(int32_t);
  hipLaunchKernelGGL(rank_kernel, dim3(a.n_tiles), dim3(256), lds, stream, a.ids, a.gates,
                     a.R, a.E, a.max_chunks, a.plan.rank_base, a.plan.chunks, a.plan.chunk_row,
                     a.plan.expert_chunk_begin, a.pair_row, a.row_pair, a.gate_perm);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const int32_t vecs = int32_t((int64_t(a.D) * a.elem_bytes) / 16);
  const int64_t blocks = (a.T + 3) / 4;
  const int grid = int(blocks < 65536 ? blocks : 65536);
  hipLaunchKernelGGL(gather_kernel, dim3(grid), dim3(256), 0, stream,
                     static_cast<const i32x4 *>(a.x), static_cast<i32x4 *>(a.x_perm),
                     a.pair_row, a.T, a.K, vecs, a.R);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Step 5: combine. y[t] = sum_k gates[t, k] * out_perm[pair_row[t*K + k]],
// k ascending, float32 accumulation, one rounding to the output type.
// ---------------------------------------------------------------------------

template <bool kBf16>
__global__ __launch_bounds__(256) void combine_kernel(const i32x4 *__restrict__ out_perm,
                                                      const int32_t *__restrict__ pair_row,
                                                      const float *__restrict__ gates,
                                                      i32x4 *__restrict__ y, int64_t T,
                                                      int32_t K, int32_t vecs) {
  const int64_t R = T * K;
  constexpr int kElems = kBf16 ? 8 : 4;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = lane_id();
  for (int64_t t = int64_t(blockIdx.x) * 4 + w; t < T; t += int64_t(gridDim.x) * 4) {
    for (int v0 = 0; v0 < vecs; v0 += kBatch * kWave) {
      float acc[kBatch][kElems];
#pragma unroll
      for (int b = 0; b < kBatch; ++b)
#pragma unroll
        for (int i = 0; i < kElems; ++i) acc[b][i] = 0.0f;
      for (int k = 0; k < K; ++k) {
        const int32_t row = pair_row[t * K + k];
        if (row < 0 || row >= R) continue;
        const float g = gates[t * K + k];
        const i32x4 *src = out_perm + int64_t(row) * vecs;
#pragma unroll
        for (int b = 0; b < kBatch; ++b) {
          const int v = v0 + b * kWave + lane;
          if (v < vecs) {
            const i32x4 q = src[v];
            if (kBf16) {
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const uint32_t u = uint32_t(q[i]);
                acc[b][2 * i] = fmaf(g, __uint_as_float(u << 16), acc[b][2 * i]);
                acc[b][2 * i + 1] = fmaf(g, __uint_as_float(u & 0xffff0000u), acc[b][2 * i + 1]);
              }
            } else {
#pragma unroll
              for (int i = 0; i < 4; ++i) acc[b][i] = fmaf(g, __int_as_float(q[i]), acc[b][i]);
            }
          }
        }
      }
      i32x4 *dst = y + t * vecs;
#pragma unroll
      for (int b = 0; b < kBatch; ++b) {
        const int v = v0 + b * kWave + lane;
        if (v < vecs) {
          i32x4 q;
          if (kBf16) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
              q[i] = int32_t(uint32_t(f32_to_bf16(acc[b][2 * i])) |
                             (uint32_t(f32_to_bf16(acc[b][2 * i + 1])) << 16));
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) q[i] = __float_as_int(acc[b][i]);
          }
          dst[v] = q;
        }
      }
    }
  }
}

hipError_t launch_combine(const CombineArgs &a, hipStream_t stream) {
  if (a.T == 0) return hipSuccess;
  const int eb = a.dtype == LLEP_BF16 ? 2 : 4;
  const int32_t vecs = int32_t((int64_t(a.D) * eb) / 16);
  const int64_t blocks = (a.T + 3) / 4;
  const int grid = int(blocks < 65536 ? blocks : 65536);
  if (a.dtype == LLEP_BF16)
    hipLaunchKernelGGL(combine_kernel<true>, dim3(grid), dim3(256), 0, stream,
                       static_cast<const i32x4 *>(a.out_perm), a.pair_row, a.gates,
                       static_cast<i32x4 *>(a.y), a.T, a.K, vecs);
  else
    hipLaunchKernelGGL(combine_kernel<false>, dim3(grid), dim3(256), 0, stream,
                       static_cast<const i32x4 *>(a.out_perm), a.pair_row, a.gates,
                       static_cast<i32x4 *>(a.y), a.T, a.K, vecs);
  return hipGetLastError();
}

}  // namespace llep
