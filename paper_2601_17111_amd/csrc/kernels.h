// Internal launch interface between the C ABI (abi.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "llep.h"

namespace llep {

constexpr int kMaxChunks = 2 * LLEP_MAX_EXPERTS + LLEP_MAX_DEVICES;

// Internal status bit: the plan tables overflowed (never expected; the chunk
// count is bounded by 2E + P).
constexpr int32_t kStatusPlanOverflow = 1 << 30;

// Pairs are counted in tiles of kRankTile pairs (one workgroup each), and
// per slice of kRankSub pairs (a wave's share of a tile); they are ranked
// slice by slice (one workgroup per slice, 64 pairs per wave). rank_base
// holds one row of E counts (then exclusive bases) per tile, a bad-id flag
// per tile, and a row of E counts per slice.
constexpr int kRankTile = 1024;
constexpr int kRankWaves = 4;
constexpr int kRankSub = kRankTile / kRankWaves;

int64_t rank_tiles(int64_t R);

struct PlanArgs {
  int64_t R;
  int32_t E, P, M, min_chunk, mode;
  int64_t cap;
  double lambda;
  int32_t n_tiles;
  const int32_t *ids;
  llep_plan_buffers buf;
};
hipError_t launch_plan(const PlanArgs &a, hipStream_t stream);

struct PermuteArgs {
  int64_t T, R;
  int32_t K, E, D;
  int32_t max_chunks;  // 2E + P: rows of the plan's chunk table
  int32_t n_tiles;
  int32_t elem_bytes;
  const int32_t *ids;
  const float *gates;
  const void *x;
  void *x_perm;
  float *gate_perm;
  int32_t *row_pair, *pair_row;
  llep_plan_buffers plan;
};
hipError_t launch_permute(const PermuteArgs &a, hipStream_t stream);

struct CombineArgs {
  int64_t T;
  int32_t K, D;
  llep_dtype dtype;
  const void *out_perm;
  const int32_t *pair_row;
  const float *gates;
  void *y;
};
hipError_t launch_combine(const CombineArgs &a, hipStream_t stream);

struct FfnArgs {
  int64_t R;
  int32_t P, E, D, F, device;
  llep_dtype dtype;
  const int32_t *groups, *group_begin;
  const void *x_perm, *w_gate_up, *w_down;
  void *out_perm;
  void *gate_up_out;  // training forward: raw gate / up values per x_perm row; null: none
  void *ws;
  size_t ws_bytes;
  int32_t *status;  // the plan's status word (LLEP_STATUS_FFN_WAIT)
};
size_t ffn_workspace_bytes(int64_t R, int32_t E, int32_t P, int32_t F,
                           llep_dtype dtype);
hipError_t launch_grouped_ffn(const FfnArgs &a, hipStream_t stream);
// Address on the current GPU of the library's LLEP_NOALLOC_SCRATCH_BYTES
// workspace array (looked up once per GPU, then cached).
hipError_t ffn_scratch_address(void **ptr);

struct FfnBwdArgs {
  int64_t R;
  int32_t P, E, D, F, device;
  llep_dtype dtype;
  const int32_t *groups, *group_begin;
  const void *x_perm, *d_out_perm, *w_gate_up, *w_gate_up_t, *w_down_t;
  const void *gate_up;  // saved by the training forward; null: recompute
  void *dx_perm;
  float *dw_gate, *dw_up, *dw_down;
  void *ws;
};
size_t ffn_backward_workspace_bytes(int64_t R, int32_t E, int32_t P, int32_t D, int32_t F,
                                    llep_dtype dtype);
// false when the weight-gradient operands of R rows are too long for the
// GEMM's 32-bit per-lane byte offsets
bool ffn_backward_rows_ok(int64_t R, int32_t E, int32_t P);
hipError_t launch_grouped_ffn_backward(const FfnBwdArgs &a, hipStream_t stream);
hipError_t launch_pack_backward(int32_t E, int32_t D, int32_t F, llep_dtype dtype, const void *w_gate,
                                const void *w_up, const void *w_down, void *gut, void *dnt,
                                hipStream_t stream);

struct CombineBwdArgs {
  int64_t T;
  int32_t K, D;
  llep_dtype dtype;
  const void *out_perm, *dy;
  const int32_t *pair_row;
  const float *gates;
  void *d_out_perm;
  float *d_gates;
};
hipError_t launch_combine_backward(const CombineBwdArgs &a, hipStream_t stream);

hipError_t launch_pack(int32_t E, int32_t D, int32_t F, llep_dtype dtype,
                       const void *w_gate, const void *w_up,
                       const void *w_down, void *gu, void *dn,
                       hipStream_t stream);

}  // namespace llep
