// C ABI of the LLEP hot path: argument checks on the host, then launches.
// No entry point allocates, synchronizes or keeps state between calls, apart
// from the calling thread's last error text and the per-GPU address of the
// library's workspace array (llep_grouped_ffn_noalloc), looked up once.
#include <stdint.h>
#include <string.h>

#include <string>

#include "kernels.h"
#include "llep.h"

namespace {

thread_local std::string g_last_error;

int fail(int code, const std::string &msg) {
  g_last_error = msg;
  return code;
}

int ok() {
  g_last_error.clear();
  return LLEP_OK;
}

int hip_result(hipError_t err, const char *where) {
  if (err == hipSuccess) return ok();
  return fail(LLEP_E_HIP, std::string(where) + ": " + hipGetErrorString(err));
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_params(const llep_plan_params *p) {
  if (!p) return fail(LLEP_E_ARG, "params is null");
  if (p->T < 0) return fail(LLEP_E_ARG, "T < 0");
  if (p->K < 1) return fail(LLEP_E_ARG, "K < 1");
  if (p->E < 1 || p->E > LLEP_MAX_EXPERTS) return fail(LLEP_E_ARG, "E outside [1, LLEP_MAX_EXPERTS]");
  if (p->P < 1 || p->P > LLEP_MAX_DEVICES) return fail(LLEP_E_ARG, "P outside [1, LLEP_MAX_DEVICES]");
  if (p->E % p->P != 0) return fail(LLEP_E_ARG, "E % P != 0");
  if (p->T > int64_t(INT32_MAX) / p->K) return fail(LLEP_E_ARG, "T * K >= 2^31");
  if (p->capacity < 1) return fail(LLEP_E_ARG, "capacity < 1");
  if (p->mode != LLEP_MODE_LLEP && p->mode != LLEP_MODE_EP) return fail(LLEP_E_ARG, "unknown mode");
  if (p->reserved != 0) return fail(LLEP_E_ARG, "reserved field is not 0");
  return LLEP_OK;
}

int check_plan_buffers(const llep_plan_buffers *b) {
  if (!b) return fail(LLEP_E_ARG, "plan buffers are null");
  if (!b->loads || !b->chunks || !b->chunk_row || !b->expert_chunk_begin || !b->groups ||
      !b->group_begin || !b->device_rows || !b->xfers || !b->rank_base || !b->info)
    return fail(LLEP_E_ARG, "a plan buffer pointer is null");
  return LLEP_OK;
}

int elem_bytes(llep_dtype d) { return d == LLEP_BF16 ? 2 : (d == LLEP_F32 ? 4 : 0); }

int check_rows(int32_t D, llep_dtype dtype) {
  const int eb = elem_bytes(dtype);
  if (eb == 0) return fail(LLEP_E_DTYPE, "unknown dtype");
  if (D < 1) return fail(LLEP_E_ARG, "D < 1");
  if (D % 8 != 0) return fail(LLEP_E_ARG, "D % 8 != 0 (rows must be whole 16-byte vectors)");
  return LLEP_OK;
}

int check_ffn_dims(int32_t D, int32_t F, llep_dtype dtype) {
  if (elem_bytes(dtype) == 0) return fail(LLEP_E_DTYPE, "unknown dtype");
  if (D < 64 || D % 64 != 0) return fail(LLEP_E_ARG, "D must be a positive multiple of 64");
  if (F < 64 || F % 64 != 0) return fail(LLEP_E_ARG, "F must be a positive multiple of 64");
  // the GEMMs address a tile's operand rows with 32-bit byte offsets
  if (D > LLEP_MAX_FFN_DIM || F > LLEP_MAX_FFN_DIM)
    return fail(LLEP_E_ARG, "D and F must be at most LLEP_MAX_FFN_DIM");
  return LLEP_OK;
}

}  // namespace

extern "C" {

const char *llep_last_error(void) { return g_last_error.c_str(); }

int32_t llep_plan_max_chunks(const llep_plan_params *params) {
  if (check_params(params) != LLEP_OK) return -1;
  return 2 * params->E + params->P;
}

int64_t llep_plan_rank_base_elems(const llep_plan_params *params) {
  if (check_params(params) != LLEP_OK) return -1;
  const int64_t tiles = llep::rank_tiles(params->T * params->K);
  // per tile: E counts (then bases), a bad-id flag, E counts per slice
  return tiles * params->E + tiles + tiles * llep::kRankWaves * params->E;
}

int llep_plan(const llep_plan_params *params, const int32_t *topk_ids,
              const llep_plan_buffers *out, hipStream_t stream) {
  int rc = check_params(params);
  if (rc != LLEP_OK) return rc;
  if ((rc = check_plan_buffers(out)) != LLEP_OK) return rc;
  const int64_t R = params->T * params->K;
  if (R > 0 && !topk_ids) return fail(LLEP_E_ARG, "topk_ids is null");
  llep::PlanArgs a;
  a.R = R;
  a.E = params->E;
  a.P = params->P;
  a.M = params->E / params->P;
  a.min_chunk = params->min_chunk < 1 ? 1 : params->min_chunk;
  a.mode = params->mode;
  a.cap = params->capacity;
  a.lambda = params->lambda;
  a.n_tiles = int32_t(llep::rank_tiles(R));
  a.ids = topk_ids;
  a.buf = *out;
  return hip_result(llep::launch_plan(a, stream), "llep_plan");
}

int llep_permute(const llep_plan_params *params, const llep_plan_buffers *plan,
                 const int32_t *topk_ids, const float *topk_gates, const void *x, int32_t D,
                 llep_dtype dtype, void *x_perm, float *gate_perm, int32_t *row_pair,
                 int32_t *pair_row, hipStream_t stream) {
  int rc = check_params(params);
  if (rc != LLEP_OK) return rc;
  if ((rc = check_plan_buffers(plan)) != LLEP_OK) return rc;
  if ((rc = check_rows(D, dtype)) != LLEP_OK) return rc;
  if (params->T > 0 &&
      (!topk_ids || !topk_gates || !x || !x_perm || !gate_perm || !row_pair || !pair_row))
    return fail(LLEP_E_ARG, "a data pointer is null");
  if (!aligned16(x) || !aligned16(x_perm)) return fail(LLEP_E_ARG, "x / x_perm not 16-byte aligned");
  llep::PermuteArgs a;
  a.T = params->T;
  a.R = params->T * params->K;
  a.K = params->K;
  a.E = params->E;
  a.max_chunks = 2 * params->E + params->P;
  a.D = D;
  a.n_tiles = int32_t(llep::rank_tiles(a.R));
  a.elem_bytes = elem_bytes(dtype);
  a.ids = topk_ids;
  a.gates = topk_gates;
  a.x = x;
  a.x_perm = x_perm;
  a.gate_perm = gate_perm;
  a.row_pair = row_pair;
  a.pair_row = pair_row;
  a.plan = *plan;
  return hip_result(llep::launch_permute(a, stream), "llep_permute");
}

size_t llep_packed_gate_up_bytes(int32_t E, int32_t D, int32_t F, llep_dtype dtype) {
  if (E < 1 || D < 1 || F < 1 || elem_bytes(dtype) == 0) return 0;
  return size_t(E) * 2 * size_t(F) * size_t(D) * elem_bytes(dtype);
}

size_t llep_packed_down_bytes(int32_t E, int32_t D, int32_t F, llep_dtype dtype) {
  if (E < 1 || D < 1 || F < 1 || elem_bytes(dtype) == 0) return 0;
  return size_t(E) * size_t(D) * size_t(F) * elem_bytes(dtype);
}

int llep_pack_weights(int32_t E, int32_t D, int32_t F, llep_dtype dtype, const void *w_gate,
                      const void *w_up, const void *w_down, void *w_gate_up_packed,
                      void *w_down_packed, hipStream_t stream) {
  if (E < 1 || E > LLEP_MAX_EXPERTS) return fail(LLEP_E_ARG, "E outside [1, LLEP_MAX_EXPERTS]");
  int rc = check_ffn_dims(D, F, dtype);
  if (rc != LLEP_OK) return rc;
  if (!w_gate || !w_up || !w_down || !w_gate_up_packed || !w_down_packed)
    return fail(LLEP_E_ARG, "a weight pointer is null");
  if (!aligned16(w_gate) || !aligned16(w_up) || !aligned16(w_down) ||
      !aligned16(w_gate_up_packed) || !aligned16(w_down_packed))
    return fail(LLEP_E_ARG, "weights not 16-byte aligned");
  return hip_result(llep::launch_pack(E, D, F, dtype, w_gate, w_up, w_down, w_gate_up_packed,
                                      w_down_packed, stream),
                    "llep_pack_weights");
}

size_t llep_grouped_ffn_workspace_bytes(const llep_plan_params *params, int32_t F,
                                        llep_dtype dtype) {
  if (check_params(params) != LLEP_OK || F < 1 || elem_bytes(dtype) == 0) return 0;
  return llep::ffn_workspace_bytes(params->T * params->K, params->E, params->P, F, dtype);
}

static int grouped_ffn(const llep_plan_params *params, const llep_plan_buffers *plan,
                       int32_t device, const void *x_perm, const void *w_gate_up_packed,
                       const void *w_down_packed, int32_t D, int32_t F, llep_dtype dtype,
                       void *out_perm, void *gate_up, void *workspace, size_t workspace_bytes,
                       hipStream_t stream, const char *name) {
  int rc = check_params(params);
  if (rc != LLEP_OK) return rc;
  if ((rc = check_plan_buffers(plan)) != LLEP_OK) return rc;
  if ((rc = check_ffn_dims(D, F, dtype)) != LLEP_OK) return rc;
  if (device < -1 || device >= params->P) return fail(LLEP_E_ARG, "device outside [-1, P)");
  if (!x_perm || !w_gate_up_packed || !w_down_packed || !out_perm)
    return fail(LLEP_E_ARG, "a data pointer is null");
  if (!aligned16(x_perm) || !aligned16(w_gate_up_packed) || !aligned16(w_down_packed) ||
      !aligned16(out_perm))
    return fail(LLEP_E_ARG, "data not 16-byte aligned");
  const size_t need = llep::ffn_workspace_bytes(params->T * params->K, params->E, params->P, F, dtype);
  if (!workspace || workspace_bytes < need)
    return fail(LLEP_E_WORKSPACE, "workspace missing or smaller than llep_grouped_ffn_workspace_bytes");
  if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
    return fail(LLEP_E_WORKSPACE, "workspace not 256-byte aligned");
  llep::FfnArgs a = {};
  a.R = params->T * params->K;
  a.P = params->P;
  a.E = params->E;
  a.D = D;
  a.F = F;
  a.device = device;
  a.dtype = dtype;
  a.groups = plan->groups;
  a.group_begin = plan->group_begin;
  a.x_perm = x_perm;
  a.w_gate_up = w_gate_up_packed;
  a.w_down = w_down_packed;
  a.out_perm = out_perm;
  a.gate_up_out = gate_up;
  a.ws = workspace;
  a.ws_bytes = workspace_bytes;
  a.status = &plan->info->status;
  return hip_result(llep::launch_grouped_ffn(a, stream), name);
}

int llep_grouped_ffn(const llep_plan_params *params, const llep_plan_buffers *plan,
                     int32_t device, const void *x_perm, const void *w_gate_up_packed,
                     const void *w_down_packed, int32_t D, int32_t F, llep_dtype dtype,
                     void *out_perm, void *workspace, size_t workspace_bytes,
                     hipStream_t stream) {
  return grouped_ffn(params, plan, device, x_perm, w_gate_up_packed, w_down_packed, D, F, dtype,
                     out_perm, nullptr, workspace, workspace_bytes, stream, "llep_grouped_ffn");
}

int llep_grouped_ffn_train(const llep_plan_params *params, const llep_plan_buffers *plan,
                           int32_t device, const void *x_perm, const void *w_gate_up_packed,
                           const void *w_down_packed, int32_t D, int32_t F, llep_dtype dtype,
                           void *out_perm, void *gate_up, void *workspace,
                           size_t workspace_bytes, hipStream_t stream) {
  if (!gate_up) return fail(LLEP_E_ARG, "gate_up is null");
  if (!aligned16(gate_up)) return fail(LLEP_E_ARG, "gate_up not 16-byte aligned");
  return grouped_ffn(params, plan, device, x_perm, w_gate_up_packed, w_down_packed, D, F, dtype,
                     out_perm, gate_up, workspace, workspace_bytes, stream,
                     "llep_grouped_ffn_train");
}

int llep_grouped_ffn_noalloc(const llep_plan_params *params, const llep_plan_buffers *plan,
                             int32_t device, const void *x_perm, const void *w_gate_up_packed,
                             const void *w_down_packed, int32_t D, int32_t F, llep_dtype dtype,
                             void *out_perm, hipStream_t stream) {
  int rc = check_params(params);
  if (rc != LLEP_OK) return rc;
  if (F < 1 || elem_bytes(dtype) == 0) return check_ffn_dims(D, F, dtype);
  const size_t need = llep::ffn_workspace_bytes(params->T * params->K, params->E, params->P, F, dtype);
  if (need > size_t(LLEP_NOALLOC_SCRATCH_BYTES))
    return fail(LLEP_E_WORKSPACE,
                "llep_grouped_ffn_noalloc: this layer needs " + std::to_string(need) +
                    " bytes of workspace, more than the library's LLEP_NOALLOC_SCRATCH_BYTES = " +
                    std::to_string(size_t(LLEP_NOALLOC_SCRATCH_BYTES)) +
                    "; use llep_grouped_ffn with a caller workspace");
  void *ws = nullptr;
  const hipError_t err = llep::ffn_scratch_address(&ws);
  if (err != hipSuccess) return hip_result(err, "llep_grouped_ffn_noalloc (scratch address)");
  return grouped_ffn(params, plan, device, x_perm, w_gate_up_packed, w_down_packed, D, F, dtype,
                     out_perm, nullptr, ws, size_t(LLEP_NOALLOC_SCRATCH_BYTES), stream,
                     "llep_grouped_ffn_noalloc");
}

int llep_combine(const llep_plan_params *params, const void *out_perm, const int32_t *pair_row,
                 const float *topk_gates, int32_t D, llep_dtype dtype, void *y,
                 hipStream_t stream) {
  int rc = check_params(params);
  if (rc != LLEP_OK) return rc;
  if ((rc = check_rows(D, dtype)) != LLEP_OK) return rc;
  // topk_gates == nullptr: every gate is 1 (sums the pairs' input gradients)
  if (params->T > 0 && (!out_perm || !pair_row || !y))
    return fail(LLEP_E_ARG, "a data pointer is null");
  if (!aligned16(out_perm) || !aligned16(y)) return fail(LLEP_E_ARG, "out_perm / y not 16-byte aligned");
  llep::CombineArgs a;
  a.T = params->T;
  a.K = params->K;
  a.D = D;
  a.dtype = dtype;
  a.out_perm = out_perm;
  a.pair_row = pair_row;
  a.gates = topk_gates;
  a.y = y;
  return hip_result(llep::launch_combine(a, stream), "llep_combine");
}

int llep_combine_backward(const llep_plan_params *params, const void *out_perm,
                          const int32_t *pair_row, const float *topk_gates, const void *dy,
                          int32_t D, llep_dtype dtype, void *d_out_perm, float *d_gates,
                          hipStream_t stream) {
  int rc = check_params(params);
  if (rc != LLEP_OK) return rc;
  if ((rc = check_rows(D, dtype)) != LLEP_OK) return rc;
  if (params->T > 0 && (!out_perm || !pair_row || !topk_gates || !dy || !d_out_perm || !d_gates))
    return fail(LLEP_E_ARG, "a data pointer is null");
  if (!aligned16(out_perm) || !aligned16(dy) || !aligned16(d_out_perm))
    return fail(LLEP_E_ARG, "out_perm / dy / d_out_perm not 16-byte aligned");
  llep::CombineBwdArgs a;
  a.T = params->T;
  a.K = params->K;
  a.D = D;
  a.dtype = dtype;
  a.out_perm = out_perm;
  a.dy = dy;
  a.pair_row = pair_row;
  a.gates = topk_gates;
  a.d_out_perm = d_out_perm;
  a.d_gates = d_gates;
  return hip_result(llep::launch_combine_backward(a, stream), "llep_combine_backward");
}

int llep_pack_weights_backward(int32_t E, int32_t D, int32_t F, llep_dtype dtype,
                               const void *w_gate, const void *w_up, const void *w_down,
                               void *w_gate_up_t_packed, void *w_down_t_packed,
                               hipStream_t stream) {
  if (E < 1 || E > LLEP_MAX_EXPERTS) return fail(LLEP_E_ARG, "E outside [1, LLEP_MAX_EXPERTS]");
  int rc = check_ffn_dims(D, F, dtype);
  if (rc != LLEP_OK) return rc;
  if (!w_gate || !w_up || !w_down || !w_gate_up_t_packed || !w_down_t_packed)
    return fail(LLEP_E_ARG, "a weight pointer is null");
  if (!aligned16(w_gate_up_t_packed) || !aligned16(w_down_t_packed))
    return fail(LLEP_E_ARG, "packed weights not 16-byte aligned");
  return hip_result(llep::launch_pack_backward(E, D, F, dtype, w_gate, w_up, w_down,
                                               w_gate_up_t_packed, w_down_t_packed, stream),
                    "llep_pack_weights_backward");
}

size_t llep_grouped_ffn_backward_workspace_bytes(const llep_plan_params *params, int32_t D,
                                                 int32_t F, llep_dtype dtype) {
  if (check_params(params) != LLEP_OK || D < 1 || F < 1 || elem_bytes(dtype) == 0) return 0;
  return llep::ffn_backward_workspace_bytes(params->T * params->K, params->E, params->P, D, F,
                                            dtype);
}

int llep_grouped_ffn_backward(const llep_plan_params *params, const llep_plan_buffers *plan,
                              int32_t device, const void *x_perm, const void *d_out_perm,
                              const void *w_gate_up_packed, const void *w_gate_up_t_packed,
                              const void *w_down_t_packed, const void *gate_up, int32_t D,
                              int32_t F, llep_dtype dtype, void *dx_perm, float *dw_gate,
                              float *dw_up, float *dw_down, void *workspace,
                              size_t workspace_bytes, hipStream_t stream) {
  int rc = check_params(params);
  if (rc != LLEP_OK) return rc;
  if ((rc = check_plan_buffers(plan)) != LLEP_OK) return rc;
  if ((rc = check_ffn_dims(D, F, dtype)) != LLEP_OK) return rc;
  if (device < -1 || device >= params->P) return fail(LLEP_E_ARG, "device outside [-1, P)");
  if (!x_perm || !d_out_perm || !w_gate_up_packed || !w_gate_up_t_packed || !w_down_t_packed ||
      !dx_perm || !dw_gate || !dw_up || !dw_down)
    return fail(LLEP_E_ARG, "a data pointer is null");
  if (!aligned16(x_perm) || !aligned16(d_out_perm) || !aligned16(w_gate_up_packed) ||
      !aligned16(w_gate_up_t_packed) || !aligned16(w_down_t_packed) || !aligned16(dx_perm) ||
      !aligned16(dw_gate) || !aligned16(dw_up) || !aligned16(dw_down) || !aligned16(gate_up))
    return fail(LLEP_E_ARG, "data not 16-byte aligned");
  if (!llep::ffn_backward_rows_ok(params->T * params->K, params->E, params->P))
    return fail(LLEP_E_ARG, "T * K too large for the backward (about 4 M pairs at most)");
  const size_t need =
      llep::ffn_backward_workspace_bytes(params->T * params->K, params->E, params->P, D, F, dtype);
  if (!workspace || workspace_bytes < need)
    return fail(LLEP_E_WORKSPACE,
                "workspace missing or smaller than llep_grouped_ffn_backward_workspace_bytes");
  if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
    return fail(LLEP_E_WORKSPACE, "workspace not 256-byte aligned");
  llep::FfnBwdArgs a = {};
  a.R = params->T * params->K;
  a.P = params->P;
  a.E = params->E;
  a.D = D;
  a.F = F;
  a.device = device;
  a.dtype = dtype;
  a.groups = plan->groups;
  a.group_begin = plan->group_begin;
  a.x_perm = x_perm;
  a.d_out_perm = d_out_perm;
  a.w_gate_up = w_gate_up_packed;
  a.w_gate_up_t = w_gate_up_t_packed;
  a.w_down_t = w_down_t_packed;
  a.gate_up = gate_up;
  a.dx_perm = dx_perm;
  a.dw_gate = dw_gate;
  a.dw_up = dw_up;
  a.dw_down = dw_down;
  a.ws = workspace;
  return hip_result(llep::launch_grouped_ffn_backward(a, stream), "llep_grouped_ffn_backward");
}

}  // extern "C"
