/*
 * llep.h -- C ABI of the LLEP expert-layer hot path on one MI355X (gfx950).
 *
 * Paper: "Least-Loaded Expert Parallelism: Load Balancing An Imbalanced
 * Mixture-of-Experts" (arXiv 2601.17111).
 *
 * The layer has T tokens, each routed to K experts (ids and gates, Eq. 1-2),
 * N = E experts spread over P devices, M = E / P experts per device (device
 * p is native to experts pM .. (p+1)M-1, Alg. 1). A token-expert pair is
 * p = t*K + k; there are R = T*K pairs. On one GPU the P devices are virtual:
 * a device is a contiguous range of rows and groups in the tables below.
 *
 * Four steps, one entry point each, all enqueued on the caller's stream:
 *   llep_plan         loads l, then the least-loaded plan (Alg. 2/3) or the
 *                     standard EP plan (Alg. 1), as device-resident tables
 *   llep_permute      gathers token rows into per-(device, expert, chunk)
 *                     order (Sec. 2.1 re-indexing; Alg. 4 sorting, gathering,
 *                     chunk building)
 *   llep_grouped_ffn  grouped SwiGLU expert GEMMs for one device's groups
 *                     (Alg. 4 grouped GEMMs over native and foreign experts;
 *                     three-matrix SwiGLU expert of Sec. 5.1);
 *                     llep_grouped_ffn_train also keeps g and u for the
 *                     backward
 *   llep_combine      gate-weighted sum of each token's K expert rows (Eq. 1;
 *                     Alg. 4 un-sorting, reshape, sum over K)
 *
 * and the backward of steps 4 and 5 (LLEP stays exact under training; the
 * weight gradients of spilled chunks return to the expert's native device,
 * Sec. 1 and Sec. 4): llep_combine_backward, llep_grouped_ffn_backward, and
 * llep_combine with null gates to sum the pairs' input gradients per token.
 *
 * Conventions for every entry point:
 *   - Every array argument is a DEVICE pointer, allocated and owned by the
 *     caller; the library never allocates, frees or keeps a pointer after the
 *     call returns. Token data pointers may be null when T == 0. Struct
 *     arguments themselves (llep_plan_params, llep_plan_buffers) are HOST
 *     memory, read during the call only.
 *   - Calls only enqueue work on `stream` and return; results are valid once
 *     the stream reaches that point. Nothing synchronizes with the host.
 *   - Return value: LLEP_OK, or a negative LLEP_E_* code when the host-side
 *     checks reject the arguments (nothing is enqueued then), or LLEP_E_HIP
 *     when a launch fails. llep_last_error() describes the last failure of
 *     the calling thread.
 *   - Row-major layouts; dense arrays, no padding between rows.
 *   - bf16 data is IEEE bfloat16 (16 bits); gates are float32.
 *   - Rows of x, x_perm, out_perm and y, and the weight arrays, must start on
 *     16-byte boundaries (base pointers 16-byte aligned, D % 8 == 0).
 *
 * Readings of the paper that bind these calls (the paper leaves them open):
 *   - capacity m_alpha (Alg. 2) is an integer count of pairs;
 *   - Alg. 2's decreasing sort of the loads breaks ties by lower expert id;
 *     Alg. 3 ranks devices by g_a + g_p ascending, then by index;
 *   - min_chunk < 1 is read as 1; Alg. 3 force-assigns to the least-loaded
 *     device other than the native one;
 *   - zero-load experts get no chunk; with P == 1 the plan is standard EP;
 *   - an expert's range [start, end) names its pairs in ascending p;
 *   - the lambda test of Alg. 4 bypasses LLA iff max(l) * E < lambda * sum(l)
 *     in IEEE double; lambda <= 0 disables it;
 *   - inside a device rows go by expert id, then chunk start; all chunks of
 *     one (device, expert) form one group;
 *   - SwiGLU: out = (silu(x Wg) * (x Wu)) Wd, no bias, no clamp; the gate is
 *     applied in the combine, not in the expert GEMMs.
 */
#ifndef LLEP_H
#define LLEP_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- return codes ------------------------------------------------------ */
#define LLEP_OK 0
#define LLEP_E_ARG (-1)       /* bad size, null pointer, misalignment */
#define LLEP_E_WORKSPACE (-2) /* workspace missing or too small */
#define LLEP_E_DTYPE (-3)     /* unsupported dtype for this call */
#define LLEP_E_HIP (-4)       /* a HIP launch failed */

/* ---- device-detected status bits (llep_plan_info.status) ---------------- */
#define LLEP_STATUS_BAD_EXPERT_ID 1 /* an id outside [0, E): pair ignored */
#define LLEP_STATUS_FFN_WAIT 2      /* set by the bf16 grouped FFN when a
                                       down-projection tile gave up waiting
                                       (about a second) for its activations;
                                       never expected, the call's outputs are
                                       then undefined */

/* ---- limits --------------------------------------------------------------- */
#define LLEP_MAX_EXPERTS 512
#define LLEP_MAX_DEVICES 64
#define LLEP_MAX_FFN_DIM 65536 /* largest D and F of the FFN entry points */

typedef enum { LLEP_F32 = 0, LLEP_BF16 = 1 } llep_dtype;
typedef enum { LLEP_MODE_LLEP = 0, LLEP_MODE_EP = 1 } llep_mode;

/* Problem statement of the plan (Alg. 2 inputs l, M, alpha, m; Alg. 4
 * lambda). Host memory, 48 bytes. */
typedef struct {
  int64_t T;         /* tokens, >= 0; T * K < 2^31 */
  int32_t K;         /* experts per token, >= 1 (ids may repeat in a token) */
  int32_t E;         /* experts, 1..LLEP_MAX_EXPERTS, E % P == 0 */
  int32_t P;         /* devices, 1..LLEP_MAX_DEVICES */
  int32_t min_chunk; /* m of Alg. 3; values < 1 are read as 1 */
  int64_t capacity;  /* m_alpha of Alg. 2 in pairs, >= 1 */
  double lambda;     /* Alg. 4 imbalance threshold; <= 0: never bypass */
  int32_t mode;      /* llep_mode: LLA plan, or standard EP plan */
  int32_t reserved;  /* must be 0 */
} llep_plan_params;

/* Summary written by llep_plan into device memory. */
typedef struct {
  int32_t status;     /* LLEP_STATUS_* bits */
  int32_t n_chunks;   /* valid rows of chunks / chunk_row */
  int32_t n_groups;   /* valid rows of groups */
  int32_t n_xfers;    /* valid rows of xfers */
  int32_t bypassed;   /* 1 when the lambda test chose the standard EP plan */
  int32_t forced;     /* force-assignments made by Alg. 3 */
  int32_t max_device; /* device with the most rows (lowest index on ties) */
  int32_t total_rows; /* sum of device_rows = number of valid pairs */
} llep_plan_info;

/* Device-resident plan tables (all DEVICE pointers, caller-allocated).
 * C = llep_plan_max_chunks(params) = 2E + P bounds the chunk, group and
 * transfer counts (at most one native and one final spilled chunk per
 * expert, plus at most one capacity-filling spill per device). */
typedef struct {
  int32_t *loads;              /* [E] pairs routed to each expert (l) */
  int32_t *chunks;             /* [C][4] device, expert, start, end; sorted by
                                  (expert, start): the assignment map A */
  int32_t *chunk_row;          /* [C] first destination row of each chunk */
  int32_t *expert_chunk_begin; /* [E+1] chunks of expert e are
                                  [begin[e], begin[e+1]) */
  int32_t *groups;             /* [C][4] device, expert, row_start, n;
                                  device-major, expert ascending */
  int32_t *group_begin;        /* [P+1] groups of device d are
                                  [group_begin[d], group_begin[d+1]) */
  int32_t *device_rows;        /* [P] rows (pairs) computed by each device */
  int32_t *xfers;              /* [C][3] expert, src, dst: the weight-transfer
                                  plan W, sorted by (expert, dst), unique */
  int32_t *rank_base;          /* [llep_plan_rank_base_elems(params)] scratch
                                  of the pair-rank scan; read by llep_permute */
  llep_plan_info *info;        /* [1] */
} llep_plan_buffers;

/* 2E + P. Returns -1 on invalid params. */
int32_t llep_plan_max_chunks(const llep_plan_params *params);
/* Elements of llep_plan_buffers.rank_base. Returns -1 on invalid params. */
int64_t llep_plan_rank_base_elems(const llep_plan_params *params);

/* Step 1+2. Counts l over topk_ids [T][K] (int32), then builds the plan:
 * mode LLEP: lambda test, then Alg. 2/3 under `capacity` and `min_chunk`;
 * mode EP:   one chunk [0, l_e) per non-empty expert on device e / M.
 * Writes every table of `out` (only the first n_* rows of each table are
 * meaningful). Ids outside [0, E) are ignored and set a status bit.
 * Errors: LLEP_E_ARG (params, null pointers). */
int llep_plan(const llep_plan_params *params, const int32_t *topk_ids,
              const llep_plan_buffers *out, hipStream_t stream);

/* Step 3. For every valid pair p of expert e with rank r among e's pairs
 * (in ascending p), inside chunk (d, e, s, t), s <= r < t:
 *   row = chunk_row + (r - s);  x_perm[row] = x[p / K];
 *   gate_perm[row] = topk_gates[p];  row_pair[row] = p;  pair_row[p] = row.
 * Invalid pairs get pair_row[p] = -1. `plan` must hold the tables of an
 * llep_plan call on the same params and topk_ids, enqueued earlier.
 * x [T][D], x_perm [T*K][D] in `dtype` (rows >= total_rows untouched);
 * gate_perm, row_pair [T*K]; pair_row [T*K].
 * Errors: LLEP_E_ARG (sizes, D % 8, alignment, nulls), LLEP_E_DTYPE. */
int llep_permute(const llep_plan_params *params, const llep_plan_buffers *plan,
                 const int32_t *topk_ids, const float *topk_gates,
                 const void *x, int32_t D, llep_dtype dtype, void *x_perm,
                 float *gate_perm, int32_t *row_pair, int32_t *pair_row,
                 hipStream_t stream);

/* Packed expert weights (untimed setup, once per set of weights).
 * Inputs, as in the paper (FFN(u) = u^T W):
 *   w_gate, w_up [E][D][F], w_down [E][F][D], in `dtype`.
 * Outputs, in `dtype`, per expert a matrix P[n][k] (n: output column of
 * the GEMM, k: contraction index, K its length) stored in blocks of 16 rows
 * x 32 k: element (n, k) at ((n/16) * (K/32) + k/32) * 512 + (n%16) * 32
 * + k%32 (so each 16-row, 32-deep piece is one contiguous run):
 *   w_gate_up_packed [E][2F*D]: K = D; P row 64j + c      = column 32j + c
 *                               of w_gate, P row 64j + 32 + c = column
 *                               32j + c of w_up (j < F/32, c < 32);
 *   w_down_packed    [E][D*F]:  K = F; P row d = column d of w_down.
 * Requires D % 64 == 0 and F % 64 == 0, both at most LLEP_MAX_FFN_DIM.
 * Errors: LLEP_E_ARG, LLEP_E_DTYPE. */
size_t llep_packed_gate_up_bytes(int32_t E, int32_t D, int32_t F,
                                 llep_dtype dtype);
size_t llep_packed_down_bytes(int32_t E, int32_t D, int32_t F,
                              llep_dtype dtype);
int llep_pack_weights(int32_t E, int32_t D, int32_t F, llep_dtype dtype,
                      const void *w_gate, const void *w_up,
                      const void *w_down, void *w_gate_up_packed,
                      void *w_down_packed, hipStream_t stream);

/* Step 4. For every group (device, e, row_start, n) of `device` (or of all
 * devices when device == -1), with X = x_perm[row_start : row_start + n]:
 *   act = silu(X Wg_e) * (X Wu_e)   (float accumulation; rounded to dtype)
 *   out_perm[row_start : row_start + n] = act Wd_e   (float accumulation)
 * The group range is read from plan->group_begin on the device: no host
 * synchronization. Weights are the llep_pack_weights outputs. bf16 uses
 * matrix cores (MFMA); f32 is a plain reference-precision path.
 * Requires D % 64 == 0, F % 64 == 0 (both at most LLEP_MAX_FFN_DIM);
 * workspace of at least
 * llep_grouped_ffn_workspace_bytes(params, F, dtype) bytes, 256-byte aligned.
 * Errors: LLEP_E_ARG, LLEP_E_DTYPE, LLEP_E_WORKSPACE. */
size_t llep_grouped_ffn_workspace_bytes(const llep_plan_params *params,
                                        int32_t F, llep_dtype dtype);
int llep_grouped_ffn(const llep_plan_params *params,
                     const llep_plan_buffers *plan, int32_t device,
                     const void *x_perm, const void *w_gate_up_packed,
                     const void *w_down_packed, int32_t D, int32_t F,
                     llep_dtype dtype, void *out_perm, void *workspace,
                     size_t workspace_bytes, hipStream_t stream);

/* Step 4 for training: llep_grouped_ffn, which also stores the gate and up
 * projections g = X Wg_e, u = X Wu_e of every row of the range (rounded to
 * dtype, as they enter the activation) so that llep_grouped_ffn_backward
 * need not recompute them. gate_up [T*K][2F] in dtype, row-major by x_perm
 * row, gate and up interleaved per 32 columns as in w_gate_up_packed:
 * g[:, 32j + c] at column 64j + c, u[:, 32j + c] at column 64j + 32 + c.
 * Rows outside the range are not written. out_perm is bit-identical to
 * llep_grouped_ffn's. gate_up non-null and 16-byte aligned.
 * Errors: as llep_grouped_ffn. */
int llep_grouped_ffn_train(const llep_plan_params *params,
                           const llep_plan_buffers *plan, int32_t device,
                           const void *x_perm, const void *w_gate_up_packed,
                           const void *w_down_packed, int32_t D, int32_t F,
                           llep_dtype dtype, void *out_perm, void *gate_up,
                           void *workspace, size_t workspace_bytes,
                           hipStream_t stream);

/* Bytes of the device array that the library holds on every GPU it runs on
 * (until the process ends) as the workspace of llep_grouped_ffn_noalloc. */
#define LLEP_NOALLOC_SCRATCH_BYTES (64u << 20)

/* llep_grouped_ffn for callers that cannot allocate device memory: code
 * under HIP graph capture, serving loops and harnesses that forbid hipMalloc.
 * The same kernels as llep_grouped_ffn with the same arguments, except that
 * the workspace is the library's own LLEP_NOALLOC_SCRATCH_BYTES array on the
 * current GPU instead of a caller buffer; out_perm is bit-identical to
 * llep_grouped_ffn's. The call allocates and frees nothing; what the kernels
 * need zeroed in the array they clear themselves (no memset node).
 * Requires llep_grouped_ffn_workspace_bytes(params, F, dtype) <=
 * LLEP_NOALLOC_SCRATCH_BYTES (for bf16 roughly (T*K + 16 (2E + P)) * F * 2
 * bytes), else LLEP_E_WORKSPACE and nothing is enqueued.
 * Every call on a GPU shares that GPU's array, which keeps the last call's
 * contents: calls on one stream are ordered and safe, but calls that overlap
 * on one GPU (other streams, other threads without ordering) race and give
 * undefined results. The first call on a GPU looks up the array's address
 * there (with that GPU current) and keeps it; make that first call outside
 * graph capture.
 * Errors: as llep_grouped_ffn (LLEP_E_WORKSPACE: too large for the array),
 * LLEP_E_HIP when the array's address cannot be obtained. */
int llep_grouped_ffn_noalloc(const llep_plan_params *params,
                             const llep_plan_buffers *plan, int32_t device,
                             const void *x_perm, const void *w_gate_up_packed,
                             const void *w_down_packed, int32_t D, int32_t F,
                             llep_dtype dtype, void *out_perm,
                             hipStream_t stream);

/* Step 5. y[t] = sum over k = 0..K-1 (ascending) of
 *   topk_gates[t*K+k] * out_perm[pair_row[t*K+k]]
 * in float32, rounded once to dtype; pairs with pair_row < 0 are skipped.
 * topk_gates may be null: every gate is then 1 (this sums the per-pair
 * input gradients dx_perm of llep_grouped_ffn_backward into dx).
 * out_perm [T*K][D], y [T][D] in `dtype`.
 * Errors: LLEP_E_ARG, LLEP_E_DTYPE. */
int llep_combine(const llep_plan_params *params, const void *out_perm,
                 const int32_t *pair_row, const float *topk_gates, int32_t D,
                 llep_dtype dtype, void *y, hipStream_t stream);

/* ---- backward (bf16) ------------------------------------------------------
 * The paper keeps LLEP exact under training: the gradients of the spilled
 * chunks computed on foreign devices go back to the expert's native device
 * and are added there (Sec. 1; Sec. 4). These calls give the backward of the
 * five steps above; the plan and permutation of the forward are reused.
 */

/* Backward of Eq. (1). For every pair p = t*K + k with r = pair_row[p] >= 0:
 *   d_out_perm[r] = topk_gates[p] * dy[t]        (rounded once to dtype)
 *   d_gates[p]    = sum_i dy[t][i] * out_perm[r][i]   (float32)
 * and d_gates[p] = 0 when pair_row[p] < 0. out_perm [T*K][D] (the forward's
 * expert outputs), dy [T][D], d_out_perm [T*K][D] in dtype; d_gates [T*K]
 * float32.
 * Errors: LLEP_E_ARG, LLEP_E_DTYPE. */
int llep_combine_backward(const llep_plan_params *params, const void *out_perm,
                          const int32_t *pair_row, const float *topk_gates,
                          const void *dy, int32_t D, llep_dtype dtype,
                          void *d_out_perm, float *d_gates, hipStream_t stream);

/* Packed weights of the backward GEMMs (untimed setup), same sizes as
 * llep_packed_gate_up_bytes / llep_packed_down_bytes, same block layout as
 * llep_pack_weights:
 *   w_gate_up_t_packed [E][D*2F]: K = 2F; P row d, k = 64j + c holds
 *                                 w_gate[d][32j + c], k = 64j + 32 + c holds
 *                                 w_up[d][32j + c] (the forward's gate/up
 *                                 interleave along the contraction);
 *   w_down_t_packed    [E][F*D]:  K = D; P row f = row f of w_down.
 * Requires D % 64 == 0, F % 64 == 0, both at most LLEP_MAX_FFN_DIM.
 * Errors: LLEP_E_ARG, LLEP_E_DTYPE. */
int llep_pack_weights_backward(int32_t E, int32_t D, int32_t F, llep_dtype dtype,
                               const void *w_gate, const void *w_up,
                               const void *w_down, void *w_gate_up_t_packed,
                               void *w_down_t_packed, hipStream_t stream);

/* Backward of step 4 for the groups of `device` (or of all devices when
 * device == -1). With X = x_perm[rows of a group (d, e, s, n)] and
 * dO = d_out_perm[same rows] (from llep_combine_backward):
 *   g = X Wg_e, u = X Wu_e, dA = dO Wd_e^T,
 *   dg = dA * u * silu'(g), du = dA * silu(g), act = silu(g) * u
 *   dx_perm[rows] = dg Wg_e^T + du Wu_e^T               (dtype)
 * and, per expert e with groups in the range, the weight gradients in
 * float32 (dw_gate, dw_up [E][D][F], dw_down [E][F][D]):
 *   dWg_e = sum over e's groups of X^T dg, dWu_e of X^T du, dWd_e of act^T dO
 * summed in gradient-return order: the group on e's native device (e / M)
 * first, then the groups on other devices by increasing device index. For
 * device == d these are d's partial gradients; for device == -1 they are the
 * totals each native device holds after the gradient return. Experts without
 * a group in the range are not written; rows outside the range are not
 * written. Weights are the llep_pack_weights (w_gate_up_packed) and
 * llep_pack_weights_backward outputs. bf16 uses matrix cores and rounds g,
 * u, dg, du and act to bf16 once each; f32 is a plain reference-precision
 * path (no intermediate rounding). g and u are read from gate_up when it
 * is non-null: the llep_grouped_ffn_train output for the same plan, x_perm
 * and weights, over the same device or over all devices (-1); the results
 * are then bit-identical to recomputing, and rows that call did not write
 * give undefined gradients. Null gate_up: g and u are recomputed (one more
 * grouped GEMM, into the workspace). Workspace of at least
 * llep_grouped_ffn_backward_workspace_bytes bytes, 256-byte aligned.
 * Requires D % 64 == 0, F % 64 == 0 (at most LLEP_MAX_FFN_DIM); dw_*
 * 16-byte aligned; T*K below about
 * 4.19 M pairs (the weight-gradient operands, each expert's rows end to end,
 * are addressed with 32-bit byte offsets; LLEP_E_ARG beyond).
 * Errors: LLEP_E_ARG, LLEP_E_DTYPE, LLEP_E_WORKSPACE. */
size_t llep_grouped_ffn_backward_workspace_bytes(const llep_plan_params *params,
                                                 int32_t D, int32_t F,
                                                 llep_dtype dtype);
int llep_grouped_ffn_backward(const llep_plan_params *params,
                              const llep_plan_buffers *plan, int32_t device,
                              const void *x_perm, const void *d_out_perm,
                              const void *w_gate_up_packed,
                              const void *w_gate_up_t_packed,
                              const void *w_down_t_packed, const void *gate_up,
                              int32_t D, int32_t F,
                              llep_dtype dtype, void *dx_perm, float *dw_gate,
                              float *dw_up, float *dw_down, void *workspace,
                              size_t workspace_bytes, hipStream_t stream);

/* Text of the calling thread's last error ("" if none). */
const char *llep_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* LLEP_H */
