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
#include <mutex>

#include "gemm.h"

namespace llep {

struct WsLayout {
  size_t tiles_off, act_off, total;
  int64_t max_mtiles;
};

static WsLayout ws_layout(int64_t R, int32_t E, int32_t P, int32_t F, llep_dtype dtype) {
  WsLayout L;
  const int64_t max_groups = 2 * int64_t(E) + P;
  L.max_mtiles = R / kTileM + max_groups + 1;
  L.tiles_off = 256;
  const size_t tiles_bytes = (size_t(L.max_mtiles) * 16 + 255) / 256 * 256;
  L.act_off = L.tiles_off + tiles_bytes;
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
// activation matrix).
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void tile_table_kernel(const int32_t *__restrict__ groups,
                                                         const int32_t *__restrict__ group_begin,
                                                         int32_t device, int32_t P, int32_t BM,
                                                         int4 *__restrict__ tiles,
                                                         int32_t *__restrict__ n_tiles) {
  __shared__ int32_t part[256], prow[256];
  __shared__ int32_t run, prun;
  const int tid = threadIdx.x;
  const int lo = device < 0 ? group_begin[0] : group_begin[device];
  const int hi = device < 0 ? group_begin[P] : group_begin[device + 1];
  if (tid == 0) {
    run = 0;
    prun = 0;
  }
  __syncthreads();
  for (int g0 = lo; g0 < hi; g0 += 256) {
    const int g = g0 + tid;
    const int n = g < hi ? groups[4 * g + 3] : 0;
    const int mt = (n + BM - 1) / BM;
    const int pr = (n + 15) / 16 * 16;
    part[tid] = mt;
    prow[tid] = pr;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
      const int32_t t = tid >= off ? part[tid - off] : 0;
      const int32_t u = tid >= off ? prow[tid - off] : 0;
      __syncthreads();
      part[tid] += t;
      prow[tid] += u;
      __syncthreads();
    }
    const int32_t base = run + part[tid] - mt;
    const int32_t pbase = prun + prow[tid] - pr;
    for (int i = 0; i < mt; ++i) tiles[base + i] = make_int4(g, i, pbase, 0);
    __syncthreads();
    if (tid == 255) {
      run += part[255];
      prun += prow[255];
    }
    __syncthreads();
  }
  if (tid == 0) *n_tiles = run;
}

hipError_t launch_tile_table(const int32_t *groups, const int32_t *group_begin, int32_t device,
                             int32_t P, int4 *tiles, int32_t *n_tiles, hipStream_t stream) {
  hipLaunchKernelGGL(tile_table_kernel, dim3(1), dim3(256), 0, stream, groups, group_begin,
                     device, P, kTileM, tiles, n_tiles);
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
// launch
// ---------------------------------------------------------------------------

hipError_t launch_grouped_ffn(const FfnArgs &a, hipStream_t stream) {
  const WsLayout L = ws_layout(a.R, a.E, a.P, a.F, a.dtype);
  char *ws = static_cast<char *>(a.ws);
  int32_t *n_mtiles = reinterpret_cast<int32_t *>(ws);
  int4 *tiles = reinterpret_cast<int4 *>(ws + L.tiles_off);
  void *act = ws + L.act_off;
  if (a.dtype == LLEP_BF16) {
    const int grid = (cu_count() + 7) / 8 * 8;  // one workgroup per CU, XCD-balanced
    hipLaunchKernelGGL(tile_table_kernel, dim3(1), dim3(256), 0, stream, a.groups, a.group_begin,
                       a.device, a.P, kTileM, tiles, n_mtiles);
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
    constexpr int NT = 64 * kWavesM * kWavesN;
    hipLaunchKernelGGL((gemm256_kernel<256, kWavesM, kWavesN, kEpiSwiglu, false, true>),
                       dim3(grid), dim3(NT), 0, stream, g1);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
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
    if (a.D % 256 != 0 && a.D % 192 == 0)
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
