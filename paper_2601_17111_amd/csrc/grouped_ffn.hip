// Step 4 of the LLEP hot path: grouped SwiGLU expert GEMMs over one device's
// groups (Alg. 4 grouped GEMMs for native and foreign experts; the
// three-matrix SwiGLU expert of Sec. 5.1).
//
// For a group (device, e, row_start, n) with X = x_perm[row_start, +n):
//   act = silu(X Wg_e) * (X Wu_e)      GEMM 1, SwiGLU fused in the epilogue
//   out = act Wd_e                      GEMM 2
//
// bf16 path: persistent workgroups walk a tile list built on the device from
// the group table (no host round trip). A tile never spans two groups. Tiles
// are handed out so that the workgroups resident on one XCD (the hardware
// deals workgroup ids round-robin over the 8 XCDs) work on neighbouring
// tiles, which share operand panels in that XCD's L2. MFMA
// v_mfma_f32_32x32x16_bf16 with fp32 accumulation; operand tiles are staged
// in LDS (double-buffered, XOR-swizzled 16-byte chunks).
//
// Packed weights (llep_pack_weights) keep the contraction dimension last, so
// both GEMMs read 16-byte runs along K for A and B alike. In the gate/up
// matrix, gate columns 32j..32j+31 are followed by the matching up columns,
// so one wave holds gate and up values of the same output element in the
// same accumulator register slot and applies SwiGLU without data exchange.
#include "common.h"
#include "kernels.h"

namespace llep {

constexpr int kBM = 128;
constexpr int kBN = 128;
constexpr int kBK = 64;
constexpr int kWavesM = 2;
constexpr int kWavesN = 2;
constexpr int kGroupM = 8;  // m-tiles per super-row of the tile order

struct WsLayout {
  size_t tiles_off, act_off, total;
  int64_t max_mtiles;
};

static WsLayout ws_layout(int64_t R, int32_t E, int32_t P, int32_t F, llep_dtype dtype) {
  WsLayout L;
  L.max_mtiles = R / kBM + (2 * int64_t(E) + P) + 1;
  L.tiles_off = 256;
  const size_t tiles_bytes = (size_t(L.max_mtiles) * 8 + 255) / 256 * 256;
  L.act_off = L.tiles_off + tiles_bytes;
  const size_t eb = dtype == LLEP_BF16 ? 2 : 4;
  L.total = L.act_off + size_t(R) * size_t(F) * eb;
  return L;
}

size_t ffn_workspace_bytes(int64_t R, int32_t E, int32_t P, int32_t F, llep_dtype dtype) {
  return ws_layout(R, E, P, F, dtype).total;
}

// ---------------------------------------------------------------------------
// tile list: one entry (group, m-tile) per BM rows of each group of the range
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void tile_table_kernel(const int32_t *__restrict__ groups,
                                                         const int32_t *__restrict__ group_begin,
                                                         int32_t device, int32_t P, int32_t BM,
                                                         int2 *__restrict__ tiles,
                                                         int32_t *__restrict__ n_tiles) {
  __shared__ int32_t part[256];
  __shared__ int32_t run;
  const int tid = threadIdx.x;
  const int lo = device < 0 ? group_begin[0] : group_begin[device];
  const int hi = device < 0 ? group_begin[P] : group_begin[device + 1];
  if (tid == 0) run = 0;
  __syncthreads();
  for (int g0 = lo; g0 < hi; g0 += 256) {
    const int g = g0 + tid;
    const int mt = g < hi ? (groups[4 * g + 3] + BM - 1) / BM : 0;
    part[tid] = mt;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
      const int32_t t = tid >= off ? part[tid - off] : 0;
      __syncthreads();
      part[tid] += t;
      __syncthreads();
    }
    const int32_t base = run + part[tid] - mt;
    for (int i = 0; i < mt; ++i) tiles[base + i] = make_int2(g, i);
    __syncthreads();
    if (tid == 255) run += part[255];
    __syncthreads();
  }
  if (tid == 0) *n_tiles = run;
}

// ---------------------------------------------------------------------------
// bf16 MFMA grouped GEMM: C[m][n] = sum_k A[m][k] B_e[n][k]
// ---------------------------------------------------------------------------

struct GemmArgs {
  const uint16_t *A;
  int64_t lda;
  const uint16_t *B;
  int64_t b_expert_stride;
  uint16_t *C;
  int64_t ldc;
  const int32_t *groups;
  const int2 *tiles;
  const int32_t *n_mtiles;
  int32_t N, Kdim;
};

__device__ __forceinline__ int lds_swz(int row, int kc) { return row * kBK + ((kc ^ (row & 7)) << 3); }

template <int BM, int BN, int WAVES_M, int WAVES_N, bool kSwiglu>
__global__ __launch_bounds__(64 * WAVES_M *WAVES_N) void gemm_bf16_kernel(GemmArgs g) {
  constexpr int NT = 64 * WAVES_M * WAVES_N;
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int A_CH = BM * kBK / 8 / NT;  // 16-byte chunks per thread
  constexpr int B_CH = BN * kBK / 8 / NT;
  static_assert(A_CH * NT * 8 == BM * kBK && B_CH * NT * 8 == BN * kBK, "tile/thread mismatch");
  static_assert(!kSwiglu || (WN % 64) == 0, "SwiGLU needs gate/up column pairs per wave");
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][BM * kBK];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][BN * kBK];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
  const int n_mt = *g.n_mtiles;
  const int n_nt = (g.N + BN - 1) / BN;
  const int total = n_mt * n_nt;
  const int G = gridDim.x;  // a multiple of 8
  const int slot = (blockIdx.x % 8) * (G / 8) + blockIdx.x / 8;
  const int nk = g.Kdim / kBK;

  for (int it = 0;; ++it) {
    const int u = it * G + slot;
    if (u >= total) break;
    // super-rows of kGroupM m-tiles; inside one, m-tile fastest
    const int sr = u / (kGroupM * n_nt);
    const int rem = u - sr * (kGroupM * n_nt);
    const int gm = min(kGroupM, n_mt - sr * kGroupM);
    const int nt = rem / gm;
    const int2 te = g.tiles[sr * kGroupM + rem % gm];
    const int32_t *gr = g.groups + 4 * te.x;
    const int e = gr[1], row0 = gr[2], n = gr[3];
    const int m0 = te.y * BM;
    const int rows_valid = min(BM, n - m0);
    const int n0 = nt * BN;
    const int cols_valid = min(BN, g.N - n0);
    const uint16_t *Ab = g.A + int64_t(row0 + m0) * g.lda;
    const uint16_t *Bb = g.B + int64_t(e) * g.b_expert_stride + int64_t(n0) * g.Kdim;

    int64_t a_off[A_CH], b_off[B_CH];
    int a_lds[A_CH], b_lds[B_CH];
#pragma unroll
    for (int i = 0; i < A_CH; ++i) {
      const int c = tid + i * NT, r = c >> 3, kc = c & 7;
      a_off[i] = int64_t(min(r, rows_valid - 1)) * g.lda + kc * 8;
      a_lds[i] = lds_swz(r, kc);
    }
#pragma unroll
    for (int i = 0; i < B_CH; ++i) {
      const int c = tid + i * NT, r = c >> 3, kc = c & 7;
      b_off[i] = int64_t(min(r, cols_valid - 1)) * g.Kdim + kc * 8;
      b_lds[i] = lds_swz(r, kc);
    }

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.0f;

    i32x4 ra[A_CH], rb[B_CH];
#pragma unroll
    for (int i = 0; i < A_CH; ++i) ra[i] = *reinterpret_cast<const i32x4 *>(Ab + a_off[i]);
#pragma unroll
    for (int i = 0; i < B_CH; ++i) rb[i] = *reinterpret_cast<const i32x4 *>(Bb + b_off[i]);
#pragma unroll
    for (int i = 0; i < A_CH; ++i) *reinterpret_cast<i32x4 *>(&sA[0][a_lds[i]]) = ra[i];
#pragma unroll
    for (int i = 0; i < B_CH; ++i) *reinterpret_cast<i32x4 *>(&sB[0][b_lds[i]]) = rb[i];
    __syncthreads();

    for (int kt = 0; kt < nk; ++kt) {
      const int cur = kt & 1;
      const bool more = kt + 1 < nk;
      if (more) {
        const int64_t k0 = int64_t(kt + 1) * kBK;
#pragma unroll
        for (int i = 0; i < A_CH; ++i) ra[i] = *reinterpret_cast<const i32x4 *>(Ab + a_off[i] + k0);
#pragma unroll
        for (int i = 0; i < B_CH; ++i) rb[i] = *reinterpret_cast<const i32x4 *>(Bb + b_off[i] + k0);
      }
#pragma unroll
      for (int ks = 0; ks < kBK / 16; ++ks) {
        const int kc = ks * 2 + (lane >> 5);
        bf16x8 af[TM], bfr[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int r = wm * WM + i * 32 + (lane & 31);
          af[i] = *reinterpret_cast<const bf16x8 *>(&sA[cur][lds_swz(r, kc)]);
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int r = wn * WN + j * 32 + (lane & 31);
          bfr[j] = *reinterpret_cast<const bf16x8 *>(&sB[cur][lds_swz(r, kc)]);
        }
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
      }
      if (more) {
#pragma unroll
        for (int i = 0; i < A_CH; ++i) *reinterpret_cast<i32x4 *>(&sA[cur ^ 1][a_lds[i]]) = ra[i];
#pragma unroll
        for (int i = 0; i < B_CH; ++i) *reinterpret_cast<i32x4 *>(&sB[cur ^ 1][b_lds[i]]) = rb[i];
      }
      __syncthreads();
    }

    // epilogue. Accumulator slot q of lane l in a 32x32 block holds
    // row 8*(q/4) + 4*(l/32) + q%4, column l%32.
    uint16_t *Cb = g.C + int64_t(row0 + m0) * g.ldc;
    if (kSwiglu) {
#pragma unroll
      for (int p = 0; p < TN / 2; ++p) {
        const int pc = n0 + wn * WN + p * 64;  // packed column of this gate block
        if (pc >= g.N) continue;
        const int f = (pc / 64) * 32 + (lane & 31);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            const int r = wm * WM + i * 32 + 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3);
            if (r < rows_valid) {
              const float gv = acc[i][2 * p][q], uv = acc[i][2 * p + 1][q];
              const float act = gv / (1.0f + __expf(-gv)) * uv;
              Cb[int64_t(r) * g.ldc + f] = f32_to_bf16(act);
            }
          }
      }
    } else {
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int col = n0 + wn * WN + j * 32 + (lane & 31);
        if (col >= g.N) continue;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            const int r = wm * WM + i * 32 + 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3);
            if (r < rows_valid) Cb[int64_t(r) * g.ldc + col] = f32_to_bf16(acc[i][j][q]);
          }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// float32 path: one thread per output element (small layers; reference
// precision, no matrix cores)
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

__global__ __launch_bounds__(256) void ffn_f32_gate_up_kernel(
    const float *__restrict__ x_perm, const float *__restrict__ wgu, float *__restrict__ act,
    const int32_t *__restrict__ groups, const int32_t *__restrict__ group_begin, int32_t device,
    int32_t P, int32_t D, int32_t F) {
  int lo, hi, row_first, rows;
  device_range(groups, group_begin, device, P, lo, hi, row_first, rows);
  const int64_t total = int64_t(rows) * F;
  for (int64_t u = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; u < total;
       u += int64_t(gridDim.x) * blockDim.x) {
    const int row = row_first + int(u / F), f = int(u % F);
    const int e = groups[4 * group_of_row(groups, lo, hi, row) + 1];
    const float *xr = x_perm + int64_t(row) * D;
    const int pg = 64 * (f / 32) + (f % 32);
    const float *wg = wgu + (int64_t(e) * 2 * F + pg) * D;
    const float *wu = wg + int64_t(32) * D;
    float gs = 0.0f, us = 0.0f;
    for (int d = 0; d < D; ++d) {
      gs = fmaf(xr[d], wg[d], gs);
      us = fmaf(xr[d], wu[d], us);
    }
    act[int64_t(row) * F + f] = gs / (1.0f + expf(-gs)) * us;
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
    const float *w = wd + (int64_t(e) * D + c) * F;
    float s = 0.0f;
    for (int f = 0; f < F; ++f) s = fmaf(ar[f], w[f], s);
    out[int64_t(row) * D + c] = s;
  }
}

// ---------------------------------------------------------------------------
// launch
// ---------------------------------------------------------------------------

static int cu_count() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 256;
  return n > 0 ? n : 256;
}

hipError_t launch_grouped_ffn(const FfnArgs &a, hipStream_t stream) {
  const WsLayout L = ws_layout(a.R, a.E, a.P, a.F, a.dtype);
  char *ws = static_cast<char *>(a.ws);
  int32_t *n_mtiles = reinterpret_cast<int32_t *>(ws);
  int2 *tiles = reinterpret_cast<int2 *>(ws + L.tiles_off);
  void *act = ws + L.act_off;
  const int grid = ((cu_count() * 2) + 7) / 8 * 8;
  if (a.dtype == LLEP_BF16) {
    hipLaunchKernelGGL(tile_table_kernel, dim3(1), dim3(256), 0, stream, a.groups, a.group_begin,
                       a.device, a.P, kBM, tiles, n_mtiles);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    GemmArgs g1;
    g1.A = static_cast<const uint16_t *>(a.x_perm);
    g1.lda = a.D;
    g1.B = static_cast<const uint16_t *>(a.w_gate_up);
    g1.b_expert_stride = int64_t(2) * a.F * a.D;
    g1.C = static_cast<uint16_t *>(act);
    g1.ldc = a.F;
    g1.groups = a.groups;
    g1.tiles = tiles;
    g1.n_mtiles = n_mtiles;
    g1.N = 2 * a.F;
    g1.Kdim = a.D;
    hipLaunchKernelGGL((gemm_bf16_kernel<kBM, kBN, kWavesM, kWavesN, true>), dim3(grid),
                       dim3(64 * kWavesM * kWavesN), 0, stream, g1);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    GemmArgs g2 = g1;
    g2.A = static_cast<const uint16_t *>(act);
    g2.lda = a.F;
    g2.B = static_cast<const uint16_t *>(a.w_down);
    g2.b_expert_stride = int64_t(a.D) * a.F;
    g2.C = static_cast<uint16_t *>(a.out_perm);
    g2.ldc = a.D;
    g2.N = a.D;
    g2.Kdim = a.F;
    hipLaunchKernelGGL((gemm_bf16_kernel<kBM, kBN, kWavesM, kWavesN, false>), dim3(grid),
                       dim3(64 * kWavesM * kWavesN), 0, stream, g2);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(ffn_f32_gate_up_kernel, dim3(1024), dim3(256), 0, stream,
                     static_cast<const float *>(a.x_perm), static_cast<const float *>(a.w_gate_up),
                     static_cast<float *>(act), a.groups, a.group_begin, a.device, a.P, a.D, a.F);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(ffn_f32_down_kernel, dim3(1024), dim3(256), 0, stream,
                     static_cast<const float *>(act), static_cast<const float *>(a.w_down),
                     static_cast<float *>(a.out_perm), a.groups, a.group_begin, a.device, a.P,
                     a.D, a.F);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// weight packing: tiled transposes (setup, not on the timed path)
// ---------------------------------------------------------------------------

// dst[b][map(c)][r] = src[b][r][c]; map: 0 identity, 1 gate slot, 2 up slot
// of the interleaved gate/up layout.
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
      dst[b * dbs + int64_t(drow) * rows + r] = tile[tx][i];
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
