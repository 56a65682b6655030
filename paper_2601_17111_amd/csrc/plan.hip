// Steps 1-2 of the LLEP hot path: the routing histogram and the plan.
//
// hist_kernel   counts, per rank tile of kRankTile pairs, how many pairs go
//               to each expert (Alg. 4, "sum of loads of global experts").
// plan_kernel   one workgroup: scans the tile counts into per-tile rank bases
//               and the loads l, runs the lambda test (Alg. 4), then the
//               least-loaded assignment (Alg. 2 with the spill loop of
//               Alg. 3) or the standard EP assignment (Alg. 1), and lays the
//               result out as chunk / group / row / transfer tables.
//
// The assignment is sequential and greedy; it runs in one wavefront whose
// lanes are the devices: lane d holds the assigned and pending loads g_a[d],
// g_p[d] of Alg. 2. Everything else (sorting, scans, table layout) uses the
// whole workgroup.
#include "common.h"
#include "kernels.h"

namespace llep {

int64_t rank_tiles(int64_t R) { return (R + kRankTile - 1) / kRankTile; }

// ---------------------------------------------------------------------------
// histogram
// ---------------------------------------------------------------------------

// rank_base layout: [n_tiles][E] counts, then [n_tiles] bad-id flags.
__global__ __launch_bounds__(256) void hist_kernel(const int32_t *__restrict__ ids,
                                                   int64_t R, int32_t E,
                                                   int32_t n_tiles,
                                                   int32_t *__restrict__ rank_base) {
  extern __shared__ int32_t cnt[];  // [E]
  const int tid = threadIdx.x;
  for (int i = tid; i < E; i += blockDim.x) cnt[i] = 0;
  __syncthreads();
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int nb = bits_for(uint32_t(E));
  const int64_t s0 = int64_t(blockIdx.x) * kRankTile + int64_t(w) * kRankSub;
  int bad = 0;
  for (int j = 0; j < kRankSub; j += kWave) {
    if (s0 + j >= R) break;  // uniform in the wave
    const int64_t p = s0 + j + lane_id();
    uint32_t e = uint32_t(E);  // sentinel: past the end or invalid
    if (p < R) {
      const int32_t v = ids[p];
      if (v >= 0 && v < E) e = uint32_t(v);
      else bad = 1;
    }
    const uint64_t m = match_any(e, nb);
    if (e < uint32_t(E) && (m & lanemask_lt()) == 0)
      atomicAdd(&cnt[e], __popcll(m));
  }
  bad = __syncthreads_or(bad);
  int32_t *row = rank_base + int64_t(blockIdx.x) * E;
  for (int i = tid; i < E; i += blockDim.x) row[i] = cnt[i];
  if (tid == 0) rank_base[int64_t(n_tiles) * E + blockIdx.x] = bad;
}

// ---------------------------------------------------------------------------
// plan
// ---------------------------------------------------------------------------

constexpr int kPlanThreads = 1024;
constexpr int kSortMax = 2048;  // power of two >= kMaxChunks

static_assert(kSortMax >= kMaxChunks, "sort buffer too small");
static_assert(kSortMax <= 2 * kPlanThreads, "scan handles 2 items per thread");

__device__ __forceinline__ int next_pow2(int v) {
  int p = 1;
  while (p < v) p <<= 1;
  return p;
}

// Ascending bitonic sort of key[0 .. n), n a power of two, whole workgroup.
template <typename K>
__device__ void bitonic_sort(K *key, int n) {
  for (int k = 2; k <= n; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = threadIdx.x; i < n; i += kPlanThreads) {
        const int ixj = i ^ j;
        if (ixj > i) {
          const K a = key[i], b = key[ixj];
          const bool up = (i & k) == 0;
          if ((a > b) == up) {
            key[i] = b;
            key[ixj] = a;
          }
        }
      }
      __syncthreads();
    }
  }
}

// In-place exclusive scan of a[0 .. n), n <= 2 * kPlanThreads; returns the
// total. Whole workgroup; part has kPlanThreads entries.
__device__ int32_t block_scan_excl(int32_t *a, int n, int32_t *part) {
  const int tid = threadIdx.x;
  const int i0 = 2 * tid, i1 = 2 * tid + 1;
  const int32_t v0 = i0 < n ? a[i0] : 0;
  const int32_t v1 = i1 < n ? a[i1] : 0;
  part[tid] = v0 + v1;
  __syncthreads();
  for (int off = 1; off < kPlanThreads; off <<= 1) {
    const int32_t t = tid >= off ? part[tid - off] : 0;
    __syncthreads();
    part[tid] += t;
    __syncthreads();
  }
  const int32_t excl = tid > 0 ? part[tid - 1] : 0;
  const int32_t total = part[kPlanThreads - 1];
  __syncthreads();
  if (i0 < n) a[i0] = excl;
  if (i1 < n) a[i1] = excl + v0;
  __syncthreads();
  return total;
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
  for (int off = 1; off < kWave; off <<= 1) {
    const uint64_t o = __shfl_xor(v, off);
    v = o < v ? o : v;
  }
  return v;
}

struct PlanShared {
  int32_t loads[LLEP_MAX_EXPERTS];
  uint64_t ekey[LLEP_MAX_EXPERTS];
  int32_t part[kPlanThreads];
  int32_t e_first[LLEP_MAX_EXPERTS];
  int32_t e_cnt[LLEP_MAX_EXPERTS + 1];
  int32_t c_dev[kMaxChunks];
  int32_t c_exp[kMaxChunks];
  int32_t c_start[kMaxChunks];
  int32_t c_end[kMaxChunks];
  int32_t c_canon[kMaxChunks];
  uint32_t skey[kSortMax];
  int32_t srow[kSortMax];
  int32_t g_row[kMaxChunks];
  int32_t g_dev[kMaxChunks];
  int32_t n_chunks, forced, status, bypass, n_groups, total_rows;
};

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(PlanArgs a) {
  __shared__ PlanShared s;
  const int tid = threadIdx.x;
  const int E = a.E, P = a.P, M = a.M;
  const int nt = a.n_tiles;
  int32_t *rb = a.buf.rank_base;

  // ---- 1. scan tile counts: per-tile exclusive bases, and loads ----------
  {
    const int G = kPlanThreads / E;  // tile segments (E <= 512: G >= 2)
    const int e = tid % E, grp = tid / E;
    const int seg = (nt + G - 1) / G;
    const int t0 = grp * seg, t1 = min(nt, t0 + seg);
    int32_t sum = 0;
    if (grp < G)
      for (int t = t0; t < t1; ++t) sum += rb[int64_t(t) * E + e];
    s.part[tid] = sum;
    if (tid < E) s.e_first[tid] = -1;
    if (tid <= E) s.e_cnt[tid] = 0;
    __syncthreads();
    if (grp < G) {
      int32_t run = 0;
      for (int g = 0; g < grp; ++g) run += s.part[g * E + e];
      for (int t = t0; t < t1; ++t) {
        const int32_t v = rb[int64_t(t) * E + e];
        rb[int64_t(t) * E + e] = run;
        run += v;
      }
      if (grp == G - 1) s.loads[e] = run;
    }
    int bad = 0;
    for (int t = tid; t < nt; t += kPlanThreads) bad |= rb[int64_t(nt) * E + t];
    bad = __syncthreads_or(bad);
    if (tid == 0) {
      s.status = bad ? LLEP_STATUS_BAD_EXPERT_ID : 0;
      s.n_chunks = 0;
      s.forced = 0;
      s.bypass = 0;
    }
    __syncthreads();
  }
  for (int e = tid; e < E; e += kPlanThreads) a.buf.loads[e] = s.loads[e];

  // ---- 2. lambda test (Alg. 4): max(l) * E < lambda * sum(l) ------------
  bool use_ep = a.mode == LLEP_MODE_EP || P == 1;
  if (!use_ep && a.lambda > 0.0) {
    if (tid < kWave) {
      int32_t mx = 0;
      int64_t sm = 0;
      for (int e = tid; e < E; e += kWave) {
        mx = max(mx, s.loads[e]);
        sm += s.loads[e];
      }
      for (int off = 1; off < kWave; off <<= 1) {
        mx = max(mx, __shfl_xor(mx, off));
        sm += __shfl_xor(sm, off);
      }
      if (tid == 0)
        s.bypass = (double(mx) * double(E) < a.lambda * double(sm)) ? 1 : 0;
    }
    __syncthreads();
    use_ep = s.bypass != 0;
  }

  // ---- 3. assignment ------------------------------------------------------
  if (use_ep) {
    // Alg. 1: one chunk [0, l_e) per non-empty expert on device e / M,
    // emitted in expert order.
    if (tid < kWave) {
      int nc = 0;
      for (int e0 = 0; e0 < E; e0 += kWave) {
        const int e = e0 + tid;
        const int32_t l = e < E ? s.loads[e] : 0;
        const uint64_t on = __ballot(l > 0);
        if (l > 0) {
          const int i = nc + __popcll(on & lanemask_lt());
          s.c_dev[i] = e / M;
          s.c_exp[i] = e;
          s.c_start[i] = 0;
          s.c_end[i] = l;
          s.e_first[e] = i;
          s.e_cnt[e] = 1;
        }
        nc += __popcll(on);
      }
      if (tid == 0) s.n_chunks = nc;
    }
    __syncthreads();
  } else {
    // Alg. 2: experts by load descending, id ascending.
    const int ne = next_pow2(E);
    for (int i = tid; i < ne; i += kPlanThreads)
      s.ekey[i] = i < E ? (uint64_t(uint32_t(0x7fffffff - s.loads[i])) << 32) | uint32_t(i)
                        : ~uint64_t(0);
    __syncthreads();
    bitonic_sort(s.ekey, ne);

    if (tid < kWave) {
      const int lane = tid;
      const int64_t cap = a.cap;
      const int64_t m = a.min_chunk < 1 ? 1 : a.min_chunk;
      int64_t ga = 0, gp = 0;  // g_a[lane], g_p[lane]
      if (lane < P)
        for (int i = lane * M; i < lane * M + M; ++i) gp += s.loads[i];
      int nc = 0, forced = 0, overflow = 0;
      auto emit = [&](int d, int e, int64_t st, int64_t en) {
        if (nc < kMaxChunks) {
          if (lane == 0) {
            s.c_dev[nc] = d;
            s.c_exp[nc] = e;
            s.c_start[nc] = int32_t(st);
            s.c_end[nc] = int32_t(en);
          }
          ++nc;
        } else {
          overflow = 1;
        }
      };
      for (int idx = 0; idx < E; ++idx) {
        const int e = int(uint32_t(s.ekey[idx]));
        const int64_t l = s.loads[e];
        if (l == 0) break;  // sorted: every remaining expert is empty
        const int ng = e / M;
        if (lane == ng) gp -= l;
        const int64_t ga_ng = __shfl(ga, ng), gp_ng = __shfl(gp, ng);
        const int64_t na = cap - ga_ng - gp_ng;  // room on the native device
        const int c0 = nc;
        if (na >= l) {
          // Case 1: the native device takes all of e
          emit(ng, e, 0, l);
          if (lane == ng) ga += l;
        } else {
          int64_t r = l, to = 0;
          if (na > 0) {
            // Case 2: the native device takes na, the rest spills
            emit(ng, e, 0, na);
            if (lane == ng) ga += na;
            r = l - na;
            to = na;
          }
          // Alg. 3. The other devices in (g_a + g_p, index) order have
          // non-increasing free room, so whenever the first one is skipped
          // (room below both m and r) every later one is skipped too and the
          // force-assign goes back to that first device: each round is one
          // argmin over the other devices.
          while (r > 0) {
            const uint64_t key = (lane < P && lane != ng) ? uint64_t(ga + gp) : ~uint64_t(0);
            const uint64_t mn = wave_min_u64(key);
            const int o = __ffsll((unsigned long long)__ballot(key == mn)) - 1;
            const int64_t room = cap - int64_t(mn);
            int64_t c;
            if (room >= r) {
              c = r;
            } else if (room >= m) {
              c = room;
            } else {
              c = r;  // force-assign the remainder
              ++forced;
            }
            emit(o, e, to, to + c);
            if (lane == o) ga += c;
            r -= c;
            to += c;
          }
        }
        if (lane == 0) {
          s.e_first[e] = c0;
          s.e_cnt[e] = nc - c0;
        }
      }
      if (lane == 0) {
        s.n_chunks = min(nc, kMaxChunks);
        s.forced = forced;
        if (overflow) s.status |= kStatusPlanOverflow;
      }
    }
    __syncthreads();
  }
  const int nc = s.n_chunks;

  // ---- 4. canonical chunk table: by expert, then start -------------------
  const int32_t n_canon = block_scan_excl(s.e_cnt, E + 1, s.part);  // e_cnt -> begin
  (void)n_canon;
  for (int e = tid; e <= E; e += kPlanThreads) a.buf.expert_chunk_begin[e] = s.e_cnt[e];
  for (int i = tid; i < nc; i += kPlanThreads) {
    const int e = s.c_exp[i];
    const int ci = s.e_cnt[e] + (i - s.e_first[e]);
    s.c_canon[i] = ci;
    int32_t *c = a.buf.chunks + 4 * ci;
    c[0] = s.c_dev[i];
    c[1] = e;
    c[2] = s.c_start[i];
    c[3] = s.c_end[i];
  }

  // ---- 5. rows: device-major, expert, then start (= emission order) -------
  __syncthreads();
  const int ns = next_pow2(nc > 0 ? nc : 1);
  for (int i = tid; i < ns; i += kPlanThreads)
    s.skey[i] = i < nc ? (uint32_t(s.c_dev[i]) << 20) | (uint32_t(s.c_exp[i]) << 11) | uint32_t(i)
                       : 0xffffffffu;
  __syncthreads();
  bitonic_sort(s.skey, ns);
  for (int j = tid; j < ns; j += kPlanThreads) {
    const int i = int(s.skey[j] & 0x7ffu);
    s.srow[j] = j < nc ? s.c_end[i] - s.c_start[i] : 0;
  }
  __syncthreads();
  // srow[j] becomes the first row of the j-th chunk in row order
  const int32_t total_rows = block_scan_excl(s.srow, ns, s.part);
  for (int j = tid; j < nc; j += kPlanThreads)
    a.buf.chunk_row[s.c_canon[int(s.skey[j] & 0x7ffu)]] = s.srow[j];
  // group heads: the first chunk of each (device, expert) in row order.
  // c_start is free from here on and holds the head flags, scanned into
  // each head's group index.
  for (int j = tid; j < nc; j += kPlanThreads)
    s.c_start[j] = (j == 0 || (s.skey[j] >> 11) != (s.skey[j - 1] >> 11)) ? 1 : 0;
  __syncthreads();
  const int32_t n_groups = block_scan_excl(s.c_start, nc, s.part);
  for (int j = tid; j < nc; j += kPlanThreads) {
    if (j == 0 || (s.skey[j] >> 11) != (s.skey[j - 1] >> 11)) {
      const int g = s.c_start[j];
      s.g_row[g] = s.srow[j];
      s.g_dev[g] = int(s.skey[j] >> 20);
      s.c_end[g] = int((s.skey[j] >> 11) & 0x1ffu);  // expert of group g
    }
  }
  __syncthreads();
  for (int g = tid; g < n_groups; g += kPlanThreads) {
    const int32_t next_row = g + 1 < n_groups ? s.g_row[g + 1] : total_rows;
    int32_t *gr = a.buf.groups + 4 * g;
    gr[0] = s.g_dev[g];
    gr[1] = s.c_end[g];
    gr[2] = s.g_row[g];
    gr[3] = next_row - s.g_row[g];
  }
  // group_begin[d] = number of groups on devices below d (binary search)
  if (tid <= P) {
    int lo = 0, hi = n_groups;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (s.g_dev[mid] < tid) lo = mid + 1;
      else hi = mid;
    }
    s.part[tid] = lo;
  }
  __syncthreads();
  if (tid <= P) a.buf.group_begin[tid] = s.part[tid];
  if (tid < P) {
    const int g0 = s.part[tid], g1 = s.part[tid + 1];
    const int32_t r0 = g0 < n_groups ? s.g_row[g0] : total_rows;
    const int32_t r1 = g1 < n_groups ? s.g_row[g1] : total_rows;
    a.buf.device_rows[tid] = r1 - r0;
    s.e_first[tid] = r1 - r0;  // e_first is free: device rows for the summary
  }
  __syncthreads();

  // ---- 6. weight transfers: unique (expert, dst) with dst != native -------
  for (int i = tid; i < ns; i += kPlanThreads) {
    uint32_t k = 0xffffffffu;
    if (i < nc && s.c_dev[i] != s.c_exp[i] / M)
      k = (uint32_t(s.c_exp[i]) << 6) | uint32_t(s.c_dev[i]);
    s.skey[i] = k;
  }
  __syncthreads();
  bitonic_sort(s.skey, ns);
  for (int j = tid; j < nc; j += kPlanThreads) {
    const uint32_t k = s.skey[j];
    s.c_start[j] = (k != 0xffffffffu && (j == 0 || k != s.skey[j - 1])) ? 1 : 0;
  }
  __syncthreads();
  const int32_t n_xfers = block_scan_excl(s.c_start, nc, s.part);
  for (int j = tid; j < nc; j += kPlanThreads) {
    const uint32_t k = s.skey[j];
    if (k != 0xffffffffu && (j == 0 || k != s.skey[j - 1])) {
      const int e = int(k >> 6), d = int(k & 63u);
      int32_t *x = a.buf.xfers + 3 * s.c_start[j];
      x[0] = e;
      x[1] = e / M;
      x[2] = d;
    }
  }

  // ---- 7. summary ----------------------------------------------------------
  if (tid == 0) {
    int best = 0;
    for (int d = 1; d < P; ++d)
      if (s.e_first[d] > s.e_first[best]) best = d;
    llep_plan_info info;
    info.status = s.status;
    info.n_chunks = nc;
    info.n_groups = n_groups;
    info.n_xfers = n_xfers;
    info.bypassed = (a.mode == LLEP_MODE_LLEP && P > 1 && use_ep) ? 1 : 0;
    info.forced = s.forced;
    info.max_device = best;
    info.total_rows = total_rows;
    *a.buf.info = info;
  }
}

hipError_t launch_plan(const PlanArgs &a, hipStream_t stream) {
  if (a.n_tiles > 0) {
    hipLaunchKernelGGL(hist_kernel, dim3(a.n_tiles), dim3(256),
                       size_t(a.E) * sizeof(int32_t), stream, a.ids, a.R, a.E,
                       a.n_tiles, a.buf.rank_base);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kPlanThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace llep
