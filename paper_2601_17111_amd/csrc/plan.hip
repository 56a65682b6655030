// Steps 1-2 of the LLEP hot path: the routing histogram and the plan.
//
// hist_kernel   counts, per rank tile of kRankTile pairs and per slice of
//               kRankSub pairs, how many pairs go to each expert (Alg. 4,
//               first step: the global per-expert loads).
// plan_kernel   one workgroup: scans the tile counts into per-tile rank bases
//               and the loads l, runs the lambda test (Alg. 4), then the
//               least-loaded assignment (Alg. 2 with the spill loop of
//               Alg. 3) or the standard EP assignment (Alg. 1), and lays the
//               result out as chunk / group / row / transfer tables.
//
// The assignment is sequential and greedy; it runs in one wavefront whose
// lanes are the devices: lane d holds the assigned and pending loads g_a[d],
// g_p[d] of Alg. 2. Sorting and table layout use the whole workgroup as
// all-pairs counts over at most 2E + P chunks (a position is the number of
// entries ahead of it), which needs two barriers instead of the dozens of a
// sorting network or a tree scan.
#include "common.h"
#include "kernels.h"

namespace llep {

int64_t rank_tiles(int64_t R) { return (R + kRankTile - 1) / kRankTile; }

// ---------------------------------------------------------------------------
// histogram
// ---------------------------------------------------------------------------

// rank_base layout: [n_tiles][E] counts (the plan turns them into each
// tile's base ranks), then [n_tiles] bad-id flags, then [n_tiles][kRankWaves][E]
// counts of each kRankSub-pair slice of a tile (a wave's share here; the
// permutation ranks slice by slice from them).
__global__ __launch_bounds__(256) void hist_kernel(const int32_t *__restrict__ ids,
                                                   int64_t R, int32_t E,
                                                   int32_t n_tiles,
                                                   int32_t *__restrict__ rank_base) {
  extern __shared__ int32_t cnt[];  // [kRankWaves][E]
  const int tid = threadIdx.x;
  for (int i = tid; i < kRankWaves * E; i += blockDim.x) cnt[i] = 0;
  __syncthreads();
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int nb = bits_for(uint32_t(E));
  const int64_t s0 = int64_t(blockIdx.x) * kRankTile + int64_t(w) * kRankSub;
  int32_t *wcnt = cnt + w * E;
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
    // one leader lane per expert value: no two lanes add to the same count
    if (e < uint32_t(E) && (m & lanemask_lt()) == 0) wcnt[e] += __popcll(m);
  }
  bad = __syncthreads_or(bad);
  int32_t *row = rank_base + int64_t(blockIdx.x) * E;
  int32_t *slices = rank_base + int64_t(n_tiles) * (E + 1) + int64_t(blockIdx.x) * kRankWaves * E;
  for (int i = tid; i < E; i += blockDim.x) {
    int32_t tot = 0;
#pragma unroll
    for (int v = 0; v < kRankWaves; ++v) {
      const int32_t c = cnt[v * E + i];
      slices[v * E + i] = c;
      tot += c;
    }
    row[i] = tot;
  }
  if (tid == 0) rank_base[int64_t(n_tiles) * E + blockIdx.x] = bad;
}

// ---------------------------------------------------------------------------
// plan
// ---------------------------------------------------------------------------

constexpr int kPlanThreads = 1024;
constexpr int kPlanWaves = kPlanThreads / kWave;

typedef int32_t i32x2 __attribute__((ext_vector_type(2)));

// Row-order key of a chunk: device, then expert, then emission index (the
// emission order of one expert's chunks is their start order). The low 20
// bits alone order chunks by (expert, start): the canonical order.
constexpr uint32_t kKeyBits = 0x3ffffffu;
constexpr uint32_t kRemoteFlag = 1u << 29;  // destination != native device
constexpr uint32_t kHeadFlag = 1u << 30;    // first chunk of its (device, expert)
static_assert(kMaxChunks <= 2048 && LLEP_MAX_EXPERTS <= 512 && LLEP_MAX_DEVICES <= 64,
              "row keys pack 6 + 9 + 11 bits");

__device__ __forceinline__ uint32_t row_key(int d, int e, int i) {
  return (uint32_t(d) << 20) | (uint32_t(e) << 11) | uint32_t(i);
}

struct PlanShared {
  // loads l[e], padded with -1 so 16-byte reads may run past E
  __attribute__((aligned(16))) int32_t loads[LLEP_MAX_EXPERTS + 4];
  int32_t sorted[LLEP_MAX_EXPERTS];  // experts by load descending, id ascending
  i32x4 chunk[kMaxChunks];           // (device, expert, start, end), emission order
  i32x2 key[kMaxChunks];             // (row key | remote flag, size)
  i32x2 key5[kMaxChunks];            // the same with the head flag
  int32_t row[kMaxChunks];           // first row of each chunk
  int32_t part[kPlanThreads];        // tile-scan segment sums
  int32_t e_cnt[LLEP_MAX_EXPERTS + 1];   // chunks per expert
  int32_t d_groups[LLEP_MAX_DEVICES + 1];  // groups per device
  int32_t dev_rows[LLEP_MAX_DEVICES];
  int32_t n_chunks, forced, status, bypass, n_groups, n_xfers, total_rows;
};

// Threads that share one chunk in the all-pairs passes over the chunk table
// (a power of two dividing the wave, so a chunk's threads are adjacent lanes).
__device__ __forceinline__ int lanes_per_chunk(int nc) {
  return nc <= 64 ? 16 : nc <= 128 ? 8 : nc <= 256 ? 4 : nc <= 512 ? 2 : 1;
}

template <typename V>
__device__ __forceinline__ V group_sum(V v, int S) {
  for (int off = 1; off < S; off <<= 1) v += __shfl_xor(v, off);
  return v;
}

// One whole wave: out[k] = in[0] + ... + in[k-1] for k < n (global store).
__device__ void wave_exclusive_scan(const int32_t *in, int n, int32_t *out) {
  const int lane = lane_id();
  const int per = (n + kWave - 1) / kWave;
  const int k0 = min(n, lane * per), k1 = min(n, k0 + per);
  int32_t sum = 0;
  for (int k = k0; k < k1; ++k) sum += in[k];
  int32_t incl = sum;
  for (int off = 1; off < kWave; off <<= 1) {
    const int32_t t = __shfl_up(incl, off);
    if (lane >= off) incl += t;
  }
  int32_t run = incl - sum;
  for (int k = k0; k < k1; ++k) {
    out[k] = run;
    run += in[k];
  }
}

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(PlanArgs a) {
  __shared__ PlanShared s;
  const int tid = threadIdx.x;
  const int wave = tid / kWave;
  const int E = a.E, P = a.P, M = a.M;
  const int nt = a.n_tiles;
  int32_t *rb = a.buf.rank_base;

  // ---- 1. scan tile counts: per-tile exclusive bases, and loads ----------
  // Each expert's column of tile counts is split into G segments; loads go
  // out eight at a time so a segment costs a few memory round trips.
  {
    const int G = kPlanThreads / E;  // E <= 512: G >= 2
    const int e = tid % E, grp = tid / E;
    const int seg = (nt + G - 1) / G;
    const int t0 = grp * seg, t1 = grp < G ? min(nt, t0 + seg) : t0;
    int32_t sum = 0;
    for (int t = t0; t < t1; t += 8) {
      int32_t v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = t + u < t1 ? rb[int64_t(t + u) * E + e] : 0;
#pragma unroll
      for (int u = 0; u < 8; ++u) sum += v[u];
    }
    s.part[tid] = sum;
    if (tid <= E) s.e_cnt[tid] = 0;
    if (tid <= P) s.d_groups[tid] = 0;
    if (tid < P) s.dev_rows[tid] = 0;
    if (tid < 4) s.loads[E + tid] = -1;
    __syncthreads();
    if (grp < G) {
      int32_t run = 0;
      for (int g = 0; g < grp; ++g) run += s.part[g * E + e];
      for (int t = t0; t < t1; t += 8) {
        int32_t v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = t + u < t1 ? rb[int64_t(t + u) * E + e] : 0;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if (t + u < t1) rb[int64_t(t + u) * E + e] = run;
          run += v[u];
        }
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
      s.n_groups = 0;
      s.n_xfers = 0;
      s.total_rows = 0;
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
  const int cmax = 2 * E + P;  // capacity of the caller's chunk tables
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
          s.chunk[i] = i32x4{e / M, e, 0, l};
          s.key[i] = i32x2{int32_t(row_key(e / M, e, i)), l};
        }
        nc += __popcll(on);
      }
      if (tid == 0) s.n_chunks = nc;
    }
  } else {
    // Alg. 2: experts by load descending, id ascending. Position of expert e
    // = number of experts ahead of it (all keys distinct).
    if (tid < E) {
      const int32_t le = s.loads[tid];
      int32_t pos = 0;
      const i32x4 *l4 = reinterpret_cast<const i32x4 *>(s.loads);
#pragma unroll 8
      for (int j4 = 0; j4 < (E + 3) / 4; ++j4) {
        const i32x4 v = l4[j4];
        const int j = 4 * j4;
        pos += (v.x > le || (v.x == le && j < tid)) ? 1 : 0;
        pos += (v.y > le || (v.y == le && j + 1 < tid)) ? 1 : 0;
        pos += (v.z > le || (v.z == le && j + 2 < tid)) ? 1 : 0;
        pos += (v.w > le || (v.w == le && j + 3 < tid)) ? 1 : 0;
      }
      s.sorted[pos] = tid;
    }
    __syncthreads();

    // The greedy loop runs in wave 0; lane d holds S[d] = g_a[d] + g_p[d].
    // Alg. 2 and 3 read g_a and g_p only through that sum: the native room
    // of expert e is cap - (S[ng] - l_e), so Case 1 holds iff S[ng] <= cap,
    // and Case 1 leaves S unchanged (l_e moves from g_p to g_a). A block of
    // 64 sorted experts is therefore tested against S at once; the experts
    // before the first one that does not fit are Case 1 and are emitted
    // together, and only experts that spill run one at a time.
    if (tid < kWave) {
      const int lane = tid;
      const int64_t cap = a.cap;
      const int64_t m = a.min_chunk < 1 ? 1 : a.min_chunk;
      int32_t S = 0;
      if (lane < P)
        for (int i = lane * M; i < lane * M + M; ++i) S += s.loads[i];
      const uint64_t dev_mask = P >= kWave ? ~uint64_t(0) : (uint64_t(1) << P) - 1;
      int nc = 0, forced = 0, overflow = 0;
      auto emit = [&](int d, int e, int ng, int64_t st, int64_t en) {
        if (nc < cmax) {
          if (lane == 0) {
            s.chunk[nc] = i32x4{d, e, int32_t(st), int32_t(en)};
            s.key[nc] = i32x2{int32_t(row_key(d, e, nc) | (d != ng ? kRemoteFlag : 0u)),
                              int32_t(en - st)};
          }
          ++nc;
        } else {
          overflow = 1;
        }
      };
      for (int b0 = 0; b0 < E; b0 += kWave) {
        const int k = b0 + lane;
        const int32_t ev = k < E ? s.sorted[k] : 0;
        const int32_t lv = k < E ? s.loads[ev] : 0;
        const int32_t nv = ev / M;
        const uint64_t live = __ballot(lv > 0);  // a prefix of the block
        int i = 0;
        while (i < kWave) {
          const int32_t s_native = __shfl(S, nv);
          const uint64_t pending = live & ~((uint64_t(1) << i) - 1);
          const uint64_t nofit = pending & __ballot(int64_t(s_native) > cap);
          const uint64_t fit =
              nofit ? pending & ((uint64_t(1) << __builtin_ctzll(nofit)) - 1) : pending;
          // Case 1 for every expert in `fit`, in order
          if ((fit >> lane) & 1) {
            const int idx = nc + __popcll(fit & lanemask_lt());
            if (idx < cmax) {
              s.chunk[idx] = i32x4{nv, ev, 0, lv};
              s.key[idx] = i32x2{int32_t(row_key(nv, ev, idx)), lv};
            }
          }
          nc += __popcll(fit);
          if (nc > cmax) {
            nc = cmax;
            overflow = 1;
          }
          if (nofit == 0) break;
          const int j = __builtin_ctzll(nofit);
          const int e = __builtin_amdgcn_readlane(ev, j);
          const int32_t l = __builtin_amdgcn_readlane(lv, j);
          const int ng = __builtin_amdgcn_readlane(nv, j);
          const int64_t na = cap - (int64_t(__builtin_amdgcn_readlane(S, ng)) - l);
          int64_t r = l, to = 0;
          if (na > 0) {
            // Case 2: the native device takes na and is then full
            emit(ng, e, ng, 0, na);
            if (lane == ng) S = int32_t(cap);
            r = l - na;
            to = na;
          } else if (lane == ng) {
            S -= l;  // Case 3: all of e leaves its native device
          }
          // Alg. 3. The other devices in (S, index) order have non-increasing
          // free room, so whenever the first one is skipped (room below both
          // m and r) every later one is skipped too and the force-assign goes
          // back to that first device: each round is one argmin over the
          // other devices (lowest index among ties).
          const uint64_t others = dev_mask & ~(uint64_t(1) << ng);
          while (r > 0) {
            int32_t best = 0;
            int o = -1;
            for (uint64_t mm = others; mm != 0; mm &= mm - 1) {
              const int d = __builtin_ctzll(mm);
              const int32_t v = __builtin_amdgcn_readlane(S, d);
              if (o < 0 || v < best) {
                best = v;
                o = d;
              }
            }
            const int64_t room = cap - int64_t(best);
            int64_t c;
            if (room >= r) {
              c = r;
            } else if (room >= m) {
              c = room;
            } else {
              c = r;  // force-assign the remainder
              ++forced;
            }
            emit(o, e, ng, to, to + c);
            if (lane == o) S += int32_t(c);
            r -= c;
            to += c;
          }
          i = j + 1;
        }
        if (live != (b0 + kWave <= E ? ~uint64_t(0) : (uint64_t(1) << (E - b0)) - 1))
          break;  // an empty expert: every later one is empty too
      }
      if (lane == 0) {
        s.n_chunks = nc;
        s.forced = forced;
        if (overflow) s.status |= kStatusPlanOverflow;
      }
    }
  }
  __syncthreads();
  const int nc = s.n_chunks;
  const int S = lanes_per_chunk(nc);

  // ---- 4. rows and the canonical chunk table ------------------------------
  // Chunk i's first row is the total size of the chunks before it in row
  // order; its canonical index is its position in (expert, start) order. Each
  // chunk's S threads split the count over j.
  for (int u = tid; u < nc * S; u += kPlanThreads) {
    const int i = u / S, q = u % S;
    const i32x2 wi = s.key[i];
    const uint32_t ki = uint32_t(wi.x) & kKeyBits;
    int32_t row = 0, canon = 0, dup = 0;
#pragma unroll 8
    for (int j = q; j < nc; j += S) {
      const i32x2 wj = s.key[j];
      const uint32_t kj = uint32_t(wj.x) & kKeyBits;
      const bool before = kj < ki;
      row += before ? wj.y : 0;
      dup += (before && (kj >> 11) == (ki >> 11)) ? 1 : 0;
      canon += (kj & 0xfffffu) < (ki & 0xfffffu) ? 1 : 0;
    }
    row = group_sum(row, S);
    canon = group_sum(canon, S);
    dup = group_sum(dup, S);
    if (q == 0) {
      const i32x4 ci = s.chunk[i];
      const bool head = dup == 0;
      s.row[i] = row;
      s.key5[i] = i32x2{int32_t(uint32_t(wi.x) | (head ? kHeadFlag : 0u)), wi.y};
      int32_t *cc = a.buf.chunks + 4 * canon;
      cc[0] = ci.x;
      cc[1] = ci.y;
      cc[2] = ci.z;
      cc[3] = ci.w;
      a.buf.chunk_row[canon] = row;
      atomicAdd(&s.dev_rows[ci.x], wi.y);
      atomicAdd(&s.total_rows, wi.y);
      atomicAdd(&s.e_cnt[ci.y], 1);
      if (head) {
        atomicAdd(&s.d_groups[ci.x], 1);
        atomicAdd(&s.n_groups, 1);
        if (uint32_t(wi.x) & kRemoteFlag) atomicAdd(&s.n_xfers, 1);
      }
    }
  }
  __syncthreads();

  // ---- 5. groups, transfers, per-device and per-expert offsets -----------
  // Group of a head chunk = heads before it in row order; its size sums the
  // chunks of its (device, expert). Transfer of a remote head = remote heads
  // before it in (expert, device) order: unique (expert, destination) pairs
  // whose destination is not the expert's native device.
  for (int u = tid; u < nc * S; u += kPlanThreads) {
    const int i = u / S, q = u % S;
    const i32x2 wi = s.key5[i];
    if (!(uint32_t(wi.x) & kHeadFlag)) continue;  // uniform over the chunk's S threads
    const uint32_t ki = uint32_t(wi.x) & kKeyBits;
    const uint32_t xi = (((ki >> 11) & 511u) << 6) | (ki >> 20);
    int32_t g = 0, n = 0, x = 0;
#pragma unroll 8
    for (int j = q; j < nc; j += S) {
      const i32x2 wj = s.key5[j];
      const uint32_t kj = uint32_t(wj.x) & kKeyBits;
      const uint32_t xj = (((kj >> 11) & 511u) << 6) | (kj >> 20);
      n += (kj >> 11) == (ki >> 11) ? wj.y : 0;
      g += ((uint32_t(wj.x) & kHeadFlag) && kj < ki) ? 1 : 0;
      x += ((uint32_t(wj.x) & kHeadFlag) && (uint32_t(wj.x) & kRemoteFlag) && xj < xi) ? 1 : 0;
    }
    g = group_sum(g, S);
    n = group_sum(n, S);
    x = group_sum(x, S);
    if (q == 0) {
      const int dev = int(ki >> 20), exp = int((ki >> 11) & 511u);
      int32_t *gr = a.buf.groups + 4 * g;
      gr[0] = dev;
      gr[1] = exp;
      gr[2] = s.row[i];
      gr[3] = n;
      if (uint32_t(wi.x) & kRemoteFlag) {
        int32_t *xr = a.buf.xfers + 3 * x;
        xr[0] = exp;
        xr[1] = exp / M;
        xr[2] = dev;
      }
    }
  }
  // expert_chunk_begin = exclusive scan of chunks per expert (last wave);
  // group_begin = exclusive scan of groups per device (the wave before it)
  if (wave == kPlanWaves - 1) wave_exclusive_scan(s.e_cnt, E + 1, a.buf.expert_chunk_begin);
  if (wave == kPlanWaves - 2) wave_exclusive_scan(s.d_groups, P + 1, a.buf.group_begin);
  if (tid < P) a.buf.device_rows[tid] = s.dev_rows[tid];

  // ---- 6. summary ----------------------------------------------------------
  if (tid == 0) {
    int best = 0;
    for (int d = 1; d < P; ++d)
      if (s.dev_rows[d] > s.dev_rows[best]) best = d;
    llep_plan_info info;
    info.status = s.status;
    info.n_chunks = nc;
    info.n_groups = s.n_groups;
    info.n_xfers = s.n_xfers;
    info.bypassed = (a.mode == LLEP_MODE_LLEP && P > 1 && use_ep) ? 1 : 0;
    info.forced = s.forced;
    info.max_device = best;
    info.total_rows = s.total_rows;
    *a.buf.info = info;
  }
}

hipError_t launch_plan(const PlanArgs &a, hipStream_t stream) {
  if (a.n_tiles > 0) {
    hipLaunchKernelGGL(hist_kernel, dim3(a.n_tiles), dim3(256),
                       size_t(kRankWaves) * a.E * sizeof(int32_t), stream, a.ids, a.R, a.E,
                       a.n_tiles, a.buf.rank_base);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kPlanThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace llep
