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
// g_p[d] of Alg. 2. The expert sort is an all-pairs count (a position is the
// number of experts ahead of it) spread over the whole workgroup. The table
// layout uses the order in which the greedy loop emits chunks: one expert's
// chunks are consecutive and in start order, so a chunk's canonical index is
// its expert's first canonical index plus its place in that run, and a
// chunk's row needs only a count over the chunks of its own device (bucketed
// by device) plus its expert's earlier chunks on the same device.
#include <type_traits>

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
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int nb = bits_for(uint32_t(E));
  const int64_t s0 = int64_t(blockIdx.x) * kRankTile + int64_t(w) * kRankSub;
  int32_t *wcnt = cnt + w * E;
  int bad = 0;
  // all of the slice's ids are requested, before the counts are cleared,
  // and only then counted (a pair past the end reads the last pair's id, in
  // bounds, and is dropped)
  constexpr int kPer = kRankSub / kWave;
  int32_t raw[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int64_t p = s0 + j * kWave + lane_id();
    raw[j] = ids[p < R ? p : R - 1];
  }
  __builtin_amdgcn_sched_barrier(0);  // the loads issue together
  for (int i = tid; i < kRankWaves * E; i += blockDim.x) cnt[i] = 0;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const bool in = s0 + j * kWave + lane_id() < R;
    const bool ok = raw[j] >= 0 && raw[j] < E;
    if (in && !ok) bad = 1;
    const uint32_t e = in && ok ? uint32_t(raw[j]) : uint32_t(E);  // sentinel: past the end or invalid
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

// Tile counts of one expert column that a thread keeps in registers
// between the two passes of the scan (and loads at once in either pass).
constexpr int kScanHold = 32;
static_assert(LLEP_MAX_EXPERTS <= kPlanThreads / 2 && LLEP_MAX_DEVICES <= kWave,
              "two threads per expert in the scan, one lane per device");

// Sort key of expert e: larger load first, then smaller id (Alg. 2's order
// with ties broken by id). Loads are non-negative.
__device__ __forceinline__ uint64_t sort_key(int32_t load, int e) {
  return (uint64_t(uint32_t(load)) << 32) | uint64_t(~uint32_t(e));
}

struct PlanShared {
  int32_t loads[LLEP_MAX_EXPERTS];   // l[e]
  int32_t sorted[LLEP_MAX_EXPERTS];  // experts by load descending, id ascending
  i32x4 chunk[kMaxChunks];           // (device, expert, start, end), emission order
  int32_t slot[kMaxChunks];          // place of the chunk in its device's bucket
  int32_t row_in[kMaxChunks];        // rows of earlier chunks of its (device, expert)
  int32_t head[kMaxChunks];          // first chunk of its (device, expert)
  int32_t bucket[kMaxChunks];        // chunks grouped by device
  int32_t part[kPlanThreads];        // tile-scan segment sums
  int32_t e_first[LLEP_MAX_EXPERTS];       // emission index of each expert's first chunk
  int32_t e_cnt[LLEP_MAX_EXPERTS + 1];     // chunks per expert -> canonical bases
  int32_t e_xfers[LLEP_MAX_EXPERTS + 1];   // remote groups per expert -> transfer bases
  int32_t d_chunks[LLEP_MAX_DEVICES + 1];  // chunks per device -> bucket bases
  int32_t d_groups[LLEP_MAX_DEVICES + 1];  // groups per device -> group bases
  int32_t dev_rows[LLEP_MAX_DEVICES + 1];  // rows per device
  int32_t d_row0[LLEP_MAX_DEVICES + 1];    // first row of each device, then the total
  int32_t n_chunks, forced, status, bypass, n_groups, n_xfers;
};

// Threads that share one chunk in the pass over its device's bucket (a power
// of two dividing the wave, so a chunk's threads are adjacent lanes).
__device__ __forceinline__ int lanes_per_chunk(int nc) {
  return nc <= 64 ? 16 : nc <= 128 ? 8 : nc <= 256 ? 4 : nc <= 512 ? 2 : 1;
}

template <typename V>
__device__ __forceinline__ V group_sum(V v, int S) {
  for (int off = 1; off < S; off <<= 1) v += __shfl_xor(v, off);
  return v;
}

// One whole wave: the minimum of x over its 64 lanes, in every lane. Row
// shifts by 1, 2, 4 and 8 leave each 16-lane row's minimum in its last lane;
// two row broadcasts carry those into lane 63. A lane whose DPP source lies
// outside its row, or in a row the step does not write, keeps its own value.
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x) {
  auto step = [&](auto ctrl, auto rows) {
    const uint32_t y = uint32_t(__builtin_amdgcn_update_dpp(int(x), int(x), decltype(ctrl)::value,
                                                            decltype(rows)::value, 0xf, false));
    x = min(x, y);
  };
  step(std::integral_constant<int, 0x111>{}, std::integral_constant<int, 0xf>{});  // row_shr:1
  step(std::integral_constant<int, 0x112>{}, std::integral_constant<int, 0xf>{});  // row_shr:2
  step(std::integral_constant<int, 0x114>{}, std::integral_constant<int, 0xf>{});  // row_shr:4
  step(std::integral_constant<int, 0x118>{}, std::integral_constant<int, 0xf>{});  // row_shr:8
  step(std::integral_constant<int, 0x142>{}, std::integral_constant<int, 0xa>{});  // row_bcast:15
  step(std::integral_constant<int, 0x143>{}, std::integral_constant<int, 0xc>{});  // row_bcast:31
  return uint32_t(__builtin_amdgcn_readlane(int(x), 63));
}

// One whole wave: out[k] = in[0] + ... + in[k-1] for k < n; out2, when given,
// gets a copy.
__device__ void wave_exclusive_scan(const int32_t *in, int n, int32_t *out,
                                    int32_t *out2 = nullptr) {
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
    const int32_t v = in[k];
    out[k] = run;
    if (out2 != nullptr) out2[k] = run;
    run += v;
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
  // Each expert's column of tile counts is split into G segments. A segment
  // of up to kScanHold tiles is loaded at once and kept in registers for the
  // second pass, so the scan costs one memory round trip (plus the stores);
  // longer segments take two passes of kScanHold loads at a time.
  {
    const int G = kPlanThreads / E;  // E <= 512: G >= 2
    const int e = tid % E, grp = tid / E;
    const int seg = (nt + G - 1) / G;
    const int t0 = grp * seg, t1 = grp < G ? min(nt, t0 + seg) : t0;
    const bool hold = seg <= kScanHold;  // uniform
    int bad = 0;
    for (int t = tid; t < nt; t += kPlanThreads) bad |= rb[int64_t(nt) * E + t];
    int32_t v[kScanHold];
    int32_t sum = 0;
    if (hold) {
      // in steps of 8 up to the (uniform) segment length
#pragma unroll
      for (int u0 = 0; u0 < kScanHold; u0 += 8) {
        if (u0 >= seg) break;
#pragma unroll
        for (int u = u0; u < u0 + 8; ++u) v[u] = t0 + u < t1 ? rb[int64_t(t0 + u) * E + e] : 0;
      }
#pragma unroll
      for (int u0 = 0; u0 < kScanHold; u0 += 8) {
        if (u0 >= seg) break;
#pragma unroll
        for (int u = u0; u < u0 + 8; ++u) sum += v[u];
      }
    } else {
      for (int t = t0; t < t1; t += kScanHold) {
#pragma unroll
        for (int u = 0; u < kScanHold; ++u) v[u] = t + u < t1 ? rb[int64_t(t + u) * E + e] : 0;
#pragma unroll
        for (int u = 0; u < kScanHold; ++u) sum += v[u];
      }
    }
    s.part[tid] = sum;
    if (tid <= E) {
      s.e_cnt[tid] = 0;
      s.e_xfers[tid] = 0;
    }
    if (tid <= P) {
      s.d_chunks[tid] = 0;
      s.d_groups[tid] = 0;
      s.dev_rows[tid] = 0;
    }
    bad = __syncthreads_or(bad);
    if (grp < G) {
      int32_t run = 0;
      for (int g = 0; g < grp; ++g) run += s.part[g * E + e];
      if (hold) {
#pragma unroll
        for (int u0 = 0; u0 < kScanHold; u0 += 8) {
          if (u0 >= seg) break;
#pragma unroll
          for (int u = u0; u < u0 + 8; ++u) {
            if (t0 + u < t1) rb[int64_t(t0 + u) * E + e] = run;
            run += v[u];
          }
        }
      } else {
        for (int t = t0; t < t1; t += kScanHold) {
#pragma unroll
          for (int u = 0; u < kScanHold; ++u) v[u] = t + u < t1 ? rb[int64_t(t + u) * E + e] : 0;
#pragma unroll
          for (int u = 0; u < kScanHold; ++u) {
            if (t + u < t1) rb[int64_t(t + u) * E + e] = run;
            run += v[u];
          }
        }
      }
      if (grp == G - 1) s.loads[e] = run;
    }
    if (tid == 0) {
      s.status = bad ? LLEP_STATUS_BAD_EXPERT_ID : 0;
      s.n_chunks = 0;
      s.forced = 0;
      s.bypass = 0;
      s.n_groups = 0;
      s.n_xfers = 0;
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
        }
        nc += __popcll(on);
      }
      if (tid == 0) s.n_chunks = nc;
    }
  } else {
    // Alg. 2: experts by load descending, id ascending. Position of expert e
    // = number of experts ahead of it (all keys distinct), counted by the G
    // adjacent threads of e (a power of two, at most a wave), each taking
    // every G-th expert.
    {
      int G = 1;
      while (G < kWave && 2 * G * E <= kPlanThreads) G *= 2;
      const int e = tid / G, q = tid % G;
      if (e < E) {  // uniform over e's G lanes
        const uint64_t ke = sort_key(s.loads[e], e);
        int32_t pos = 0;
#pragma unroll 8
        for (int j = q; j < E; j += G) pos += sort_key(s.loads[j], j) > ke ? 1 : 0;
        pos = group_sum(pos, G);
        if (q == 0) s.sorted[pos] = e;
      }
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
          if (lane == 0) s.chunk[nc] = i32x4{d, e, int32_t(st), int32_t(en)};
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
            if (idx < cmax) s.chunk[idx] = i32x4{nv, ev, 0, lv};
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
          const bool other = ((dev_mask >> lane) & 1) && lane != ng;
          while (r > 0) {
            // the smallest S among the other devices (S >= 0, so unsigned
            // order is S's order), then the lowest lane that holds it
            const uint32_t least = wave_min_u32(other ? uint32_t(S) : 0xffffffffu);
            const int o = __builtin_ctzll(__ballot(other && uint32_t(S) == least));
            const int32_t best = int32_t(least);
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

  // ---- 4. table layout ----------------------------------------------------
  // Both assignments emit one expert's chunks consecutively and in start
  // order. Row order is (device, expert, start); canonical order is (expert,
  // start).
  // (a) per chunk: its expert's first chunk, its place in its device's
  //     bucket, and the per-expert chunk and per-device row counts.
  for (int i = tid; i < nc; i += kPlanThreads) {
    const i32x4 ci = s.chunk[i];
    if (i == 0 || s.chunk[i - 1].y != ci.y) s.e_first[ci.y] = i;
    s.slot[i] = atomicAdd(&s.d_chunks[ci.x], 1);
    atomicAdd(&s.e_cnt[ci.y], 1);
    atomicAdd(&s.dev_rows[ci.x], ci.w - ci.z);
  }
  __syncthreads();
  // (b) per chunk: rows of its expert's earlier chunks on the same device
  //     (none: it heads a group); group and transfer counts. Scans of the
  //     counts so far: canonical bases, bucket bases, device first rows.
  for (int i = tid; i < nc; i += kPlanThreads) {
    const i32x4 ci = s.chunk[i];
    int32_t before = 0, head = 1;
    for (int j = s.e_first[ci.y]; j < i; ++j) {
      const i32x4 cj = s.chunk[j];
      if (cj.x == ci.x) {
        before += cj.w - cj.z;
        head = 0;
      }
    }
    s.row_in[i] = before;
    s.head[i] = head;
    if (head) {
      atomicAdd(&s.d_groups[ci.x], 1);
      atomicAdd(&s.n_groups, 1);
      if (ci.x != ci.y / M) {
        atomicAdd(&s.e_xfers[ci.y], 1);
        atomicAdd(&s.n_xfers, 1);
      }
    }
  }
  if (wave == kPlanWaves - 1) wave_exclusive_scan(s.e_cnt, E + 1, s.e_cnt, a.buf.expert_chunk_begin);
  if (wave == kPlanWaves - 2) wave_exclusive_scan(s.d_chunks, P + 1, s.d_chunks);
  if (wave == kPlanWaves - 3) wave_exclusive_scan(s.dev_rows, P + 1, s.d_row0);
  __syncthreads();
  // (c) bucket the chunks by device; scans of the group and transfer counts.
  for (int i = tid; i < nc; i += kPlanThreads) s.bucket[s.d_chunks[s.chunk[i].x] + s.slot[i]] = i;
  if (wave == kPlanWaves - 1) wave_exclusive_scan(s.e_xfers, E + 1, s.e_xfers);
  if (wave == kPlanWaves - 2) wave_exclusive_scan(s.d_groups, P + 1, s.d_groups, a.buf.group_begin);
  __syncthreads();
  // (d) per chunk, S threads over its device's bucket: rows and groups of
  //     smaller experts on the device give its row and group index; its
  //     expert's run of chunks gives its canonical index, its group's size and
  //     its transfer index (remote groups of the expert on smaller devices).
  //     Every index is checked against its table before the store.
  for (int u = tid; u < nc * S; u += kPlanThreads) {
    const int i = u / S, q = u % S;
    const i32x4 ci = s.chunk[i];
    const int b0 = s.d_chunks[ci.x], b1 = s.d_chunks[ci.x + 1];
    int32_t rows = 0, heads = 0;
#pragma unroll 4
    for (int k = b0 + q; k < b1; k += S) {
      const int j = s.bucket[k];
      const i32x4 cj = s.chunk[j];
      if (cj.y < ci.y) {
        rows += cj.w - cj.z;
        heads += s.head[j];
      }
    }
    rows = group_sum(rows, S);
    heads = group_sum(heads, S);
    if (q == 0) {
      const int32_t row = s.d_row0[ci.x] + rows + s.row_in[i];
      const int f = s.e_first[ci.y];
      const int canon = s.e_cnt[ci.y] + (i - f);
      if (canon >= 0 && canon < nc) {
        int32_t *cc = a.buf.chunks + 4 * canon;
        cc[0] = ci.x;
        cc[1] = ci.y;
        cc[2] = ci.z;
        cc[3] = ci.w;
        a.buf.chunk_row[canon] = row;
      }
      if (s.head[i]) {
        const bool remote = ci.x != ci.y / M;
        const int f1 = min(nc, s.e_cnt[ci.y + 1] - s.e_cnt[ci.y] + f);
        int32_t n = 0, x = 0;
        for (int j = f; j < f1; ++j) {
          const i32x4 cj = s.chunk[j];
          if (cj.x == ci.x) n += cj.w - cj.z;
          if (s.head[j] && cj.x < ci.x && cj.x != ci.y / M) ++x;
        }
        const int g = s.d_groups[ci.x] + heads;
        if (g >= 0 && g < s.n_groups) {
          int32_t *gr = a.buf.groups + 4 * g;
          gr[0] = ci.x;
          gr[1] = ci.y;
          gr[2] = row;
          gr[3] = n;
        }
        x += s.e_xfers[ci.y];
        if (remote && x >= 0 && x < s.n_xfers) {
          int32_t *xr = a.buf.xfers + 3 * x;
          xr[0] = ci.y;
          xr[1] = ci.y / M;
          xr[2] = ci.x;
        }
      }
    }
  }
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
    info.total_rows = s.d_row0[P];
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
