"""Plain CPU oracle of the LLEP expert-layer hot path (test infrastructure).

Only tests, the smoke entry point and the benchmark's CPU baseline leg may use
this module. It shares no code with the HIP library.

Paper: "Least-Loaded Expert Parallelism: Load Balancing An Imbalanced
Mixture-of-Experts" (arXiv 2601.17111).

What is computed, and where the paper defines it:

* expert loads l                 -- Alg. 4, first step (global per-expert loads)
* the LLA plan                    -- Alg. 2 (least-loaded assignment) and
                                     Alg. 3 (least-loaded assignment spill),
                                     with the constraints paragraph of Sec. 4
* the standard EP plan            -- Alg. 1 (experts [pM, (p+1)M-1] on device p)
* the lambda bypass               -- Alg. 4, the max/mean imbalance test
* the permutation                 -- Sec. 2.1, implementation paragraph
                                     (re-indexing by expert, token order kept
                                     inside an expert); Alg. 4's sorting,
                                     gathering and chunk-building steps
* the expert outputs              -- Eq. (1)-(2) with the three-matrix SwiGLU
                                     expert of Sec. 5.1; plan-free, float64

Readings taken where the paper is silent or ambiguous (the same readings bind
the GPU library):

* capacity is an integer number of token-expert pairs; a real alpha is turned
  into one by ceil(alpha * sum(l) / P) with alpha as an exact rational;
* sorting the loads (Alg. 2) orders by load descending, expert id ascending;
* the other devices that Alg. 3 ranks by assigned plus pending load are
  ranked by that sum, then by device index;
* a minimum chunk size m below 1 is read as 1 (with m = 0 Alg. 3 could assign
  empty chunks forever);
* the force-assign of Alg. 3 goes to the least-loaded *other* device (the
  algorithm box), not to the native one;
* empty chunks (zero-load experts in Case 1) are dropped;
* the range [start, end) of expert e names e's token-expert pairs in
  ascending pair index p = t*K + k;
* the lambda test bypasses LLA iff  max(l) * N < lambda * sum(l)  evaluated in
  IEEE double, over all N experts; lambda <= 0 disables it;
* with a single device (P = 1) the plan is the standard EP plan;
* inside a device, rows are ordered by expert id, then by chunk start; several
  chunks of one (device, expert) form a single group;
* SwiGLU has no bias and no clamp: (silu(x Wg) * (x Wu)) Wd;
* an expert id outside [0, N) is not counted, gets no row and sets status
  bit 1.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field
from fractions import Fraction
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

STATUS_BAD_EXPERT_ID = 1


# ---------------------------------------------------------------------------
# Step 1: expert loads (Alg. 4, first step: the global per-expert loads)
# ---------------------------------------------------------------------------

def expert_loads(ids_flat: Sequence[int], E: int) -> Tuple[List[int], int]:
    """Count the token-expert pairs routed to each expert.

    Returns (loads, status). Ids outside [0, E) are not counted and set
    STATUS_BAD_EXPERT_ID in the status word.
    """
    loads = [0] * E
    status = 0
    for e in ids_flat:
        e = int(e)
        if 0 <= e < E:
            loads[e] += 1
        else:
            status |= STATUS_BAD_EXPERT_ID
    return loads, status


def capacity_from_alpha(total_load: int, alpha: Fraction, P: int) -> int:
    """Per-device capacity m_alpha = alpha * sum(l) / P (Alg. 2; Sec. 4,
    Constraints), rounded up to a whole number of pairs."""
    alpha = Fraction(alpha)
    return int(math.ceil(alpha * total_load / P))


# ---------------------------------------------------------------------------
# Step 2: the plan (Alg. 2 LLA, Alg. 3 LLAS, Alg. 1 standard EP)
# ---------------------------------------------------------------------------

class DeviceLedger:
    """Per-device bookkeeping of the least-loaded assignment (Alg. 2).

    placed[d]  -- pairs already given to device d (native or foreign);
    pending[d] -- pairs of d's own experts that have not been visited yet,
                  held in reserve so that a device keeps room for its own
                  experts before it accepts foreign ones;
    cap        -- the integer capacity m_alpha.

    A device's occupancy is placed + pending; its free room is cap minus
    that (negative once the device is over capacity).
    """

    def __init__(self, native_load: List[int], cap: int):
        self.placed = [0] * len(native_load)
        self.pending = list(native_load)
        self.cap = cap

    def occupancy(self, d: int) -> int:
        return self.placed[d] + self.pending[d]

    def free(self, d: int) -> int:
        return self.cap - self.occupancy(d)

    def give(self, d: int, n: int) -> None:
        self.placed[d] += n


def spill_to_least_loaded(ledger: DeviceLedger, home: int, remaining: int,
                          offset: int, m: int) -> Tuple[List[Tuple[int, int, int]], int]:
    """The spill step (Alg. 3): place `remaining` pairs of an expert whose
    native device is `home`, starting at pair offset `offset`, on the other
    devices.

    Each round ranks every other device by occupancy (ties: lower index) and
    walks that ranking from the emptiest device on. A device is taken if the
    piece it could hold -- its free room, at most the pairs still to place --
    is at least m pairs, or is everything that is left. If no device
    qualifies, all remaining pairs go to the emptiest other device even
    though that exceeds its capacity (a force-assignment).

    Returns the pieces (device, start, end) in the order they were made and
    the number of force-assignments.
    """
    P = len(ledger.placed)
    pieces: List[Tuple[int, int, int]] = []
    forced = 0
    while remaining > 0:
        ranking = sorted((d for d in range(P) if d != home),
                         key=lambda d: (ledger.occupancy(d), d))
        target, take = None, 0
        for d in ranking:
            room = min(remaining, ledger.free(d))
            if room >= m or room == remaining:
                target, take = d, room
                break
        if target is None:
            target, take = ranking[0], remaining
            forced += 1
        pieces.append((target, offset, offset + take))
        ledger.give(target, take)
        offset += take
        remaining -= take
    return pieces, forced


def least_loaded_assignment(loads: Sequence[int], M: int, cap: int, m: int
                            ) -> Tuple[Dict[int, List[Tuple[int, int, int]]],
                                       List[Tuple[int, int, int]], int]:
    """The least-loaded assignment (Alg. 2).

    loads: per-expert load l (length N = P*M); M: experts per device;
    cap: integer capacity m_alpha; m: minimum pairs per spilled GEMM.

    Experts are visited from the largest load to the smallest (ties: lower
    expert id). Visiting an expert releases its reserved pairs from its
    native device's pending load; the native device then keeps as many of
    the expert's pairs as its free room allows (all of them, some, or none:
    the three cases of Alg. 2), and the rest goes through the spill step.

    Returns (assignments, transfers, forced):
      assignments[e] = [(device, start, end), ...], non-empty pieces in the
                       order they were made;
      transfers      = sorted unique (expert, src, dst) weight moves: a piece
                       of expert e on a device q other than its native one
                       needs e's weights copied native -> q (the transfer
                       plan W of Alg. 2);
      forced         = number of force-assignments.
    """
    N = len(loads)
    assert N % M == 0
    P = N // M
    m = max(1, int(m))
    loads = [int(v) for v in loads]
    if P == 1:
        # no other device to spill to: the plan is the standard EP plan
        return standard_ep_assignment(loads, M), [], 0
    ledger = DeviceLedger([sum(loads[d * M:(d + 1) * M]) for d in range(P)], cap)
    assignments: Dict[int, List[Tuple[int, int, int]]] = {}
    forced = 0
    for e in sorted(range(N), key=lambda i: (-loads[i], i)):
        home = e // M
        ledger.pending[home] -= loads[e]
        keep = min(loads[e], max(0, ledger.free(home)))
        pieces: List[Tuple[int, int, int]] = []
        if keep > 0:
            pieces.append((home, 0, keep))
            ledger.give(home, keep)
        if loads[e] > keep:
            spilled, f = spill_to_least_loaded(ledger, home, loads[e] - keep, keep, m)
            pieces += spilled
            forced += f
        assignments[e] = [(d, s, t) for (d, s, t) in pieces if t > s]
    transfers = sorted({(e, e // M, d)
                        for e, pieces in assignments.items()
                        for (d, s, t) in pieces if d != e // M})
    return assignments, transfers, forced


def standard_ep_assignment(loads: Sequence[int], M: int
                           ) -> Dict[int, List[Tuple[int, int, int]]]:
    """Alg. 1: device p computes all pairs of experts pM .. (p+1)M-1."""
    return {e: ([(e // M, 0, int(l))] if int(l) > 0 else [])
            for e, l in enumerate(loads)}


def bypass_to_standard_ep(loads: Sequence[int], lam: float) -> bool:
    """Alg. 4: run standard EP when max(l) / mean(l) < lambda.

    Evaluated as  max(l) * N < lambda * sum(l)  in IEEE double; lambda <= 0
    never bypasses.
    """
    if lam <= 0.0:
        return False
    N = len(loads)
    return float(max(loads)) * float(N) < float(lam) * float(sum(loads))


@dataclass
class PlanResult:
    """Plan tables, in the layout the GPU library also produces.

    chunks      : list of (device, expert, start, end), sorted by (expert, start)
    chunk_row   : first destination row of each chunk (same order)
    expert_chunk_begin : length N+1; chunks of expert e are
                  chunks[expert_chunk_begin[e]:expert_chunk_begin[e+1]]
    groups      : list of (device, expert, row_start, n), device-major, then
                  expert ascending; one group per (device, expert)
    group_begin : length P+1; groups of device d are
                  groups[group_begin[d]:group_begin[d+1]]
    device_rows : rows computed by each device
    transfers   : sorted unique (expert, src, dst)
    """
    loads: List[int]
    chunks: List[Tuple[int, int, int, int]]
    chunk_row: List[int]
    expert_chunk_begin: List[int]
    groups: List[Tuple[int, int, int, int]]
    group_begin: List[int]
    device_rows: List[int]
    transfers: List[Tuple[int, int, int]]
    status: int = 0
    bypassed: bool = False
    forced: int = 0
    capacity: int = 0
    extra: dict = field(default_factory=dict)

    @property
    def max_device(self) -> int:
        best = 0
        for d, v in enumerate(self.device_rows):
            if v > self.device_rows[best]:
                best = d
        return best


def plan_tables(assignments: Dict[int, List[Tuple[int, int, int]]],
                loads: Sequence[int], P: int, M: int) -> dict:
    """Lay an assignment map out as chunk, group and row tables.

    Rows are numbered device by device; inside a device by expert id, then by
    chunk start (Alg. 4 builds per-destination chunks and each device computes
    its native and foreign experts' GEMMs).
    """
    N = len(loads)
    chunks = []
    for e in range(N):
        for (d, s, t) in sorted(assignments.get(e, []), key=lambda c: c[1]):
            chunks.append((d, e, s, t))
    expert_chunk_begin = [0] * (N + 1)
    for (_, e, _, _) in chunks:
        expert_chunk_begin[e + 1] += 1
    for e in range(N):
        expert_chunk_begin[e + 1] += expert_chunk_begin[e]
    # rows: device-major, then expert, then chunk start
    by_row = sorted(range(len(chunks)),
                    key=lambda c: (chunks[c][0], chunks[c][1], chunks[c][2]))
    chunk_row = [0] * len(chunks)
    groups: List[List[int]] = []
    row = 0
    for c in by_row:
        d, e, s, t = chunks[c]
        chunk_row[c] = row
        if groups and groups[-1][0] == d and groups[-1][1] == e:
            groups[-1][3] += t - s
        else:
            groups.append([d, e, row, t - s])
        row += t - s
    group_begin = [0] * (P + 1)
    for g in groups:
        group_begin[g[0] + 1] += 1
    for d in range(P):
        group_begin[d + 1] += group_begin[d]
    device_rows = [0] * P
    for g in groups:
        device_rows[g[0]] += g[3]
    transfers = sorted({(e, e // M, d) for (d, e, s, t) in chunks
                        if d != e // M})
    return dict(chunks=chunks, chunk_row=chunk_row,
                expert_chunk_begin=expert_chunk_begin,
                groups=[tuple(g) for g in groups], group_begin=group_begin,
                device_rows=device_rows, transfers=transfers)


def plan(ids_flat: Sequence[int], E: int, P: int, cap: int, m: int = 1,
         mode: str = "llep", lam: float = 0.0) -> PlanResult:
    """The full plan step: loads, then (optionally) the lambda bypass, then
    LLA or the standard EP assignment, laid out as tables.

    mode: "llep" (Alg. 4 with Alg. 2/3) or "ep" (Alg. 1).
    """
    assert E % P == 0
    M = E // P
    loads, status = expert_loads(ids_flat, E)
    bypassed = False
    forced = 0
    if mode == "ep":
        A = standard_ep_assignment(loads, M)
    elif mode == "llep":
        if P == 1 or bypass_to_standard_ep(loads, lam):
            bypassed = P > 1
            A = standard_ep_assignment(loads, M)
        else:
            A, _, forced = least_loaded_assignment(loads, M, cap, m)
    else:
        raise ValueError(mode)
    t = plan_tables(A, loads, P, M)
    return PlanResult(loads=loads, status=status, bypassed=bypassed,
                      forced=forced, capacity=cap, **t)


# ---------------------------------------------------------------------------
# Step 3: the permutation (Sec. 2.1 re-indexing; Alg. 4 sorting and gathering)
# ---------------------------------------------------------------------------

def pair_ranks(ids_flat: Sequence[int], E: int) -> List[int]:
    """Rank of each pair among the pairs of its expert, in pair order
    (a stable counting sort by expert, Sec. 2.1). -1 for invalid ids."""
    seen = [0] * E
    rank = []
    for e in ids_flat:
        e = int(e)
        if 0 <= e < E:
            rank.append(seen[e])
            seen[e] += 1
        else:
            rank.append(-1)
    return rank


def permute(ids_flat: Sequence[int], pl: PlanResult, E: int
            ) -> Tuple[np.ndarray, np.ndarray]:
    """Destination row of every pair under plan `pl`.

    Pair p of expert e with rank r lies in the chunk (d, e, s, t) with
    s <= r < t, and goes to row chunk_row + (r - s).

    Returns (pair_row[R], row_pair[rows]); pair_row is -1 for invalid ids.
    """
    ranks = pair_ranks(ids_flat, E)
    R = len(ranks)
    total = sum(pl.device_rows)
    pair_row = np.full(R, -1, dtype=np.int64)
    row_pair = np.full(total, -1, dtype=np.int64)
    for p in range(R):
        r = ranks[p]
        if r < 0:
            continue
        e = int(ids_flat[p])
        for c in range(pl.expert_chunk_begin[e], pl.expert_chunk_begin[e + 1]):
            d, ce, s, t = pl.chunks[c]
            if s <= r < t:
                row = pl.chunk_row[c] + (r - s)
                pair_row[p] = row
                row_pair[row] = p
                break
    return pair_row, row_pair


# ---------------------------------------------------------------------------
# Step 4: expert outputs (Eq. 1-2, SwiGLU expert of Sec. 5.1), float64
# ---------------------------------------------------------------------------

def silu(z):
    """silu(z) = z * sigmoid(z) = z / (1 + exp(-z))."""
    z = np.asarray(z, dtype=np.float64)
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def swiglu_ffn(v: np.ndarray, wg: np.ndarray, wu: np.ndarray, wd: np.ndarray
               ) -> np.ndarray:
    """FFN(v) = (silu(v Wg) * (v Wu)) Wd for rows v (n x D), in float64.

    wg, wu: D x F; wd: F x D.
    """
    v = np.asarray(v, dtype=np.float64)
    h = silu(v @ np.asarray(wg, dtype=np.float64))
    u = v @ np.asarray(wu, dtype=np.float64)
    return (h * u) @ np.asarray(wd, dtype=np.float64)


def moe_output(x: np.ndarray, ids: np.ndarray, gates: np.ndarray,
               expert_weights, tokens: Optional[Sequence[int]] = None
               ) -> np.ndarray:
    """Eq. (1): y[t] = sum_k gates[t, k] * FFN_{ids[t, k]}(x[t]), float64.

    Plan-free: LLEP does not change the layer's output, so the oracle never
    looks at the plan here.

    x: T x D; ids, gates: T x K; expert_weights(e) -> (Wg, Wu, Wd);
    tokens: the tokens to compute (default all). Returns len(tokens) x D.
    Pairs with an id outside [0, N) contribute nothing.
    """
    T, K = ids.shape
    if tokens is None:
        tokens = list(range(T))
    tokens = [int(t) for t in tokens]
    D = x.shape[1]
    y = np.zeros((len(tokens), D), dtype=np.float64)
    # group (sample index, k) by expert so each expert's weights load once
    by_expert: Dict[int, List[Tuple[int, int]]] = {}
    for i, t in enumerate(tokens):
        for k in range(K):
            by_expert.setdefault(int(ids[t, k]), []).append((i, k))
    for e, items in sorted(by_expert.items()):
        w = expert_weights(e)
        if w is None:
            continue
        wg, wu, wd = w
        rows = np.array([tokens[i] for (i, _) in items])
        out = swiglu_ffn(np.asarray(x, dtype=np.float64)[rows], wg, wu, wd)
        for j, (i, k) in enumerate(items):
            y[i] += np.float64(gates[tokens[i], k]) * out[j]
    return y


def combine(pair_out: np.ndarray, gates: np.ndarray) -> np.ndarray:
    """Eq. (1) given each pair's expert output: y[t] = sum_k gates[t, k] *
    pair_out[t, k] (float64). pair_out: T x K x D; gates: T x K."""
    return np.einsum("tk,tkd->td", np.asarray(gates, dtype=np.float64),
                     np.asarray(pair_out, dtype=np.float64))


# ---------------------------------------------------------------------------
# Per-device peak memory of a plan (Sec. 3.2, Eq. 4)
# ---------------------------------------------------------------------------

def m_local(groups: Sequence[Tuple[int, int, int, int]], P: int, D: int, F: int,
            matrices: int = 3) -> List[int]:
    """Eq. (4): the peak memory of the MoE layer on one device, in elements,
    M_local = sum over the device's groups i of (B_i D + matrices D H + B_i H),
    with B_i the group's rows (token-expert pairs), H = F the expert's hidden
    size and `matrices` weight matrices of D x H per expert.

    Eq. (4) counts one D x H matrix per expert; the SwiGLU expert of
    Sec. 5.1 has three (gate, up, down), so the default is 3, and
    matrices=1 gives Eq. (4) as printed. Each group is one (device, expert)
    GEMM problem, so a spilled expert counts its weights once on every
    device that holds a piece of it.

    groups: (device, expert, row_start, n) rows of a plan. Returns a list of
    P element counts.
    """
    out = [0] * P
    for (d, _e, _r0, n) in groups:
        out[int(d)] += int(n) * D + matrices * D * F + int(n) * F
    return out


# ---------------------------------------------------------------------------
# Exhaustive optimum on tiny inputs (a pin for the plan's quality)
# ---------------------------------------------------------------------------

def min_max_load_exhaustive(loads: Sequence[int], P: int, M: int,
                            cap: Optional[int] = None) -> Tuple[int, Optional[int]]:
    """Exhaustively split every expert's load over the P devices.

    Returns (opt, min_foreign):
      opt         = the smallest achievable max device load;
      min_foreign = over all splits with max load <= cap, the fewest
                    (expert, device) pairs with device != native(expert) and a
                    non-empty share (None when cap is None or infeasible).
    Exponential; meant for N <= 4, P <= 3, loads <= 6.
    """
    states: Dict[Tuple[int, ...], int] = {tuple([0] * P): 0}
    for e, l in enumerate(loads):
        l = int(l)
        splits = _compositions(l, P)
        nxt: Dict[Tuple[int, ...], int] = {}
        for st, foreign in states.items():
            for sp in splits:
                ld = tuple(st[d] + sp[d] for d in range(P))
                f = foreign + sum(1 for d in range(P)
                                  if sp[d] > 0 and d != e // M)
                if ld not in nxt or f < nxt[ld]:
                    nxt[ld] = f
        states = nxt
    opt = min(max(st) for st in states)
    min_foreign = None
    if cap is not None:
        feas = [f for st, f in states.items() if max(st) <= cap]
        min_foreign = min(feas) if feas else None
    return opt, min_foreign


def _compositions(n: int, parts: int) -> List[Tuple[int, ...]]:
    if parts == 1:
        return [(n,)]
    out = []
    for first in range(n + 1):
        for rest in _compositions(n - first, parts - 1):
            out.append((first,) + rest)
    return out
