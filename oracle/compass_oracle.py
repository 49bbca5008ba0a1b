"""Plain fp64 CPU oracle of the Compass hot path.

TEST INFRASTRUCTURE ONLY. Nothing on the product path may import, call or
execute this module: only the tests, the smoke check and the benchmark's
CPU-baseline leg use it. It shares no code with the HIP path; the only common
module is the seeded input generator (``synth``), which holds no arithmetic
of the method.

Paper: "Compass: Dissecting Communication and Computation Operators for
Efficient LLM Training" (arXiv 2609.10549). Citations name sections,
equations, tables and figures of that paper.

Contents
  * bf16 decoding / encoding (the oracle's own, fp64 <-> bf16 bits)
  * GEMM parts, by their textbook definitions:
      - ``ag_gemm``: explicit AllGather (shards stacked in rank order) then
        A_g @ B  (Section II-A, Fig. 1: AllGather before GEMM0)
      - ``gemm_rs``: A @ B, row chunk c summed with the incoming partial of
        chunk c  (Section II-A: ReduceScatter after GEMM1)
      - ``decomp_ag`` / ``decomp_rs``: d independent sub-operators over row
        pieces, scattered back (Section II-B, Fig. 2(c); Section IV)
      - ``tile_ordered_ag`` / ``tile_ordered_rs``: the same products computed
        tile by tile in a caller-given order (Section II-B: IntraFusion
        reorders GEMM tiles)
  * ring schedules and a message-passing ring simulator (Section III-A,
    Fig. 5; Section III-B, Fig. 6)
  * the performance models: Eq. 2-5 (InterDecom), Eq. 6-8 (IntraFusion and
    selection), Algorithm 1, and the calibration fits (Section IV-C,
    Section V)

Where the paper leaves a point open, the function states the reading it
takes. ``DOUBLE_SPLIT`` (a double ring whose chunk rows are split between
the directions in proportion to their rates) is not the paper's design,
which splits every chunk in halves; it is an extension of it. ``ALLTOALL``
is the comparison pattern of Section III-A (every rank pushes its chunk to
every other at once, two NUMA domains of n/2 ranks), AllGather only.

Parity status
  * GEMM parts, schedules, ring bandwidths, Eq. 2-8 identities: pinned by
    the not-gpu tests (brute force, integer-exact inputs, ring simulation,
    printed closed forms and Table I).
  * Calibrated constants (alpha/beta, T_comp/T_comm coefficients): the paper
    prints no values — parity unpinned; only the fitting procedure is pinned
    (recovery of planted parameters).
"""
from __future__ import annotations

import math
from typing import Sequence

import numpy as np

AG = "ag"
RS = "rs"
SINGLE = "single"
DOUBLE = "double"
DOUBLE_SPLIT = "double_split"   # double ring, chunk rows split in proportion to the two rates
ALLTOALL = "alltoall"           # direct pushes, two NUMA domains (AllGather only)

# --------------------------------------------------------------------------
# bf16 <-> fp64
# --------------------------------------------------------------------------


def bf16_to_f64(bits) -> np.ndarray:
    """Exact value of bf16 bit patterns (uint16) as fp64: a bf16 pattern is
    the upper half of an IEEE binary32 pattern."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f64_to_bf16_rne(x) -> np.ndarray:
    """Round fp64 values to bf16 (8 significant bits), ties to even, and
    return the bit patterns. Finite, normal-range values only."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                    # x = m * 2**e, 0.5 <= |m| < 1
    r = np.rint(m * 256.0) * np.ldexp(1.0, e - 8)   # rint: half to even
    r32 = r.astype(np.float32)            # exact: r has <= 8 significant bits
    return (np.ascontiguousarray(r32).view(np.uint32) >> 16).astype(np.uint16)


# --------------------------------------------------------------------------
# GEMM parts (textbook definitions)
# --------------------------------------------------------------------------


def gather(shards: Sequence[np.ndarray]) -> np.ndarray:
    """AllGather of row shards: rank q's shard becomes rows
    [q*M/n, (q+1)*M/n) of the gathered matrix (Section II-A)."""
    return np.vstack([np.asarray(s, dtype=np.float64) for s in shards])


def ag_gemm(shards: Sequence[np.ndarray], W: np.ndarray) -> np.ndarray:
    """AllGather+GEMM: C = gather(shards) @ B with B = W^T (W is N x K).
    Section II-A (Fig. 1): the column-parallel GEMM0 needs the full input."""
    A_g = gather(shards)
    return A_g @ np.asarray(W, dtype=np.float64).T


def gemm_rs(A: np.ndarray, W: np.ndarray, P_in: Sequence[np.ndarray], n: int) -> np.ndarray:
    """GEMM+ReduceScatter seen from one rank: P = A @ W^T, then every row
    chunk c (rows [c*M/n, (c+1)*M/n)) is summed with the incoming partial
    P_in[c] (Section II-A; Section III-B, ReduceScatter case)."""
    A = np.asarray(A, dtype=np.float64)
    P = A @ np.asarray(W, dtype=np.float64).T
    M = A.shape[0]
    rows = M // n
    out = np.empty_like(P)
    for c in range(n):
        out[c * rows:(c + 1) * rows] = P[c * rows:(c + 1) * rows] + np.asarray(P_in[c], dtype=np.float64)
    return out


def decomp_ag(shards: Sequence[np.ndarray], W: np.ndarray, d: int) -> np.ndarray:
    """InterDecom AllGather+GEMM with degree d (Section II-B, Fig. 2(c)):
    sub-operator j gathers row piece j (rows [j*M/(n d), (j+1)*M/(n d)) of
    every shard), multiplies it by B, and its rows land at their global
    positions."""
    n = len(shards)
    rows = np.asarray(shards[0]).shape[0]
    if rows % d:
        raise ValueError("shard rows must be divisible by d")
    piece = rows // d
    Wt = np.asarray(W, dtype=np.float64).T
    C = np.empty((n * rows, Wt.shape[1]), dtype=np.float64)
    for j in range(d):
        A_j = np.vstack([np.asarray(s, dtype=np.float64)[j * piece:(j + 1) * piece] for s in shards])
        C_j = A_j @ Wt
        for q in range(n):
            C[q * rows + j * piece:q * rows + (j + 1) * piece] = C_j[q * piece:(q + 1) * piece]
    return C


def decomp_rs(A: np.ndarray, W: np.ndarray, P_in: Sequence[np.ndarray], n: int, d: int) -> np.ndarray:
    """InterDecom GEMM+ReduceScatter with degree d: sub-operator j computes
    row piece j of every chunk and reduces it with piece j of the chunk's
    incoming partial."""
    A = np.asarray(A, dtype=np.float64)
    M = A.shape[0]
    rows = M // n
    if rows % d:
        raise ValueError("chunk rows must be divisible by d")
    piece = rows // d
    Wt = np.asarray(W, dtype=np.float64).T
    out = np.empty((M, Wt.shape[1]), dtype=np.float64)
    for j in range(d):
        idx = np.concatenate([np.arange(c * rows + j * piece, c * rows + (j + 1) * piece) for c in range(n)])
        P_j = A[idx] @ Wt
        for c in range(n):
            r0 = c * rows + j * piece
            out[r0:r0 + piece] = P_j[c * piece:(c + 1) * piece] + \
                np.asarray(P_in[c], dtype=np.float64)[j * piece:(j + 1) * piece]
    return out


def _tile_rows_cols(M, N, BM, BN, t):
    tm, tn = divmod(t, -(-N // BN))
    return (tm * BM, min(M, (tm + 1) * BM)), (tn * BN, min(N, (tn + 1) * BN))


def tile_ordered_ag(shards, W, order: Sequence[int], BM: int, BN: int) -> np.ndarray:
    """AllGather+GEMM computed one output tile at a time in the given order
    (tile t = row tile t // tilesN, column tile t % tilesN). IntraFusion only
    reorders tiles (Section II-B), so the result must not depend on order."""
    A_g = gather(shards)
    Wt = np.asarray(W, dtype=np.float64).T
    M, N = A_g.shape[0], Wt.shape[1]
    C = np.full((M, N), np.nan)
    for t in order:
        (r0, r1), (c0, c1) = _tile_rows_cols(M, N, BM, BN, t)
        C[r0:r1, c0:c1] = A_g[r0:r1] @ Wt[:, c0:c1]
    return C


def tile_ordered_rs(A, W, P_in, n, order: Sequence[int], BM: int, BN: int) -> np.ndarray:
    """GEMM+ReduceScatter computed tile by tile in the given order; each tile
    row is reduced with the incoming partial of the chunk that owns it."""
    A = np.asarray(A, dtype=np.float64)
    Wt = np.asarray(W, dtype=np.float64).T
    M, N = A.shape[0], Wt.shape[1]
    rows = M // n
    Pfull = np.vstack([np.asarray(p, dtype=np.float64) for p in P_in])
    assert Pfull.shape == (M, N)
    out = np.full((M, N), np.nan)
    for t in order:
        (r0, r1), (c0, c1) = _tile_rows_cols(M, N, BM, BN, t)
        out[r0:r1, c0:c1] = A[r0:r1] @ Wt[:, c0:c1] + Pfull[r0:r1, c0:c1]
    _ = rows
    return out


# --------------------------------------------------------------------------
# Ring schedules (Section III-A Fig. 5; Section III-B Fig. 6)
# --------------------------------------------------------------------------
# Readings: rank r owns chunk r (rows [r*M/n, (r+1)*M/n)); under the double
# ring, chunk c is split by rows into partition 2c (first half, carried by the
# backward ring, "even") and 2c+1 (second half, forward ring, "odd"); the
# forward ring sends r -> r+1, the backward ring r -> r-1; within a step the
# forward-ring partition is listed first. ReduceScatter follows the textbook
# ring order, which leaves the local chunk last (Section III-B).


def schedule(pattern: str, ring: str, n: int, r: int) -> list:
    """Order in which rank r processes chunks (single ring: chunk ids) or
    partitions (double ring: partition ids 2c+h)."""
    if n < 1 or not 0 <= r < n:
        raise ValueError("bad n / rank")
    out = []
    if pattern == AG and ring == SINGLE:
        # step s: the chunk that has travelled s hops on the forward ring
        for s in range(n):
            out.append((r - s) % n)
    elif pattern == AG and ring in (DOUBLE, DOUBLE_SPLIT):
        out += [2 * r, 2 * r + 1]            # local data first
        for s in range(1, n):
            out.append(2 * ((r - s) % n) + 1)   # odd, forward ring, from r-1
            out.append(2 * ((r + s) % n))       # even, backward ring, from r+1
    elif pattern == AG and ring == ALLTOALL:
        # Reading: the paper fixes no arrival order for the AlltoAll pattern.
        # The chunks of the own domain (direct fast links) come first, from
        # r+1 onward within the domain, then the other domain's in rank order
        # (they share the cross-domain link and land together).
        if n % 2:
            raise ValueError("AlltoAll needs an even n")
        h = n // 2
        d0 = (r // h) * h
        out.append(r)
        out += [d0 + (r - d0 + i) % h for i in range(1, h)]
        out += [(d0 + h) % n + i for i in range(h)]
    elif pattern == RS and ring == SINGLE:
        for s in range(n):
            out.append((r - 1 - s) % n)         # local chunk r comes last
    elif pattern == RS and ring in (DOUBLE, DOUBLE_SPLIT):
        for s in range(n):
            out.append(2 * ((r - 1 - s) % n) + 1)
            out.append(2 * ((r + 1 + s) % n))
    else:
        raise ValueError("bad pattern / ring")
    return out


def backward_rows(rows: int, fwd_Bps: float, bwd_Bps: float, ring: str) -> int:
    """Rows of a chunk (or of an InterDecom piece of one) that the backward
    ring carries. The paper's double ring splits every chunk in two halves
    (Section III-B). Reading for the rate-proportional extension
    (DOUBLE_SPLIT, both rates paced): the backward share is the rate share
    B_bwd / (B_fwd + B_bwd) of the rows, moved to a multiple of G rows
    (G = 128, the smaller tile's height, when the block has at least 1024
    rows, else 8) and kept within [lo, rows - lo], lo = min(G, rows // 2).
    Of the two nearest such multiples, the one whose step
    max(h / f_bwd, (rows - h) / f_fwd) is shorter wins; a tie goes to the
    smaller."""
    if ring != DOUBLE_SPLIT or not (fwd_Bps > 0 and bwd_Bps > 0):
        return rows // 2
    fb = bwd_Bps / (fwd_Bps + bwd_Bps)
    G = 128 if rows >= 1024 else 8
    lo = min(G, rows // 2)

    def clamp(h):
        return min(max(h, lo), rows - lo)

    down = clamp(math.floor(rows * fb / G) * G)
    up = clamp(math.ceil(rows * fb / G) * G)

    def step(h):
        return max(h / fb, (rows - h) / (1.0 - fb))

    return up if step(up) < step(down) else down


def partition_layout(pattern: str, ring: str, n: int, r: int, M: int, fwd_Bps: float = 0.0,
                     bwd_Bps: float = 0.0, sub: int = 1):
    """The partitions rank r moves and gates on: (order, row0, rows).

    Base partitions: chunk c (single ring, AlltoAll), or its backward part
    2c and forward part 2c + 1 (double ring, Section III-B), in the order of
    ``schedule``. With sub-chunk flags (sub >= 2) every base partition's
    cnt rows are cut into sub pieces of consecutive rows, piece t holding
    rows [cnt t // sub, cnt (t+1) // sub) of it; partition b * sub + t is
    piece t of base partition b and the pieces of a base partition follow
    one another in the order. Returns the order and, per partition id, its
    first global row and row count."""
    rows = M // n
    two = ring in (DOUBLE, DOUBLE_SPLIT)
    base = []
    for c in range(n):
        if two:
            h0 = backward_rows(rows, fwd_Bps, bwd_Bps, ring)
            base += [(c * rows, h0), (c * rows + h0, rows - h0)]
        else:
            base.append((c * rows, rows))
    row0, cnt = [], []
    for start, size in base:
        for t in range(sub):
            lo, hi = size * t // sub, size * (t + 1) // sub
            row0.append(start + lo)
            cnt.append(hi - lo)
    order = [b * sub + t for b in schedule(pattern, ring, n, r) for t in range(sub)]
    return order, row0, cnt


def simulate_ring_allgather(n: int, ring: str) -> list:
    """Message-passing simulation of a ring AllGather over n ranks.

    Every rank starts with its own chunk (or its two partitions). At each of
    the n-1 steps, every rank forwards on each ring the item it received in
    the previous step (its own item at the first step) to its ring
    neighbour. Returns, per rank, the list of item ids in the order the rank
    holds them (own items first, then arrivals step by step, forward ring
    before backward ring). Raises if a rank would forward an item it does
    not hold."""
    held = []
    last_fwd = []
    last_bwd = []
    for q in range(n):
        if ring == SINGLE:
            held.append([q])
            last_fwd.append(q)
            last_bwd.append(None)
        else:
            held.append([2 * q, 2 * q + 1])
            last_fwd.append(2 * q + 1)      # odd partitions travel forward
            last_bwd.append(2 * q)          # even partitions travel backward
    for _step in range(1, n):
        inbox_f = [None] * n
        inbox_b = [None] * n
        for q in range(n):
            item = last_fwd[q]
            if item not in held[q]:
                raise AssertionError("forwarding an item not held")
            inbox_f[(q + 1) % n] = item
            if ring == DOUBLE:
                item = last_bwd[q]
                if item not in held[q]:
                    raise AssertionError("forwarding an item not held")
                inbox_b[(q - 1) % n] = item
        for q in range(n):
            held[q].append(inbox_f[q])
            last_fwd[q] = inbox_f[q]
            if ring == DOUBLE:
                held[q].append(inbox_b[q])
                last_bwd[q] = inbox_b[q]
    return held


def ring_arrival_times(n: int, r: int, piece_bytes: float, hop_Bps: Sequence[float], d: int = 1) -> list:
    """Arrival times at rank r of a single-ring collective whose hops run at
    different rates (Section III-A: the cross-NUMA ring, where only some hops
    cross the slow link). Hop q carries rank q -> q+1 at hop_Bps[q].

    Reading: the ring has no global step barrier. Every hop carries one
    piece at a time, and a rank forwards a piece once it holds all of it
    (store and forward). So the piece rank q receives at step s is in
    flight once the sender q-1 holds it (its own piece at s = 1, else its
    arrival at step s-1) and the hop q-1 -> q has delivered the previous
    piece, and it lands piece_bytes / hop_Bps[q-1] later. With d
    sub-collectives (InterDecom), sub-collective j runs its n-1 steps after
    j-1's on the same hops. The same times hold for the incoming running
    sums of a ring ReduceScatter whose emulated ranks add instantly.

    Returns d*(n-1) times, sub-collective-major, step s = 1..n-1 within."""
    T = [piece_bytes / hop_Bps[q] for q in range(n)]
    link_free = [0.0] * n          # the hop into rank q delivered its last piece
    out = []
    for _j in range(d):
        held = [0.0] * n           # rank q holds the piece it forwards next
        for _s in range(1, n):
            now = [max(held[(q - 1) % n], link_free[q]) + T[(q - 1) % n] for q in range(n)]
            link_free = now
            held = now
            out.append(now[r])
    return out


def simulate_timed_ring_allgather(n: int, chunk_bytes: float, hop_Bps: Sequence[float]) -> list:
    """Event-driven simulation of a single-ring AllGather with per-hop
    rates: every rank queues its own chunk on its outgoing hop; a hop sends
    the pieces queued on it one at a time, first in first out; a rank that
    receives a chunk records it and queues it onward unless the next rank is
    the chunk's owner. Returns, per rank, the (time, chunk) arrivals in the
    order they happen."""
    import heapq
    queue = [[(0.0, q)] if n > 1 else [] for q in range(n)]   # (ready time, chunk) waiting on hop q
    busy_until = [0.0] * n
    arrivals = [[] for _ in range(n)]
    events = []                                # (time, seq, hop, chunk): hop delivers chunk
    seq = 0

    def start(q):
        nonlocal seq
        if not queue[q]:
            return
        ready, c = queue[q].pop(0)
        t = max(ready, busy_until[q]) + chunk_bytes / hop_Bps[q]
        busy_until[q] = t
        heapq.heappush(events, (t, seq, q, c))
        seq += 1

    sending = [False] * n                      # a delivery of hop q is pending
    for q in range(n):
        start(q)
        sending[q] = True
    while events:
        t, _, q, c = heapq.heappop(events)
        sending[q] = False
        dst = (q + 1) % n
        arrivals[dst].append((t, c))
        if (dst + 1) % n != c:
            queue[dst].append((t, c))
        for h in (q, dst):
            if not sending[h] and queue[h]:
                start(h)
                sending[h] = True
    return arrivals


def simulate_ring_reduce_scatter(partials: Sequence[np.ndarray], ring: str):
    """Message-passing simulation of a ring ReduceScatter.

    ``partials[q]`` is rank q's full (M x N) partial result. Chunk c (rows
    [c*M/n, (c+1)*M/n)) must end, fully reduced, at rank c. Single ring: the
    running sum of chunk c starts at rank c+1 and moves forward one rank per
    step, each rank adding its own rows. Double ring: the first row-half of
    each chunk travels on the backward ring (starting at rank c-1), the
    second half on the forward ring (starting at rank c+1).

    Returns (result, order): result[q] is what rank q holds for its own
    chunk; order[q] lists the items (chunk or partition ids) in the order
    rank q adds its contribution."""
    n = len(partials)
    P = [np.asarray(p, dtype=np.float64) for p in partials]
    M = P[0].shape[0]
    rows = M // n
    order = [[] for _ in range(n)]

    def rows_of(item):
        if ring == SINGLE:
            return slice(item * rows, (item + 1) * rows)
        c, h = divmod(item, 2)
        half = rows // 2
        return slice(c * rows + h * half, c * rows + (h + 1) * half)

    if ring == SINGLE:
        items = [(c, +1) for c in range(n)]
    else:
        items = [(2 * c + 1, +1) for c in range(n)] + [(2 * c, -1) for c in range(n)]
    result_parts = {}
    # running sums per item; item travelling direction d starts at owner+d
    running = {}
    pos = {}
    for item, dr in items:
        owner = item if ring == SINGLE else item // 2
        pos[item] = (owner + dr) % n
        running[item] = None
    for _step in range(n):
        for item, dr in items:
            q = pos[item]
            contrib = P[q][rows_of(item)]
            running[item] = contrib.copy() if running[item] is None else running[item] + contrib
            order[q].append(item)
            owner = item if ring == SINGLE else item // 2
            if q == owner:
                result_parts[item] = running[item]
            else:
                pos[item] = (q + dr) % n
    result = []
    for q in range(n):
        if ring == SINGLE:
            result.append(result_parts[q])
        else:
            result.append(np.vstack([result_parts[2 * q], result_parts[2 * q + 1]]))
    # per-rank order: within a step forward-ring item first (as listed)
    return result, order


# --------------------------------------------------------------------------
# Performance models (Sections IV and V)
# --------------------------------------------------------------------------


def comm_bytes_per_step(pattern: str, ring: str, M: int, N: int, K: int, n: int,
                        a_bytes: int = 2, p_bytes: int = 4, o_bytes: int = 2):
    """Bytes one ring link carries per step (Section III-A: each step moves a
    chunk of m/n on a single ring; the double ring splits it in two halves,
    one per ring). AllGather moves bf16 rows of A (M*K in total);
    ReduceScatter receives fp32 partial rows (M*N) and sends the bf16 sum
    onward on the opposite side of the link.

    Returns (incoming_bytes, outgoing_bytes) per link per step."""
    if pattern == AG:
        total_in = M * K * a_bytes
        total_out = 0
    else:
        total_in = M * N * p_bytes
        total_out = M * N * o_bytes
    div = n if ring == SINGLE else 2 * n
    return total_in / div, total_out / div


def t_comm(pattern: str, ring: str, M: int, N: int, K: int, n: int,
           fwd_Bps: float, bwd_Bps: float, tau: float = 0.0,
           a_bytes: int = 2, p_bytes: int = 4, o_bytes: int = 2) -> float:
    """Communication time of the ring collective: n-1 steps; per step the
    slowest active ring sets the pace (Section III-A). A per-step latency tau
    is added. Under ReduceScatter, the incoming and outgoing halves of a step
    use the two directions of the link and overlap."""
    if ring == ALLTOALL:
        # one round in which every flow runs at once (Section III-A)
        if pattern != AG or n % 2:
            raise ValueError("AlltoAll: AllGather over an even n only")
        c_in, _ = comm_bytes_per_step(pattern, SINGLE, M, N, K, n, a_bytes, p_bytes, o_bytes)
        h = n // 2
        intra = c_in / fwd_Bps if h > 1 else 0.0     # n = 2: no peer inside a domain
        return max(intra, h * h * c_in / bwd_Bps) + tau
    if ring == DOUBLE_SPLIT:
        # each step's chunk (m/n) is split between the rings in proportion to
        # their rates, so both rings finish the step together
        c_in, c_out = comm_bytes_per_step(pattern, SINGLE, M, N, K, n, a_bytes, p_bytes, o_bytes)
        f_bwd = bwd_Bps / (fwd_Bps + bwd_Bps)
        step = max(max(x * (1.0 - f_bwd) / fwd_Bps, x * f_bwd / bwd_Bps) for x in (c_in, c_out))
        return (n - 1) * (step + tau)
    b_in, b_out = comm_bytes_per_step(pattern, ring, M, N, K, n, a_bytes, p_bytes, o_bytes)
    rates = [fwd_Bps] if ring == SINGLE else [fwd_Bps, bwd_Bps]
    step = max(max(b_in / r, b_out / r) for r in rates)
    return (n - 1) * (step + tau)


def alltoall_link_time(n: int, chunk_bytes: float, intra_Bps: float, cross_Bps: float) -> float:
    """Brute-force time of an AlltoAll AllGather on two NUMA domains of n/2
    ranks (Section III-A): every rank sends its chunk to every other rank at
    once. A pair inside one domain has a link of its own at ``intra_Bps``;
    every flow from one domain to the other crosses that direction of the
    single cross-domain link (``cross_Bps``). Flows on one link share it
    equally, so the collective ends when the most loaded link has drained:
    max over links of bytes / rate."""
    h = n // 2
    load = {}
    for src in range(n):
        for dst in range(n):
            if src == dst:
                continue
            if src // h == dst // h:
                link = ("intra", src, dst)
            else:
                link = ("cross", src // h, dst // h)
            load[link] = load.get(link, 0.0) + chunk_bytes
    return max(b / (intra_Bps if k[0] == "intra" else cross_Bps) for k, b in load.items())


def effective_bandwidth(ring: str, n: int, B: float) -> float:
    """Effective AllGather bandwidth S / T_comm of a ring with equal link
    rates B, for a gathered size S (Section III-A)."""
    S = float(n * 1024 * 1024)
    t = t_comm(AG, ring, M=n * 1024, N=1, K=S / (n * 1024 * 2), n=n, fwd_Bps=B, bwd_Bps=B)
    return S / t


def t_comp(M: int, N: int, K: int, a_c: float, b_c: float) -> float:
    """Base computation time, linear in the GEMM's flop count 2*M*N*K
    (Section IV-B: base times are linear in workload parameters)."""
    return a_c + b_c * (2.0 * M * N * K)


def eta(d: float, alpha: float, beta: float) -> float:
    """Eq. 3: overhead factor, linear in the decomposition degree."""
    return alpha + beta * d


def t_decomp(Tc: float, Tm: float, d: int, alpha: float, beta: float) -> float:
    """Eq. 2: (d-1) overlapped stages of max(Tc, Tm)/d, each scaled by
    eta(d), plus the non-overlapped first/last portion Tc/d + Tm/d."""
    t_stage = max(Tc / d, Tm / d)
    return (d - 1) * t_stage * eta(d, alpha, beta) + Tc / d + Tm / d


def p2(x: float) -> int:
    """Nearest power of two, measured in log2 (ties go to the smaller power);
    values below 1 give 1."""
    if not x > 1.0:
        return 1
    lg = math.log2(x)
    k = math.floor(lg)
    frac = lg - k
    return 2 ** (k + 1) if frac > 0.5 else 2 ** k


def d_continuous(lam: float, alpha: float, beta: float, literal: bool = False) -> float:
    """Stationary point of Eq. 2 in d (the square root of Eq. 5).

    The paper's Eq. 5 uses 1/lambda, which is the minimiser when computation
    dominates (lambda >= 1). When communication dominates the same
    derivation gives lambda in its place; ``literal=False`` uses
    min(lambda, 1/lambda), ``literal=True`` the printed form."""
    if beta <= 0.0:
        return math.inf
    r = (1.0 / lam) if literal else min(lam, 1.0 / lam)
    num = 1.0 - alpha + r
    if num <= 0.0:
        return 0.0
    return math.sqrt(num / beta)


def d_candidate(lam: float, alpha: float, beta: float, d_max: int = 16,
                literal: bool = False) -> int:
    """Eq. 5: P2 of the stationary point, clamped to [1, d_max]."""
    x = d_continuous(lam, alpha, beta, literal)
    if math.isinf(x):
        return d_max
    d = p2(x)
    return max(1, min(d, d_max))


def d_final(Tc: float, Tm: float, alpha: float, beta: float, d_max: int = 16,
            literal: bool = False) -> int:
    """Eq. 4: keep the candidate only if it beats the sequential d = 1."""
    lam = Tc / Tm
    dc = d_candidate(lam, alpha, beta, d_max, literal)
    if t_decomp(Tc, Tm, dc, alpha, beta) < t_decomp(Tc, Tm, 1, alpha, beta):
        return dc
    return 1


def t_overhead_fusion(n_chunks: int, alpha_f: float, beta_f: float, m: float) -> float:
    """Eq. 8: (n_chunks - 1) synchronisation points, each alpha_f + beta_f*m."""
    return (n_chunks - 1) * (alpha_f + beta_f * m)


def t_fusion(comp_chunks: Sequence[float], comm_chunks: Sequence[float],
             alpha_f: float, beta_f: float, m: float) -> float:
    """Eq. 7: sum over chunks 2..n of max(comp, comm), plus the exposed
    computation of chunk 1, plus the Eq. 8 overhead."""
    n = len(comp_chunks)
    body = sum(max(comp_chunks[i], comm_chunks[i]) for i in range(1, n))
    return body + comp_chunks[0] + t_overhead_fusion(n, alpha_f, beta_f, m)


def fusion_m(pattern: str, M: int, N: int, K: int) -> float:
    """Communication volume m of Eq. 8: M*K for AllGather, M*N for
    ReduceScatter (elements)."""
    return float(M * K) if pattern == AG else float(M * N)


def select_strategy(t_fus: float, t_dec: float):
    """Eq. 6: the strategy with the lower predicted time, TA-IntraFusion only
    when strictly lower (a tie keeps ODP-InterDecom, as the selection
    algorithm of Section V-C states); returns it with that time."""
    s = "intra_fusion" if t_fus < t_dec else "inter_decom"
    return s, min(t_fus, t_dec)


def feasible_degree(chunk_rows: int, d_max: int) -> int:
    """Largest power of two d <= d_max whose sub-operators split a chunk's
    rows evenly (every sub-operator takes chunk_rows / d rows of each
    chunk)."""
    d = 1
    while d * 2 <= d_max and chunk_rows % (d * 2) == 0:
        d *= 2
    return d


def pick_strategy(pattern: str, ring: str, M: int, N: int, K: int, n: int,
                  fwd_Bps: float, bwd_Bps: float, tau: float,
                  a_c: float, b_c: float, alpha_d: float, beta_d: float,
                  alpha_f: float, beta_f: float, d_max: int = 16,
                  literal: bool = False) -> dict:
    """Strategy selection of Section V (Algorithm 1) from its models: the
    calibrated base times, ODP-InterDecom's predicted time at the degree of
    Eq. 4-5 (limited to degrees that split every chunk's rows evenly), and
    TA-IntraFusion's predicted time by Eq. 7-8 with one chunk of computation
    Tc/n against one ring step of communication; the lower one wins
    (Eq. 6)."""
    Tc = t_comp(M, N, K, a_c, b_c)
    Tm = t_comm(pattern, ring, M, N, K, n, fwd_Bps, bwd_Bps, tau)
    d_cap = feasible_degree(M // n, d_max)
    dc = d_candidate(Tc / Tm, alpha_d, beta_d, d_cap, literal)
    d_star = d_final(Tc, Tm, alpha_d, beta_d, d_cap, literal)
    Tdec = t_decomp(Tc, Tm, d_star, alpha_d, beta_d)
    step_comm = Tm / (n - 1) if n > 1 else 0.0
    comp_chunks = [Tc / n] * n
    comm_chunks = [0.0] + [step_comm] * (n - 1)
    Tfus = t_fusion(comp_chunks, comm_chunks, alpha_f, beta_f, fusion_m(pattern, M, N, K))
    s, T = select_strategy(Tfus, Tdec)
    return dict(strategy=s, t_star=T, d_star=d_star, d_cand=dc, lam=Tc / Tm, t_comp=Tc,
                t_comm=Tm, t_fusion=Tfus, t_decomp=Tdec, t_decomp1=t_decomp(Tc, Tm, 1, alpha_d, beta_d))


# --------------------------------------------------------------------------
# Calibration (Section IV-C: offline linear regression; Eq. 3 and Eq. 8)
# --------------------------------------------------------------------------


def fit_line(x: Sequence[float], y: Sequence[float]):
    """Ordinary least squares y ~ a + b*x; returns (a, b)."""
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    X = np.stack([np.ones_like(x), x], axis=1)
    coef, *_ = np.linalg.lstsq(X, y, rcond=None)
    return float(coef[0]), float(coef[1])


def eta_observed(t_meas: float, Tc: float, Tm: float, d: int) -> float:
    """Invert Eq. 2 for the overhead factor at one measured point (d >= 2)."""
    return (t_meas - (Tc + Tm) / d) * d / ((d - 1) * max(Tc, Tm))


def fusion_overhead_observed(t_meas: float, comp_chunks, comm_chunks) -> float:
    """Invert Eq. 7 for the per-synchronisation overhead of Eq. 8."""
    n = len(comp_chunks)
    base = sum(max(comp_chunks[i], comm_chunks[i]) for i in range(1, n)) + comp_chunks[0]
    return (t_meas - base) / (n - 1)


# --------------------------------------------------------------------------
# Table IV grid
# --------------------------------------------------------------------------

TABLE4 = dict(K=(4096, 8192, 16384), N=(2048, 4096, 8192, 16384), world=(4, 8),
              d=(2, 4, 8, 16), M=(2048, 4096, 8192, 12288, 16384, 32768),
              pattern=(AG, RS))


def table4_workloads(pattern=None, world=None) -> list:
    """Enumerate the workload grid of Table IV (every parameter but d)."""
    out = []
    for p in TABLE4["pattern"]:
        if pattern is not None and p != pattern:
            continue
        for w in TABLE4["world"]:
            if world is not None and w != world:
                continue
            for K in TABLE4["K"]:
                for N in TABLE4["N"]:
                    for M in TABLE4["M"]:
                        out.append((p, M, N, K, w))
    return out
