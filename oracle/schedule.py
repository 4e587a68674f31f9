"""Oracle of the schedule algebra -- TEST INFRASTRUCTURE ONLY.

Only ``tests/`` may import this module; the library never loads it.  Plain
Python, written from the paper's Sec. 4.1 (the algebra, Table 2, Lemma 1, the
instantiation of <transpose, 1f1b>, the VPP-3 derivation) and Sec. 4.3 (the
cost model, makespan and bubble).  Indices are 0-based: region j here is the
paper's region j + 1, micro-batch m is its m + 1; ranks are 0..P-1 as in the
paper.

Events are tuples in the paper's notation:
    ("Fwd", j, r, m)  ("Bwd", j, r, m)  ("Coll", comm, s, m)
    ("DpReduce", j, group)  ("Loss", m)  ("StepBarrier",)
where s is the seam between regions s and s + 1.  Edges are (src, dst, kind)
with kind in EDGE_KINDS.

Where the paper leaves a choice open this module takes these readings:
  * ByLayer splits a region of n layers into P contiguous slabs whose
    boundaries are lo + floor(r n / P);
  * inside a Sharded region the forward chain of a micro-batch passes ranks
    0..P-1 and the backward chain P-1..0, with no Coll event between ranks of
    one region (only seams are collectives);
  * each Fwd has an Activation edge to the Bwd of the same stage and
    micro-batch (the stored activation);
  * a reverse seam collective hands on to the next backward by a Gradient edge;
  * with no backward anywhere, each Loss has a Sequence edge to StepBarrier;
  * the Loss of m runs on the rank of the last forward stage (rank P-1 under a
    Sharded last region, the owner of m when the only region is Replicated);
  * a rank's sequence: a Replicated first region's owned forwards first, the
    Sharded regions' events in the skeleton's order, the Replicated region's
    owned backwards last; 1f1b is the one-forward-one-backward flush schedule
    with P-1-r warmup forwards, several 1f1b regions use the interleaved
    schedule (warmup 2(P-1-r) + (S-1)P virtual micro-batches, every one of them
    when M == P), gpipe runs all forwards region by region, then all backwards
    in reverse region order;
  * the order is only built when the Sharded regions share one skeleton, a
    Replicated region (if any) is the first one, and the interleaved schedule
    has M a multiple of P; otherwise ``order`` is None.
"""
from __future__ import annotations

import heapq
from typing import Dict, List, Optional, Sequence, Tuple

SKELETONS = ("1f1b", "gpipe", "transpose")
EDGE_KINDS = ("Activation", "Gradient", "Turnaround", "Accumulate", "Sequence")

# Table 2: (layout_j, layout_{j+1}) -> (forward collective, reverse collective)
SEAM_TABLE = {
    ("Replicated", "Sharded"): ("Gather", "Scatter"),
    ("Sharded", "Sharded"): ("Send", "RecvGrad"),
    ("Sharded", "Replicated"): ("Scatter", "Gather"),
}


def layout(skeleton: str) -> str:
    """transpose is the Replicated skeleton; 1f1b and gpipe are Sharded (Sec. 4.1)."""
    return "Replicated" if skeleton == "transpose" else "Sharded"


def valid(cut: Sequence[int], n_layers: int, schedule: Sequence[str]) -> bool:
    """The cut tiles the layers and no two adjacent regions are Replicated (normal form)."""
    k = len(schedule)
    if k < 1 or len(cut) != k - 1 or any(s not in SKELETONS for s in schedule):
        return False
    bounds = [0] + list(cut) + [n_layers]
    if any(bounds[i] >= bounds[i + 1] for i in range(k)):
        return False
    return not any(layout(schedule[i]) == "Replicated" == layout(schedule[i + 1])
                   for i in range(k - 1))


def gates(trainable: Sequence[bool]):
    """Lemma 1 for regions in input-to-loss order.

    sends[j]:    region j sends its input gradient upstream iff some i < j is trainable;
    receives[j]: region j receives a gradient (runs any backward) iff some i <= j is;
    reduces[j]:  region j reduces weight gradients iff it is trainable."""
    k = len(trainable)
    sends = [any(trainable[i] for i in range(j)) for j in range(k)]
    receives = [any(trainable[i] for i in range(j + 1)) for j in range(k)]
    reduces = [bool(t) for t in trainable]
    return sends, receives, reduces


def _slabs(lo: int, hi: int, P: int) -> Dict[int, Tuple[int, int]]:
    n = hi - lo
    return {r: (lo + r * n // P, lo + (r + 1) * n // P) for r in range(P)}


def derive(cut, n_layers, schedule, trainable, P, M, owner=None) -> dict:
    """placement x collectives x order for a valid (cut, schedule) (Sec. 4.1)."""
    assert valid(cut, n_layers, schedule), "derive takes a valid schedule"
    k = len(schedule)
    bounds = [0] + list(cut) + [n_layers]
    owner = [m % P for m in range(M)] if owner is None else list(owner)
    lay = [layout(s) for s in schedule]
    sends, receives, reduces = gates(trainable)

    placement = []
    for j in range(k):
        if lay[j] == "Replicated":
            placement.append(("Replicated", ("ByMicrobatch", {m: owner[m] for m in range(M)})))
        else:
            placement.append(("Sharded", ("ByLayer", _slabs(bounds[j], bounds[j + 1], P))))
    seams = []
    for j in range(k - 1):
        fwd, bwd = SEAM_TABLE[(lay[j], lay[j + 1])]
        # the reverse collective carries region j+1's input gradient: it fires iff j+1 sends
        seams.append(((j, j + 1), fwd, bwd if sends[j + 1] else None))
    reduce_list = [(j, "ReplicaGroup" if lay[j] == "Replicated" else "DataGroup")
                   for j in range(k) if reduces[j]]
    out = {"layout": lay, "placement": placement, "seams": seams, "reduces": reduce_list,
           "runs_bwd": receives, "sends": sends, "owner": owner, "order": None}

    sharded = [j for j in range(k) if lay[j] == "Sharded"]
    sk = {schedule[j] for j in sharded}
    if any(lay[j] == "Replicated" for j in range(1, k)) or len(sk) > 1:
        return out
    if len(sharded) > 1 and "1f1b" in sk and M % P:
        return out

    def ranks(j, m):   # the ranks region j's forward of m passes, in order
        return [owner[m]] if lay[j] == "Replicated" else list(range(P))

    events, edges = [], []
    for m in range(M):
        prev = None
        for j in range(k):
            for r in ranks(j, m):
                e = ("Fwd", j, r, m)
                events.append(e)
                if prev is not None:
                    edges.append((prev, e, "Activation"))
                prev = e
            if j + 1 < k:
                c = ("Coll", seams[j][1], j, m)
                events.append(c)
                edges.append((prev, c, "Activation"))
                prev = c
        events.append(("Loss", m))
        edges.append((prev, ("Loss", m), "Activation"))
        prev, kind = ("Loss", m), "Turnaround"
        for j in reversed(range(k)):
            if not receives[j]:
                break
            for r in reversed(ranks(j, m)):
                e = ("Bwd", j, r, m)
                events.append(e)
                edges.append((prev, e, kind))
                edges.append((("Fwd", j, r, m), e, "Activation"))
                prev, kind = e, "Gradient"
            if sends[j]:
                c = ("Coll", seams[j - 1][2], j - 1, m)
                events.append(c)
                edges.append((prev, c, "Gradient"))
                prev = c
    for j, g in reduce_list:
        events.append(("DpReduce", j, g))
    events.append(("StepBarrier",))
    for j, g in reduce_list:
        for m in range(M):
            for r in ranks(j, m):
                edges.append((("Bwd", j, r, m), ("DpReduce", j, g), "Accumulate"))
        edges.append((("DpReduce", j, g), ("StepBarrier",), "Sequence"))
    if not receives[k - 1]:
        for m in range(M):
            edges.append((("Loss", m), ("StepBarrier",), "Sequence"))

    loss_rank = (lambda m: P - 1) if lay[-1] == "Sharded" else (lambda m: owner[m])
    bwd_events = set(e for e in events if e[0] == "Bwd")
    nodes = {}
    for r in range(P):
        seq: List[tuple] = []

        def fwd(j, m):
            seq.append(("Fwd", j, r, m))
            if j == k - 1 and loss_rank(m) == r:
                seq.append(("Loss", m))

        def bwd(j, m):
            if ("Bwd", j, r, m) in bwd_events:
                seq.append(("Bwd", j, r, m))

        mine = [m for m in range(M) if owner[m] == r]
        if lay[0] == "Replicated":
            for m in mine:
                fwd(0, m)
        S = len(sharded)
        if S == 0 or not receives[k - 1]:
            for m in range(M):
                for j in sharded:
                    fwd(j, m)
        elif "gpipe" in sk:
            for j in sharded:
                for m in range(M):
                    fwd(j, m)
            for j in reversed(sharded):
                for m in range(M):
                    bwd(j, m)
        elif S == 1:
            j = sharded[0]
            warm = min(P - 1 - r, M)
            for m in range(warm):
                fwd(j, m)
            for i in range(M - warm):
                fwd(j, warm + i)
                bwd(j, i)
            for i in range(M - warm, M):
                bwd(j, i)
        else:
            # virtual micro-batches: groups of P micro-batches, each group passing every chunk
            f_list = [(sharded[c], g * P + i) for g in range(M // P)
                      for c in range(S) for i in range(P)]
            b_list = [(sharded[S - 1 - c], g * P + i) for g in range(M // P)
                      for c in range(S) for i in range(P)]
            total = len(f_list)
            warm = total if M == P else min(2 * (P - 1 - r) + (S - 1) * P, total)
            for q in range(warm):
                fwd(*f_list[q])
            for q in range(total - warm):
                fwd(*f_list[warm + q])
                bwd(*b_list[q])
            for q in range(total - warm, total):
                bwd(*b_list[q])
        if lay[0] == "Replicated" and receives[k - 1]:
            for m in mine:
                bwd(0, m)
        nodes[r] = seq
    out["order"] = {"events": events, "edges": edges, "nodes": nodes}
    return out


def stage_index(event, P: int) -> int:
    """stage = rank + region * P for Fwd/Bwd (0-based form of the paper's numbering)."""
    return event[2] + event[1] * P


def event_costs(d: dict, cut, n_layers, fwd_cost, bwd_cost, seam_bytes, reduce_bytes,
                alpha, beta, loss_cost) -> Dict[tuple, float]:
    """Sec. 4.3: a compute event costs its slab's share of the region's roofline time,
    a collective or reduce alpha + beta * n, a Loss loss_cost, StepBarrier nothing."""
    bounds = [0] + list(cut) + [n_layers]
    out = {}
    for e in d["order"]["events"]:
        if e[0] in ("Fwd", "Bwd"):
            _, j, r, m = e
            c = (fwd_cost if e[0] == "Fwd" else bwd_cost)[j][m]
            if d["layout"][j] == "Sharded":
                lo, hi = d["placement"][j][1][1][r]
                c = c * (hi - lo) / (bounds[j + 1] - bounds[j])
            out[e] = c
        elif e[0] == "Coll":
            out[e] = alpha + beta * seam_bytes[e[2]][e[3]]
        elif e[0] == "DpReduce":
            out[e] = alpha + beta * reduce_bytes[e[1]]
        elif e[0] == "Loss":
            out[e] = loss_cost
        else:
            out[e] = 0.0
    return out


def simulate(order: dict, cost: Dict[tuple, float]):
    """Discrete-event simulation of one step: a rank runs its nodes(r) one at a time,
    each as soon as the rank is free and every predecessor has finished; collective
    events run as soon as their predecessors have finished.  Returns (T, bubble, start,
    finish) with bubble[r] = T - sum of the costs in nodes(r) (Sec. 4.3)."""
    events, nodes = order["events"], order["nodes"]
    preds: Dict[tuple, List[tuple]] = {e: [] for e in events}
    for a, b, _ in order["edges"]:
        preds[b].append(a)
    rank_of = {e: r for r, seq in nodes.items() for e in seq}
    nxt = {r: 0 for r in nodes}
    busy = {r: False for r in nodes}
    done: Dict[tuple, float] = {}
    start: Dict[tuple, float] = {}
    waiting = list(events)
    running: List[Tuple[float, int, tuple]] = []
    t, tick = 0.0, 0
    while waiting or running:
        launched = True
        while launched:   # start everything that can start at time t
            launched = False
            rest = []
            for e in waiting:
                ready = all(p in done for p in preds[e])
                r = rank_of.get(e)
                if ready and r is not None:
                    ready = not busy[r] and nodes[r][nxt[r]] == e
                if ready:
                    start[e] = t
                    heapq.heappush(running, (t + cost[e], tick, e))
                    tick += 1
                    if r is not None:
                        busy[r] = True
                    launched = True
                else:
                    rest.append(e)
            waiting = rest
        if not running:
            raise RuntimeError("deadlock: events wait on each other")
        t, _, e = heapq.heappop(running)
        done[e] = t
        r = rank_of.get(e)
        if r is not None:
            busy[r] = False
            nxt[r] += 1
    T = max(done.values()) if done else 0.0
    bubble = {r: T - sum(cost[e] for e in seq) for r, seq in nodes.items()}
    return T, bubble, start, done


def memory_peak(d: dict, act_bytes: Dict[tuple, float]) -> Dict[int, float]:
    """Memory read off placement and order (Sec. 4.1): on rank r, in nodes(r) order, a
    Fwd's bytes are live from the Fwd until the Bwd of the same stage and micro-batch;
    a Fwd whose region runs no backward holds them only while it runs."""
    order = d["order"]
    bwds = set(e for e in order["events"] if e[0] == "Bwd")
    peak = {}
    for r, seq in order["nodes"].items():
        live, top = 0.0, 0.0
        for e in seq:
            if e[0] == "Fwd":
                live += act_bytes[e]
                top = max(top, live)
                if ("Bwd",) + e[1:] not in bwds:
                    live -= act_bytes[e]
            elif e[0] == "Bwd":
                live -= act_bytes[("Fwd",) + e[1:]]
        peak[r] = top
    return peak
