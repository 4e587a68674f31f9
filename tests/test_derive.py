"""The schedule algebra through the C ABI (include/mpipe_derive.h) against the oracle
(oracle/schedule.py): placement, collectives, events, typed edges, per-rank sequences,
event costs, makespan, bubbles and memory peaks, over skeleton mixes, rank and
micro-batch counts, every trainable mask and ByMicrobatch owners; plus the argument
checks.  Host only."""
import itertools
import random
import zlib

import numpy as np
import pytest

import paper_2607_03229_amd as mp
from oracle import schedule as S

SK = {"1f1b": mp.SK_1F1B, "gpipe": mp.SK_GPIPE, "transpose": mp.SK_TRANSPOSE}
COMM = {mp.COMM_GATHER: "Gather", mp.COMM_SCATTER: "Scatter", mp.COMM_SEND: "Send",
        mp.COMM_RECVGRAD: "RecvGrad"}
GROUP = {mp.GROUP_REPLICA: "ReplicaGroup", mp.GROUP_DATA: "DataGroup"}
EDGE = {mp.EDGE_ACTIVATION: "Activation", mp.EDGE_GRADIENT: "Gradient",
        mp.EDGE_TURNAROUND: "Turnaround", mp.EDGE_ACCUMULATE: "Accumulate",
        mp.EDGE_SEQUENCE: "Sequence"}
LAYOUT = {mp.LAYOUT_SHARDED: "Sharded", mp.LAYOUT_REPLICATED: "Replicated"}


def _event(row):
    kind, region, rank, mb, stage, comm, seam, group = (int(x) for x in row)
    if kind == mp.EV_FWD:
        return ("Fwd", region, rank, mb)
    if kind == mp.EV_BWD:
        return ("Bwd", region, rank, mb)
    if kind == mp.EV_COLL:
        return ("Coll", COMM[comm], seam, mb)
    if kind == mp.EV_DPREDUCE:
        return ("DpReduce", region, GROUP[group])
    if kind == mp.EV_LOSS:
        return ("Loss", mb)
    assert kind == mp.EV_STEP_BARRIER
    return ("StepBarrier",)


def _cut_for(sched, P):
    """Region sizes 2P+1, P, P+2, ... so that slabs are uneven; a Replicated region 3."""
    sizes = [3 if s == "transpose" else (2 * P + 1, P, P + 2, 2 * P)[j % 4]
             for j, s in enumerate(sched)]
    bounds = list(itertools.accumulate(sizes))
    return bounds[:-1], bounds[-1]


SCHEDULES = [
    ("1f1b",), ("gpipe",), ("transpose",),
    ("transpose", "1f1b"), ("transpose", "gpipe"),
    ("1f1b", "1f1b"), ("1f1b", "1f1b", "1f1b"), ("transpose", "1f1b", "1f1b"),
    ("gpipe", "gpipe"), ("1f1b", "1f1b", "1f1b", "1f1b"),
    # valid, but no order (a transposed sink, mixed Sharded skeletons)
    ("transpose", "1f1b", "transpose"), ("1f1b", "gpipe"), ("1f1b", "transpose"),
]


def _compare(sched, P, M, mask, owner, rng, timing):
    cut, L = _cut_for(sched, P)
    o = S.derive(cut, L, list(sched), list(mask), P, M, owner=owner)
    d = mp.Derived(cut, L, [SK[s] for s in sched], [int(t) for t in mask], P, M, owner=owner)
    k = len(sched)
    tag = (sched, P, M, mask, owner)
    # placement
    assert [LAYOUT[int(x)] for x in d.layout] == o["layout"], tag
    assert [bool(x) for x in d.runs_bwd] == o["runs_bwd"], tag
    assert list(d.owner) == o["owner"], tag
    for j in range(k):
        lay, (kind, own) = o["placement"][j]
        if lay == "Sharded":
            assert [(int(d.slab_lo[j, r]), int(d.slab_hi[j, r])) for r in range(P)] == \
                [own[r] for r in range(P)], tag
        else:
            assert (d.slab_lo[j] == -1).all() and (d.slab_hi[j] == -1).all(), tag
    # collectives
    seams = [((int(a), int(a) + 1), COMM[int(f)], None if int(b) == mp.COMM_NONE else COMM[int(b)])
             for a, f, b in d.seams]
    assert seams == o["seams"], tag
    assert [(int(j), GROUP[int(g)]) for j, g in d.reduces] == o["reduces"], tag
    # order
    assert d.has_order == (o["order"] is not None), tag
    if not d.has_order:
        assert d.events.shape[0] == 0 and all(len(n) == 0 for n in d.nodes)
        return
    ev = [_event(r) for r in d.events]
    assert len(set(ev)) == len(ev), tag
    assert set(ev) == set(o["order"]["events"]), tag
    for row, e in zip(d.events, ev):
        if e[0] in ("Fwd", "Bwd"):
            assert int(row[4]) == S.stage_index(e, P), tag
        else:
            assert int(row[4]) == -1, tag
    edges = [(ev[a], ev[b], EDGE[int(kd)]) for a, b, kd in d.edges]
    assert len(set(edges)) == len(edges), tag
    assert set(edges) == set(o["order"]["edges"]), tag
    for r in range(P):
        assert [ev[i] for i in d.nodes[r]] == o["order"]["nodes"][r], (tag, r)
    if not timing:
        return
    # event costs of the cost model
    fwd = [[rng.uniform(0.5, 4.0) for _ in range(M)] for _ in range(k)]
    bwd = [[rng.uniform(0.5, 8.0) for _ in range(M)] for _ in range(k)]
    seam_b = [[rng.uniform(0, 1e3) for _ in range(M)] for _ in range(k - 1)]
    red_b = [rng.uniform(0, 1e4) for _ in range(k)]
    alpha, beta, loss = 0.05, 1e-4, 0.3
    oc = S.event_costs(o, cut, L, fwd, bwd, seam_b, red_b, alpha, beta, loss)
    cc = d.event_costs(fwd, bwd, np.array(seam_b).reshape(k - 1, M), red_b, alpha, beta, loss)
    np.testing.assert_allclose(cc, [oc[e] for e in ev], rtol=1e-14, atol=0)
    # makespan on independent random costs keyed by event identity
    cost = {e: rng.uniform(0.0, 3.0) for e in o["order"]["events"]}
    T, bub, start, fin = d.makespan([cost[e] for e in ev])
    oT, obub, ostart, ofin = S.simulate(o["order"], cost)
    assert T == pytest.approx(oT, rel=1e-12), tag
    np.testing.assert_allclose(bub, [obub[r] for r in range(P)], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(fin, [ofin[e] for e in ev], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(start, [ostart[e] for e in ev], rtol=1e-12, atol=1e-12)
    # memory read-out
    act = {e: rng.uniform(1.0, 100.0) for e in ev if e[0] == "Fwd"}
    peak = d.memory_peak([act.get(e, 0.0) for e in ev])
    opeak = S.memory_peak(o, act)
    np.testing.assert_allclose(peak, [opeak[r] for r in range(P)], rtol=1e-12)


@pytest.mark.parametrize("sched", SCHEDULES, ids=lambda s: "-".join(s))
def test_derive_matches_oracle(sched):
    rng = random.Random(zlib.crc32("-".join(sched).encode()))
    k = len(sched)
    masks = list(itertools.product([False, True], repeat=k))
    n = 0
    for P in (1, 2, 3, 4):
        for M in (1, 2, 3, 4, 8):
            for mi, mask in enumerate(masks):
                owner = None if (mi + M) % 2 else [rng.randrange(P) for _ in range(M)]
                timing = mi in (0, len(masks) - 1) or mi == (P + M) % len(masks)
                _compare(sched, P, M, mask, owner, rng, timing)
                n += 1
    assert n == 20 * len(masks)


def test_mpipe_shape_at_paper_scale():
    """<transpose, 1f1b> at the scale of the paper's runs: 16 ranks, 64 micro-batches,
    a 32-layer encoder and a 61-layer backbone; one order, costs and makespan."""
    P, M = 16, 64
    rng = random.Random(3)
    owner = [rng.randrange(P) for _ in range(M)]
    sched = ["transpose", "1f1b"]
    o = S.derive([32], 93, sched, [True, True], P, M, owner=owner)
    d = mp.Derived([32], 93, [SK[s] for s in sched], [1, 1], P, M, owner=owner)
    ev = [_event(r) for r in d.events]
    assert set(ev) == set(o["order"]["events"])
    cost = {e: rng.uniform(0.1, 1.0) for e in ev}
    T, _, _, _ = d.makespan([cost[e] for e in ev])
    oT, _, _, _ = S.simulate(o["order"], cost)
    assert T == pytest.approx(oT, rel=1e-12)


def test_transposed_encoder_spill_special_cases():
    """With uniform backbone stages and free collectives: encoder work of zero cost
    leaves the 1F1B makespan (M + P - 1)(f + b); encoder work placed on rank 0, which
    has no warmup slack, adds its whole forward and backward to the step."""
    P, M, f, b = 4, 8, 1.0, 2.0
    sched = [SK["transpose"], SK["1f1b"]]
    for e_f, want_extra in [(0.0, 0.0), (0.75, None)]:
        owner = [0] * M
        d = mp.Derived([3], 3 + P, sched, [1, 1], P, M, owner=owner)
        fwd = [[e_f] * M, [f * P] * M]
        bwd = [[2 * e_f] * M, [b * P] * M]
        c = d.event_costs(fwd, bwd, np.zeros((1, M)), [0.0, 0.0], 0.0, 0.0, 0.0)
        T, bub, _, _ = d.makespan(c)
        base = (M + P - 1) * (f + b)
        if want_extra == 0.0:
            assert T == pytest.approx(base)
        else:
            assert T == pytest.approx(base + M * e_f + M * 2 * e_f)
            assert bub[0] == pytest.approx((P - 1) * (f + b))


# ---------------------------------------------------------------------------
# argument checks
# ---------------------------------------------------------------------------

def test_schedule_valid_through_the_abi():
    assert mp.schedule_valid([4], 8, [SK["transpose"], SK["1f1b"]])[0]
    assert mp.schedule_valid([2, 6], 8, [SK["transpose"], SK["1f1b"], SK["transpose"]])[0]
    ok, why = mp.schedule_valid([4], 8, [SK["transpose"], SK["transpose"]])
    assert not ok and "normal form" in why
    for cut, L, sched in [([0], 8, [0, 0]), ([8], 8, [0, 0]), ([5, 3], 8, [0, 0, 0]),
                          ([4], 8, [0, 7]), ([], 0, [0])]:
        assert not mp.schedule_valid(cut, L, sched)[0]


def test_derive_rejects_bad_arguments():
    with pytest.raises(mp.MpipeError, match="normal form"):
        mp.Derived([4], 8, [2, 2], [1, 1], 2, 2)
    with pytest.raises(mp.MpipeError, match="one layer per rank"):
        mp.Derived([2], 8, [0, 0], [1, 1], 4, 4)
    with pytest.raises(mp.MpipeError, match="owner"):
        mp.Derived([4], 8, [2, 0], [1, 1], 2, 2, owner=[0, 2])
    with pytest.raises(mp.MpipeError):
        mp.Derived([4], 8, [2, 0], [1, 1], 0, 2)
    with pytest.raises(mp.MpipeError):
        mp.Derived([4], 8, [2, 0], [1, 1], 2, 0)


def test_no_order_calls_are_unsupported():
    d = mp.Derived([2, 6], 8, [2, 0, 2], [1, 1, 1], 2, 4)
    assert not d.has_order
    with pytest.raises(mp.MpipeError, match="UNSUPPORTED"):
        d.makespan([])
    with pytest.raises(mp.MpipeError, match="UNSUPPORTED"):
        d.memory_peak([])
    d = mp.Derived([4], 8, [0, 0], [1, 1], 2, 3)   # interleaved with M % P != 0
    assert not d.has_order
    L = mp.load()
    assert L.mpipe_derived_nodes(d._h, 2, None, 0) == -1   # rank out of range


def test_costs_must_be_finite_and_nonnegative():
    d = mp.Derived([3], 7, [2, 0], [1, 1], 2, 2)
    n = d.events.shape[0]
    with pytest.raises(mp.MpipeError, match="finite"):
        d.makespan([-1.0] + [0.0] * (n - 1))
    with pytest.raises(mp.MpipeError, match="finite"):
        d.makespan([float("nan")] + [0.0] * (n - 1))
    with pytest.raises(mp.MpipeError, match="finite"):
        d.event_costs([[1, 1], [1, -1]], [[1, 1], [1, 1]], [[0, 0]], [0, 0], 0, 0, 0)
    with pytest.raises(mp.MpipeError, match="finite"):
        d.memory_peak([float("inf")] * n)
