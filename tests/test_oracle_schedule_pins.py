"""Pins of the schedule-algebra oracle (oracle/schedule.py) against what the paper and
textbook results fix, not against the oracle itself:

  * validity: the three schedules Sec. 4.1 classifies;
  * the <transpose, 1f1b> instantiation and its frozen footprint, as printed
    (tests/golden/derive_instantiation.txt);
  * the VPP-3 derivation: two Send/RecvGrad seams, no gradient sent by region 1,
    one slab of every region per rank, stage = rank + region * P;
  * Lemma 1 against autograd: which backward nodes torch runs for every trainable
    mask of a chain of regions;
  * Corollary 1: the backward footprint of one cut is the same under every schedule;
  * makespans in closed form: (M + P - 1)(f + b) for 1F1B and GPipe with uniform
    stages, (M S + P - 1)(f + b) for interleaved 1F1B with S chunks of cost f, b;
  * memory in closed form: 1F1B keeps min(P - r, M) activations on rank r, GPipe
    keeps M, interleaved 1F1B min(warmup + 1, M S); the transposed encoder keeps every
    owned micro-batch's activation across the step when trainable and none when frozen;
  * Table 2 row by row, on a schedule that has both cross-layout seams;
  * the cost model's shares: the slab costs of a Sharded region sum to the region's.

MPIPE_SCHEDULE_ORACLE may name another copy of the oracle source (the planted-mistake
meta-test uses it)."""
import importlib.util
import itertools
import os
import random

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLDEN = os.path.join(ROOT, "tests", "golden", "derive_instantiation.txt")


def _load_oracle():
    path = os.environ.get("MPIPE_SCHEDULE_ORACLE", os.path.join(ROOT, "oracle", "schedule.py"))
    spec = importlib.util.spec_from_file_location("schedule_oracle_under_test", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


S = _load_oracle()


# ---------------------------------------------------------------------------
# validity (Sec. 4.1: the examples it classifies)
# ---------------------------------------------------------------------------

def test_validity_examples():
    assert S.valid([4], 8, ["transpose", "1f1b"])
    assert S.valid([2, 6], 8, ["transpose", "1f1b", "transpose"])
    assert not S.valid([4], 8, ["transpose", "transpose"])
    assert S.valid([], 8, ["transpose"])          # what <transpose, transpose> reduces to
    assert S.valid([3, 5], 8, ["1f1b", "1f1b", "1f1b"])   # VPP-3


def test_validity_cut_must_tile():
    assert not S.valid([0], 8, ["transpose", "1f1b"])
    assert not S.valid([8], 8, ["transpose", "1f1b"])
    assert not S.valid([5, 3], 8, ["1f1b", "1f1b", "1f1b"])
    assert not S.valid([4, 4], 8, ["1f1b", "1f1b", "1f1b"])
    assert not S.valid([4], 8, ["1f1b"])          # one boundary too many
    assert not S.valid([4], 8, ["wave", "1f1b"])  # not a skeleton of the algebra


# ---------------------------------------------------------------------------
# the <transpose, 1f1b> instantiation, as printed
# ---------------------------------------------------------------------------

def _parse_event(tok):
    t = tok.split()
    if t[0] in ("Fwd", "Bwd"):
        return (t[0], int(t[1]), 0, 0)
    if t[0] == "Coll":
        return ("Coll", t[1], int(t[2]), 0)
    if t[0] == "DpReduce":
        return ("DpReduce", int(t[1]), t[2])
    if t[0] == "Loss":
        return ("Loss", 0)
    assert t == ["StepBarrier"]
    return ("StepBarrier",)


def _golden():
    cases, cur = {}, None
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        if line.startswith("["):
            cur = cases.setdefault(line.strip("[]"), {"placement": [], "seams": [],
                                                      "reduces": [], "edges": set()})
            continue
        head, _, rest = line.partition(" ")
        if head == "placement":
            j, lay, own = rest.split()
            cur["placement"].append((int(j), lay, own))
        elif head == "seam":
            a, b, f, r = rest.split()
            cur["seams"].append(((int(a), int(b)), f, None if r == "-" else r))
        elif head == "reduce":
            j, g = rest.split()
            cur["reduces"].append((int(j), g))
        elif head == "edge":
            kind, body = rest.split(" ", 1)
            src, dst = body.split("|")
            dst = dst.replace("reading", "")
            cur["edges"].add((_parse_event(src.strip()), _parse_event(dst.strip()), kind))
    return cases


@pytest.mark.parametrize("case", ["trainable", "frozen"])
def test_instantiation_matches_the_paper(case):
    g = _golden()[case]
    d = S.derive([4], 8, ["transpose", "1f1b"], [case == "trainable", True], P=1, M=1)
    assert [(j, lay, own[0]) for j, (lay, own) in enumerate(d["placement"])] == g["placement"]
    assert d["seams"] == g["seams"]
    assert d["reduces"] == g["reduces"]
    assert set(d["order"]["edges"]) == g["edges"]
    ends = {e for a, b, _ in g["edges"] for e in (a, b)}
    assert set(d["order"]["events"]) == ends
    if case == "frozen":   # freezing deletes every optional element
        assert not any(e[0] == "Bwd" and e[1] == 0 for e in d["order"]["events"])
        assert not any(e[0] == "Coll" and e[1] == "Scatter" for e in d["order"]["events"])


def test_instantiation_forward_order_unchanged_by_freezing():
    """Freezing leaves the placement and the forward order unchanged."""
    P, M = 4, 8
    a = S.derive([4], 8, ["transpose", "1f1b"], [True, True], P, M)
    b = S.derive([4], 8, ["transpose", "1f1b"], [False, True], P, M)
    fw = lambda d: [(x, y, k) for x, y, k in d["order"]["edges"]
                    if k == "Activation" and y[0] != "Bwd"]
    assert a["placement"] == b["placement"]
    assert fw(a) == fw(b)
    for r in range(P):
        fa = [e for e in a["order"]["nodes"][r] if e[0] in ("Fwd", "Loss")]
        fb = [e for e in b["order"]["nodes"][r] if e[0] in ("Fwd", "Loss")]
        assert fa == fb


def test_transpose_places_encoder_in_warmup_and_cooldown():
    """Each rank runs the encoder forwards its ByMicrobatch owner gives it before any
    backbone event, and their backwards after every backbone event (Sec. 4.1, 4.2)."""
    P, M = 4, 8
    owner = [3, 2, 1, 0, 3, 3, 1, 2]
    d = S.derive([4], 8, ["transpose", "1f1b"], [True, True], P, M, owner=owner)
    for r in range(P):
        seq = d["order"]["nodes"][r]
        mine = [m for m in range(M) if owner[m] == r]
        n = len(mine)
        assert seq[:n] == [("Fwd", 0, r, m) for m in mine]
        assert seq[len(seq) - n:] == [("Bwd", 0, r, m) for m in mine]
        assert all(e[1] == 1 or e[0] == "Loss" for e in seq[n:len(seq) - n])


# ---------------------------------------------------------------------------
# VPP-3 (Sec. 4.1, "A second derivation")
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("mask", list(itertools.product([False, True], repeat=3)))
def test_vpp3_derivation(mask):
    P, M = 4, 8
    d = S.derive([4, 8], 12, ["1f1b"] * 3, list(mask), P, M)
    assert d["layout"] == ["Sharded"] * 3
    assert [own[0] for _, own in d["placement"]] == ["ByLayer"] * 3
    fires = [any(mask[:1]), any(mask[:2])]
    assert d["seams"] == [((0, 1), "Send", "RecvGrad" if fires[0] else None),
                          ((1, 2), "Send", "RecvGrad" if fires[1] else None)]
    ev = d["order"]["events"]
    # region 0 sends no input gradient: no reverse collective before it
    assert not any(e[0] == "Coll" and e[2] < 0 for e in ev)
    # every rank owns one slab of each region
    for j in range(3):
        slabs = d["placement"][j][1][1]
        assert sorted(slabs) == list(range(P))
        assert all(hi - lo == 1 for lo, hi in slabs.values())
    # stage = rank + region * P enumerates the 3P virtual stages once each
    stages = {(e[1], e[2]): S.stage_index(e, P) for e in ev if e[0] == "Fwd"}
    assert sorted(stages.values()) == list(range(3 * P))


# ---------------------------------------------------------------------------
# Lemma 1 against autograd, Corollary 1
# ---------------------------------------------------------------------------

def _autograd_footprint(mask):
    """Run a chain of k regions (one weight each, requires_grad = trainable) and record
    which region outputs and inputs receive a gradient and which weights get one."""
    import torch
    k = len(mask)
    ws = [torch.tensor([1.5 + j], dtype=torch.float64, requires_grad=bool(t))
          for j, t in enumerate(mask)]
    h = torch.tensor([0.5, -1.0], dtype=torch.float64)
    got_out, got_in = [False] * k, [False] * k
    hs = []
    for j in range(k):
        if h.requires_grad:
            def mark_in(g, j=j):
                got_in[j] = True
            h.register_hook(mark_in)
        h = torch.tanh(h * ws[j])
        if h.requires_grad:
            def mark_out(g, j=j):
                got_out[j] = True
            h.register_hook(mark_out)
        hs.append(h)
    loss = (h * h).sum()
    if loss.requires_grad:
        loss.backward()
    reduced = [w.grad is not None for w in ws]
    return got_in, got_out, reduced


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_lemma1_matches_autograd(k):
    for mask in itertools.product([False, True], repeat=k):
        sends, receives, reduces = S.gates(list(mask))
        got_in, got_out, reduced = _autograd_footprint(mask)
        assert sends == got_in, mask
        assert receives == got_out, mask
        assert reduces == reduced, mask
        # the trainable source receives but does not send
        for j in range(k):
            assert (receives[j] and not sends[j]) == (mask[j] and not any(mask[:j]))


def _footprint(d):
    ev = d["order"]["events"] if d["order"] else []
    bwd_regions = sorted({e[1] for e in ev if e[0] == "Bwd"})
    return (tuple(d["runs_bwd"]), tuple(s[2] is not None for s in d["seams"]),
            tuple(j for j, _ in d["reduces"]), tuple(bwd_regions) if d["order"] else None)


@pytest.mark.parametrize("k", [2, 3])
def test_corollary1_footprint_is_schedule_invariant(k):
    P, M = 2, 4
    cut = [2 * (i + 1) for i in range(k - 1)]
    L = 2 * k
    for mask in itertools.product([False, True], repeat=k):
        seen = set()
        for sched in itertools.product(S.SKELETONS, repeat=k):
            if not S.valid(cut, L, list(sched)):
                continue
            d = S.derive(cut, L, list(sched), list(mask), P, M)
            fp = _footprint(d)
            seen.add(fp[:3])
            if fp[3] is not None:
                assert fp[3] == tuple(j for j in range(k) if d["runs_bwd"][j])
        assert len(seen) == 1, (mask, seen)


# ---------------------------------------------------------------------------
# makespan and bubble in closed form (Sec. 4.3 with textbook pipeline results)
# ---------------------------------------------------------------------------

def _uniform_costs(d, f, b):
    return {e: (f if e[0] == "Fwd" else b if e[0] == "Bwd" else 0.0) for e in d["order"]["events"]}


@pytest.mark.parametrize("sk", ["1f1b", "gpipe"])
@pytest.mark.parametrize("P,M", [(1, 1), (1, 5), (2, 1), (3, 2), (4, 4), (4, 7), (5, 12)])
def test_single_region_makespan_closed_form(sk, P, M):
    d = S.derive([], P, [sk], [True], P, M)
    f, b = 1.25, 2.5
    T, bub, _, _ = S.simulate(d["order"], _uniform_costs(d, f, b))
    assert T == pytest.approx((M + P - 1) * (f + b))
    for r in range(P):
        assert bub[r] == pytest.approx((P - 1) * (f + b))


@pytest.mark.parametrize("P,S_,M", [(2, 2, 2), (2, 2, 4), (2, 3, 6), (4, 2, 4), (4, 2, 8),
                                    (4, 3, 8), (3, 2, 9), (4, 4, 12)])
def test_interleaved_makespan_closed_form(P, S_, M):
    cut = [P * (i + 1) for i in range(S_ - 1)]
    d = S.derive(cut, P * S_, ["1f1b"] * S_, [True] * S_, P, M)
    f, b = 1.0, 2.0
    T, bub, _, _ = S.simulate(d["order"], _uniform_costs(d, f, b))
    assert T == pytest.approx((M * S_ + P - 1) * (f + b))


def test_frozen_everything_is_a_forward_pipeline():
    P, M, f = 4, 6, 1.5
    d = S.derive([], 4, ["1f1b"], [False], P, M)
    assert not any(e[0] == "Bwd" for e in d["order"]["events"])
    T, _, _, _ = S.simulate(d["order"], _uniform_costs(d, f, 0.0))
    assert T == pytest.approx((M + P - 1) * f)


def test_simulation_agrees_with_a_plain_longest_path():
    """On random costs the simulated step time equals the longest path through the
    order graph plus the rank sequences (the agreement Sec. 4.3 states)."""
    rng = random.Random(7)
    for sched, cut, L, P, M in [(["transpose", "1f1b"], [3], 11, 4, 8),
                                (["1f1b", "1f1b", "1f1b"], [4, 8], 12, 4, 8),
                                (["transpose", "gpipe"], [2], 6, 3, 5)]:
        d = S.derive(cut, L, sched, [True] * len(sched), P, M)
        cost = {e: rng.uniform(0.1, 3.0) for e in d["order"]["events"]}
        T, _, _, fin = S.simulate(d["order"], cost)
        preds = {e: [] for e in d["order"]["events"]}
        for a, b, _ in d["order"]["edges"]:
            preds[b].append(a)
        for seq in d["order"]["nodes"].values():
            for a, b in zip(seq, seq[1:]):
                preds[b].append(a)
        memo = {}

        def longest(e):
            if e not in memo:
                memo[e] = cost[e] + max((longest(p) for p in preds[e]), default=0.0)
            return memo[e]
        import sys
        sys.setrecursionlimit(10000)
        assert T == pytest.approx(max(longest(e) for e in preds))
        for e in preds:
            assert fin[e] == pytest.approx(longest(e))


# ---------------------------------------------------------------------------
# memory in closed form
# ---------------------------------------------------------------------------

def _unit_bytes(d, enc=0.0):
    return {e: (enc if e[1] == 0 and d["layout"][0] == "Replicated" else 1.0)
            for e in d["order"]["events"] if e[0] == "Fwd"}


@pytest.mark.parametrize("P,M", [(1, 3), (2, 5), (4, 3), (4, 8), (6, 6)])
def test_memory_1f1b_and_gpipe(P, M):
    d = S.derive([], P, ["1f1b"], [True], P, M)
    peak = S.memory_peak(d, _unit_bytes(d))
    assert [peak[r] for r in range(P)] == [min(P - r, M) for r in range(P)]
    d = S.derive([], P, ["gpipe"], [True], P, M)
    peak = S.memory_peak(d, _unit_bytes(d))
    assert [peak[r] for r in range(P)] == [M] * P


@pytest.mark.parametrize("P,S_,M", [(2, 2, 4), (4, 2, 8), (4, 3, 8), (3, 2, 3)])
def test_memory_interleaved(P, S_, M):
    cut = [P * (i + 1) for i in range(S_ - 1)]
    d = S.derive(cut, P * S_, ["1f1b"] * S_, [True] * S_, P, M)
    peak = S.memory_peak(d, _unit_bytes(d))
    total = M * S_
    for r in range(P):
        warm = total if M == P else min(2 * (P - 1 - r) + (S_ - 1) * P, total)
        assert peak[r] == min(warm + 1, total)


@pytest.mark.parametrize("trainable_enc", [True, False])
def test_memory_transposed_encoder(trainable_enc):
    """The trainable transposed encoder is one long Activation edge: each owned
    micro-batch's encoder activation is live across the backbone's whole span.  A
    frozen encoder keeps none (its output is consumed by the seam gather)."""
    P, M, a = 4, 8, 10.0
    owner = [0, 1, 2, 3, 3, 2, 3, 3]
    d = S.derive([2], 6, ["transpose", "1f1b"], [trainable_enc, True], P, M, owner=owner)
    peak = S.memory_peak(d, _unit_bytes(d, enc=a))
    for r in range(P):
        n = owner.count(r)
        llm = min(P - r, M)
        want = n * a + llm if trainable_enc else max(a if n else 0.0, llm)
        assert peak[r] == want


# ---------------------------------------------------------------------------
# Table 2 and the cost model
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("mask", list(itertools.product([False, True], repeat=3)))
def test_seam_table_rows(mask):
    """Table 2 row by row on <transpose, 1f1b, transpose>, a valid schedule that has both
    cross-layout seams (their rows are mirrors), with Lemma 1 gating each reverse one."""
    d = S.derive([2, 6], 8, ["transpose", "1f1b", "transpose"], list(mask), 2, 4)
    assert d["layout"] == ["Replicated", "Sharded", "Replicated"]
    assert d["seams"] == [((0, 1), "Gather", "Scatter" if mask[0] else None),
                          ((1, 2), "Scatter", "Gather" if (mask[0] or mask[1]) else None)]
    assert d["reduces"] == [(j, "ReplicaGroup" if j != 1 else "DataGroup")
                            for j in range(3) if mask[j]]
    assert d["order"] is None   # a transposed sink is outside the ordered cases


def test_cost_model_shares_and_collectives():
    """Sec. 4.3: a Sharded region's slabs share its cost by layer count (the slab costs
    of one micro-batch sum to the region's), the Replicated region's forward of m costs
    its whole encode on owner(m), a collective costs alpha + beta n."""
    P, M, L, cut = 3, 3, 12, [2]          # the Sharded region has 10 layers on 3 ranks
    d = S.derive(cut, L, ["transpose", "1f1b"], [True, True], P, M, owner=[2, 0, 1])
    fwd = [[1.0, 2.0, 3.0], [30.0, 60.0, 90.0]]
    bwd = [[2.0, 4.0, 6.0], [60.0, 120.0, 180.0]]
    seam = [[100.0, 200.0, 300.0]]
    c = S.event_costs(d, cut, L, fwd, bwd, seam, [7.0, 11.0], 0.5, 0.01, 4.0)
    for m in range(M):
        assert sum(c[("Fwd", 1, r, m)] for r in range(P)) == pytest.approx(fwd[1][m])
        assert sum(c[("Bwd", 1, r, m)] for r in range(P)) == pytest.approx(bwd[1][m])
        assert c[("Fwd", 1, 0, m)] == pytest.approx(fwd[1][m] * 3 / 10)   # layers 2..4
        assert c[("Fwd", 1, 1, m)] == pytest.approx(fwd[1][m] * 3 / 10)   # layers 5..7
        assert c[("Fwd", 1, 2, m)] == pytest.approx(fwd[1][m] * 4 / 10)   # layers 8..11
        o = d["owner"][m]
        assert c[("Fwd", 0, o, m)] == fwd[0][m] and c[("Bwd", 0, o, m)] == bwd[0][m]
        assert c[("Coll", "Gather", 0, m)] == pytest.approx(0.5 + 0.01 * seam[0][m])
        assert c[("Coll", "Scatter", 0, m)] == pytest.approx(0.5 + 0.01 * seam[0][m])
        assert c[("Loss", m)] == 4.0
    assert c[("DpReduce", 0, "ReplicaGroup")] == pytest.approx(0.5 + 0.07)
    assert c[("DpReduce", 1, "DataGroup")] == pytest.approx(0.5 + 0.11)
    assert c[("StepBarrier",)] == 0.0


def test_bylayer_slabs_tile_the_region():
    for n, P in [(10, 3), (7, 7), (64, 5), (9, 4)]:
        d = S.derive([], n, ["1f1b"], [True], P, 1)
        slabs = d["placement"][0][1][1]
        assert slabs[0][0] == 0 and slabs[P - 1][1] == n
        assert all(slabs[r][1] == slabs[r + 1][0] for r in range(P - 1))
        sizes = [hi - lo for lo, hi in slabs.values()]
        assert max(sizes) - min(sizes) <= 1 and min(sizes) >= 1
