"""Host-side model of the large GEMM kernel's K-tile schedule (gemm_big.hip).

The kernel fills an NST-stage LDS ring by DMA (NST = 4 for 256x256 tiles, 3 for
128x256 tiles): the prologue issues tiles 0..NST-1, the steady-state passes (entered
while t + 2 NST + 1 <= nk) issue tile t + NST from unclamped sources and read
fragments without the ragged-K mask, and the tail bodies issue tile t + NST through
the clamping path.  This model replays that control flow for
many K ranges and split sizes and checks that every tile is filled exactly once,
that no unclamped source or unmasked read ever touches the last, ragged tile, and
that each wait leaves exactly the later tiles pending.  It catches schedule changes
that would read past the end of an operand before they reach a GPU.
"""
import pytest

BK = 32


def _schedule(kbeg, kend, nst=4):
    nk = (kend - kbeg + BK - 1) // BK if kend > kbeg else 0
    def full(tile):
        return kbeg + (tile + 1) * BK <= kend
    issued = []            # (tile, path) in issue order
    problems = []
    for tile in range(min(nst, nk)):
        issued.append((tile, "clamped"))
    t = 0
    while t + 2 * nst + 1 <= nk:
        for b in range(nst):
            tb = t + b
            if tb % nst != b:
                problems.append(("stage of tile is not tile % NST", tb))
            issued.append((tb + nst, "fast"))
            if not (full(tb + nst) and full(0)):
                problems.append(("unclamped DMA of a ragged tile", tb + nst))
            if not (full(tb) and full(tb + 1)):
                problems.append(("unmasked read of a ragged tile", tb))
            # the wait before the barrier keeps NST-2 tiles pending: they must all be
            # tiles issued after tb+1
            pending_after = min(tb + nst - 1, nk - 1) - (tb + 1)
            if pending_after < nst - 2:
                problems.append(("steady wait would not cover tile", tb + 1))
        t += nst
    while t < nk:
        for b in range(nst):
            tb = t + b
            if tb < nk and tb + nst < nk:
                issued.append((tb + nst, "clamped"))
        t += nst
    tiles = sorted(x for x, _ in issued)
    if tiles != list(range(nk)):
        problems.append(("tiles not filled exactly once", tiles))
    return problems


@pytest.mark.parametrize("nst", [3, 4])
@pytest.mark.parametrize("K", list(range(1, 700, 7)) + [1216, 1280, 3840, 5120, 42940])
def test_schedule_unsplit(K, nst):
    assert _schedule(0, K, nst) == []


@pytest.mark.parametrize("nst", [3, 4])
@pytest.mark.parametrize("K,kps", [(1000, 256), (42940, 2688), (42940, 4352), (5000, 64),
                                   (999, 320), (42940, 42944), (300, 128)])
def test_schedule_split(K, kps, nst):
    splits = (K + kps - 1) // kps
    for s in range(splits):
        assert _schedule(s * kps, min(K, (s + 1) * kps), nst) == [], (K, kps, s)


def test_model_flags_the_old_bound():
    """Entering the steady state at t + 8 <= nk would DMA the ragged last tile unclamped
    (K range 232 = 8 tiles, the last one partial); the model must see that."""
    def old(kbeg, kend):
        nk = (kend - kbeg + BK - 1) // BK
        bad = []
        t = 0
        while t + 8 <= nk:
            for b in range(4):
                if kbeg + (t + b + 5) * BK > kend:
                    bad.append(t + b + 4)
            t += 4
        return bad
    assert old(768, 1000) == [7]
    assert _schedule(768, 1000) == []
