"""Host-side models of the large GEMM kernels' K-tile schedules (gemm_big.hip).

The 256x256 weight-gradient kernel fills an NST-stage LDS ring by DMA (NST = 4): the
prologue issues tiles 0..NST-1, the steady-state passes (entered while t + 2 NST + 1 <= nk)
issue tile t + NST from unclamped sources and read fragments without the ragged-K mask,
and the tail bodies issue tile t + NST through the clamping path.  The 128x256 NN kernel
fills A two K tiles at a time into two pair stages and B into three stages.  The NT kernel
takes 64-deep tiles in two stages and issues tile t + 2 after the barrier in tile t.  These models
replay the control flow for many K ranges and split sizes and check that every tile
is filled exactly once, that no unclamped source or unmasked read ever touches the
last, ragged tile, that each wait leaves only later DMAs pending and that no stage is
refilled before its last read.  They catch schedule changes that would read past the
end of an operand before they reach a GPU.
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


@pytest.mark.parametrize("K", list(range(1, 700, 7)) + [1216, 1280, 3840, 5120, 42940])
def test_schedule_unsplit(K):
    assert _schedule(0, K) == []


@pytest.mark.parametrize("K,kps", [(1000, 256), (42940, 2688), (42940, 4352), (5000, 64),
                                   (999, 320), (42940, 42944), (300, 128)])
def test_schedule_split(K, kps):
    splits = (K + kps - 1) // kps
    for s in range(splits):
        assert _schedule(s * kps, min(K, (s + 1) * kps)) == [], (K, kps, s)
        assert _nn_schedule(s * kps, min(K, (s + 1) * kps)) == [], (K, kps, s)


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


def _nn_schedule(kbeg, kend, widen_odd_wait=0):
    """The NN kernel: B(t) into stage t % 3, A pair (2P, 2P+1) into pair stage P % 2;
    4 B and 4 A DMA instructions per wave per fill.  Body b reads tile b's second half
    before its barrier (time b) and tile b+1's first half after it (time b + 0.5), when
    its DMAs are issued too.  widen_odd_wait lets the model check itself: it loosens the
    odd tiles' waits by that many instructions."""
    IA = IB = 4
    nk = (kend - kbeg + BK - 1) // BK if kend > kbeg else 0
    problems = []
    def full(tile):
        return kbeg + (tile + 1) * BK <= kend
    issued = []                     # (kind, first tile, n instructions)
    b_fill, a_fill = [], []
    stage_b, stage_a = {}, {}       # stage -> tile (first tile of the pair)
    last_read = {}                  # tile -> time of its last fragment read
    def refill_ok(old_tiles, time):
        return all(last_read.get(o, -9) < time for o in old_tiles)
    def dma_b(t, fast, time):
        if fast and not full(t):
            problems.append(("fast B DMA of a ragged tile", t))
        old = stage_b.get(t % 3)
        if old is not None and not refill_ok([old], time):
            problems.append(("B stage refilled before its last read", t))
        stage_b[t % 3] = t
        issued.append(("B", t, IB))
        b_fill.append(t)
    def dma_a(t, fast, time):
        if fast and not full(t + 1):
            problems.append(("fast A pair DMA past the end", t))
        old = stage_a.get((t // 2) % 2)
        if old is not None and not refill_ok([old, old + 1], time):
            problems.append(("pair stage refilled before its last read", t))
        stage_a[(t // 2) % 2] = t
        issued.append(("A", t, IA))
        a_fill.append(t)
    def check_wait(pending, tile):
        # every DMA of `tile` must be outside the last `pending` instructions issued
        tail, n = [], 0
        for kind, t0, cnt in reversed(issued):
            if n >= pending:
                break
            tail.append((kind, t0))
            n += cnt
        if ("B", tile) in tail or ("A", tile - tile % 2) in tail:
            problems.append(("wait does not cover tile", tile))
    def read(t, masked_ok, time):
        if not masked_ok and not full(t):
            problems.append(("unmasked read of a ragged tile", t))
        last_read[t] = time
    if nk == 0:
        return problems
    # prologue, as bodies -3, -2, -1
    dma_b(0, False, -3.5); dma_a(0, False, -3.5)
    if nk > 1: dma_b(1, False, -2.5)
    if nk > 2: dma_b(2, False, -1.5); dma_a(2, False, -1.5)
    check_wait(2 * IB + IA if nk > 2 else IB if nk == 2 else 0, 0)
    read(0, True, -0.5)
    nfast = (nk - 5) // 4 * 4 if nk >= 6 else 0
    t = 0
    while t < nfast:
        for i in range(4):
            tt = t + i
            if tt + 6 > nk:
                problems.append(("fast body outside the steady state", tt))
            read(tt, False, tt)
            check_wait(IB + IA if tt % 2 == 0 else IB + widen_odd_wait, tt + 1)
            dma_b(tt + 3, True, tt + 0.5)
            if tt % 2:
                dma_a(tt + 3, True, tt + 0.5)
            read(tt + 1, False, tt + 0.5)
        t += 4
    while t < nk:
        for i in range(4):
            tt = t + i
            if tt >= nk:
                break
            read(tt, True, tt)
            if tt + 1 < nk:
                check_wait((IB + widen_odd_wait if tt % 2 else IB + IA) if tt + 2 < nk else 0, tt + 1)
            if tt + 3 < nk:
                dma_b(tt + 3, False, tt + 0.5)
                if tt % 2:
                    dma_a(tt + 3, False, tt + 0.5)
            if tt + 1 < nk:
                read(tt + 1, True, tt + 0.5)
        t += 4
    if sorted(b_fill) != list(range(nk)):
        problems.append(("B tiles not filled exactly once", b_fill))
    if sorted(a_fill) != list(range(0, nk, 2)):
        problems.append(("A pairs not filled exactly once", a_fill))
    return problems


@pytest.mark.parametrize("K", list(range(1, 900, 7)) + [1216, 1280, 3840, 5120, 42940])
def test_nn_schedule(K):
    assert _nn_schedule(0, K) == []


def test_nn_model_flags_a_loose_wait():
    """Letting the odd tiles' waits keep one more A pair in flight would leave tile t+1's
    pair unfinished; the model must see that."""
    assert _nn_schedule(0, 40 * BK) == []
    assert ("wait does not cover tile", 2) in _nn_schedule(0, 40 * BK, widen_odd_wait=4)


def _nt64_schedule(kbeg, kend, steady_bound=4):
    """The NT kernel with 64-deep K tiles: tile t in stage t % 2, 8 A + 8 B DMA
    instructions per wave per tile.  The prologue issues tiles 0 and 1 and waits for tile
    0; body t reads K steps 1..3 of tile t, waits for every DMA issued (tile t+1), passes
    the barrier, issues tile t+2 into stage t % 2 and reads K step 0 of tile t+1.  Bodies
    run fenced and unguarded ("full") while t + steady_bound <= nfull, two at a time, and
    guarded after that.  steady_bound lets the model check itself (the kernel uses 4)."""
    BK64 = 64
    nk = (kend - kbeg + BK64 - 1) // BK64 if kend > kbeg else 0
    nfull = (kend - kbeg) // BK64 if kend > kbeg else 0
    problems = []
    stage = {}                  # stage -> tile it holds
    landed, pending = set(), set()
    reads_left = {}             # tile -> K steps not yet read
    filled = []
    def dma(t, unclamped):
        if unclamped and t >= nfull:
            problems.append(("unclamped DMA of a ragged tile", t))
        s = t % 2
        old = stage.get(s)
        if old is not None and reads_left.get(old, 0) > 0:
            problems.append(("stage refilled before its last read", t))
        stage[s] = t
        pending.add(t)
        reads_left[t] = 4
        filled.append(t)
    def wait_all():
        landed.update(pending)
        pending.clear()
    def read(t, step, masked):
        if stage.get(t % 2) != t or t not in landed:
            problems.append(("read of a tile not landed in its stage", (t, step)))
        if not masked and t >= nfull:
            problems.append(("unmasked read of a ragged tile", t))
        reads_left[t] -= 1
    def body(t, full):
        if full and not (t + 2 < nfull):
            problems.append(("unguarded body without a whole tile t+2", t))
        for step in (1, 2, 3):
            read(t, step, not full)
        wait_all()
        if full:
            dma(t + 2, True)
        elif t + 2 < nk:
            dma(t + 2, t + 2 < nfull)
        if full or t + 1 < nk:
            read(t + 1, 0, not full)
    if nk == 0:
        return problems
    dma(0, 0 < nfull)
    if nk > 1:
        dma(1, 1 < nfull)
        pending.discard(0)          # wait_vm<16>: tile 0 landed, tile 1 may stay pending
        landed.add(0)
    else:
        wait_all()
    read(0, 0, True)
    t = 0
    while t + steady_bound <= nfull:
        body(t, True)
        body(t + 1, True)
        t += 2
    while t < nk:
        body(t, False)
        if t + 1 < nk:
            body(t + 1, False)
        t += 2
    if sorted(filled) != list(range(nk)):
        problems.append(("tiles not filled exactly once", filled))
    if any(v != 0 for v in reads_left.values()):
        problems.append(("a tile not read in full", reads_left))
    return problems


@pytest.mark.parametrize("K", list(range(8, 1200, 8)) + [1280, 3840, 5120, 42944])
def test_nt64_schedule(K):
    assert _nt64_schedule(0, K) == []


@pytest.mark.parametrize("K,kps", [(1000, 256), (42944, 2688), (5000, 64), (1000, 320),
                                   (300, 128), (4096, 1024)])
def test_nt64_schedule_split(K, kps):
    for s in range((K + kps - 1) // kps):
        assert _nt64_schedule(s * kps, min(K, (s + 1) * kps)) == [], (K, kps, s)


def test_nt64_model_flags_a_loose_steady_bound():
    """Entering the unguarded bodies while t + 3 <= nfull would issue tile t+2 unclamped
    from the second body of the pair at K = 5 * 64 + 32 (the last tile ragged)."""
    assert _nt64_schedule(0, 5 * 64 + 32) == []
    bad = _nt64_schedule(0, 5 * 64 + 32, steady_bound=3)
    assert any(p[0] == "unguarded body without a whole tile t+2" for p in bad), bad
