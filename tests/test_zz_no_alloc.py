"""The allocation-free index check (mpipe_merge_check_indices_noalloc) against the
existing entry point that takes a caller buffer, through the C ABI, on two calls in a
row (the second smaller, so stale counters of the first would show), plus its size
limit and the host-side constant's agreement with the header."""
import os
import re

import numpy as np
import pytest

import workload as W
from tests.gpu_util import announce, torch_dev

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_noalloc_limit_matches_header():
    import paper_2607_03229_amd as mp
    src = open(os.path.join(ROOT, "include", "mpipe.h")).read()
    m = re.search(r"#define MPIPE_CHECK_NOALLOC_MAX_ROWS \(1 << (\d+)\)", src)
    assert m and mp.CHECK_NOALLOC_MAX_ROWS == 1 << int(m.group(1))


@pytest.mark.gpu
def test_noalloc_check_matches_buffered_check():
    import paper_2607_03229_amd as mp
    torch, dev = torch_dev()
    rng = np.random.default_rng(21)
    wl = W.make_workload("c4_qwen2vl_trained", 0)
    big_rows = wl.emb_rows
    cases = [
        # (indices, n_rows): the benchmark's placeholders, then smaller problems that reuse
        # rows the previous call marked
        (wl.placeholders(), big_rows),
        (np.array([3, 17, 3, 99], np.int64), 100),               # a repeat
        (np.array([0, 5, 100], np.int64), 100),                  # out of range
        (rng.permutation(64)[:40].astype(np.int64), 64),          # clean, rows marked before
        (np.array([], np.int64), 10),                            # nothing to check
        (np.array([-1, 2, 2], np.int64), 3),                     # both
    ]
    status_a = torch.empty(1, dtype=torch.int32, device=dev)
    status_b = torch.empty(1, dtype=torch.int32, device=dev)
    for idx, n_rows in cases:
        announce(f"noalloc index check: {len(idx)} indices over {n_rows} rows")
        t = torch.from_numpy(idx).to(dev)
        marks = torch.empty(max(n_rows, 1), dtype=torch.int32, device=dev)
        status_a.fill_(-7)
        status_b.fill_(-7)
        mp.merge_check_indices(t, n_rows, marks, status_a)
        mp.merge_check_indices_noalloc(t, n_rows, status_b)
        torch.cuda.synchronize()
        a, b = int(status_a.item()), int(status_b.item())
        want = (1 if ((idx < 0) | (idx >= n_rows)).any() else 0) | \
               (2 if len(np.unique(idx[(idx >= 0) & (idx < n_rows)])) <
                ((idx >= 0) & (idx < n_rows)).sum() else 0)
        assert a == b == want, (len(idx), n_rows, a, b, want)
    # beyond the built-in scratch: rejected on the host, nothing enqueued
    status_b.fill_(-7)
    with pytest.raises(mp.MpipeError) as e:
        mp.merge_check_indices_noalloc(torch.zeros(1, dtype=torch.int64, device=dev),
                                       mp.CHECK_NOALLOC_MAX_ROWS + 1, status_b)
    assert e.value.status == -3
    torch.cuda.synchronize()
    assert int(status_b.item()) == -7
