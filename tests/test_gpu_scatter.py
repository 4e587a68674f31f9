"""Seam scatter / gather on the GPU: bit-exact against the oracle's row copy."""
import numpy as np
import pytest

import oracle
import workload as W
from tests.gpu_util import announce, torch_dev

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype,H,n_rows,n_m", [("bf16", 3584, 4096, 1000), ("f32", 256, 512, 40),
                                                 ("bf16", 3, 50, 7), ("bf16", 1, 10, 0)])
def test_scatter_gather_bit_exact(dtype, H, n_rows, n_m):
    import paper_2607_03229_amd as mp
    torch, dev = torch_dev()
    announce(f"scatter/gather {dtype} H={H} rows={n_rows} n={n_m}")
    rng = np.random.default_rng(H + n_m)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    udt = np.uint16 if dtype == "bf16" else np.uint32
    # arbitrary bit patterns, including NaN and Inf encodings
    mbits = rng.integers(0, np.iinfo(udt).max, (n_m, H), dtype=udt, endpoint=True)
    ebits = rng.integers(0, np.iinfo(udt).max, (n_rows, H), dtype=udt, endpoint=True)
    idx = rng.permutation(n_rows)[:n_m].astype(np.int64)
    itype = torch.int16 if dtype == "bf16" else torch.int32
    merged = torch.from_numpy(mbits.view(np.int16 if dtype == "bf16" else np.int32)).to(dev).view(tdt)
    emb = torch.from_numpy(ebits.view(np.int16 if dtype == "bf16" else np.int32)).to(dev).view(tdt)
    tidx = torch.from_numpy(idx).to(dev)
    mp.merge_scatter(merged, tidx, emb)
    got = emb.view(itype).cpu().numpy().view(udt)
    ref = oracle.merge_scatter(mbits, idx, ebits)
    np.testing.assert_array_equal(got, ref)
    out = torch.zeros_like(merged)
    mp.merge_gather(emb, tidx, out)
    np.testing.assert_array_equal(out.view(itype).cpu().numpy().view(udt), mbits)


def test_scatter_workload_placeholders():
    import paper_2607_03229_amd as mp
    torch, dev = torch_dev()
    announce("scatter c4 placeholders")
    wl = W.make_workload("c4_qwen2vl_trained", 0)
    idx = wl.placeholders()
    rng = np.random.default_rng(0)
    H = wl.cfg.llm_hidden
    merged = torch.from_numpy(rng.integers(-30000, 30000, (len(idx), H), dtype=np.int16)).to(dev)
    emb = torch.zeros((wl.emb_rows, H), dtype=torch.int16, device=dev)
    mp.merge_scatter(merged.view(torch.bfloat16), torch.from_numpy(idx).to(dev),
                     emb.view(torch.bfloat16))
    ref = oracle.merge_scatter(merged.cpu().numpy(), idx, np.zeros((wl.emb_rows, H), np.int16))
    np.testing.assert_array_equal(emb.cpu().numpy(), ref)


def test_check_indices():
    import paper_2607_03229_amd as mp
    torch, dev = torch_dev()
    announce("check_indices")
    marks = torch.empty(100, dtype=torch.int32, device=dev)
    status = torch.empty(1, dtype=torch.int32, device=dev)
    for idx, want in (([0, 5, 99], 0), ([0, 5, 5], 2), ([0, 100], 1), ([-1, 3, 3], 3), ([], 0)):
        t = torch.tensor(idx, dtype=torch.int64, device=dev)
        mp.merge_check_indices(t, 100, marks, status)
        torch.cuda.synchronize()
        assert int(status.item()) == want, (idx, int(status.item()))
