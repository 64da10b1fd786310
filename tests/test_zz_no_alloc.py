"""shc_compact_mask_noalloc (the compaction that takes no workspace) against
shc_compact_mask and the oracle, bit for bit, on two calls in a row: a
density-sweep batch, then a smaller mask whose call finds the first one's
counts still in the library's scratch."""
import numpy as np
import pytest
import torch

from oracle import shc_oracle as O
from paper_2608_09388_amd import binding as shc
from paper_2608_09388_amd import synth
from tests.gpu_util import Compaction, down, require_gpu, up

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


def run_noalloc(mask, host):
    """The allocation-free call on fresh sentinel-filled outputs."""
    B, V = mask.shape
    md = up(mask.reshape(-1).astype(np.uint8))
    coords = torch.full((B * V, 2), -7, dtype=torch.int32, device="cuda")
    inv = torch.full((B * V,), -7, dtype=torch.int32, device="cuda")
    row_ptr = torch.full((B + 1,), -7, dtype=torch.int32, device="cuda")
    n_dev = torch.full((4,), -7, dtype=torch.int32, device="cuda")
    if host == "pinned":
        hc = torch.full((1,), -9, dtype=torch.int64).pin_memory()
        n = shc.compact_mask_noalloc(md, B, V, coords, inv, row_ptr, n_dev, host_count=hc)
    elif host == "pageable":
        n = shc.compact_mask_noalloc(md, B, V, coords, inv, row_ptr, n_dev)
    else:
        shc.compact_mask_noalloc(md, B, V, coords, inv, row_ptr, n_dev, want_host_count=False)
        torch.cuda.synchronize()
        n = int(n_dev[0])
    torch.cuda.synchronize()
    return n, down(coords)[:n], down(inv), down(row_ptr), int(n_dev[0])


@pytest.mark.parametrize("host", ["pinned", "pageable", "none"])
def test_noalloc_matches_compact_mask_twice(dev, host):
    big = synth.workload_c4(0.05).mask            # 128 x 10475
    rng = np.random.default_rng(5)
    small = (rng.random((4, 655)) < 0.1).astype(np.uint8)
    for mask in (big, small):
        B, V = mask.shape
        n, coords, inv, rp, n_dev = run_noalloc(mask, host)
        ref = Compaction(mask)
        n_ref = ref.run(want_host=True)
        torch.cuda.synchronize()
        assert n == n_ref == n_dev
        assert np.array_equal(coords, down(ref.coords)[:n_ref])
        assert np.array_equal(inv, down(ref.inv))
        assert np.array_equal(rp, down(ref.row_ptr))
        oc, oi, orp, on = O.compact(mask)
        assert n == on and np.array_equal(coords, oc)
        assert np.array_equal(inv, oi) and np.array_equal(rp, orp)


def test_noalloc_capacity_error(dev):
    """N' above cap: SHC_ERR_CAPACITY, as for shc_compact_mask."""
    mask = np.ones((2, 300), np.uint8)
    md = up(mask.reshape(-1))
    coords = torch.empty((100, 2), dtype=torch.int32, device="cuda")
    inv = torch.empty(600, dtype=torch.int32, device="cuda")
    rp = torch.empty(3, dtype=torch.int32, device="cuda")
    nd = torch.empty(4, dtype=torch.int32, device="cuda")
    with pytest.raises(shc.ShcError) as e:
        shc.compact_mask_noalloc(md, 2, 300, coords, inv, rp, nd)
    assert e.value.status == -2
    torch.cuda.synchronize()
