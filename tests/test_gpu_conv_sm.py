"""The sparse neighbour conv from a table on the shapes its slot-major kernel
serves (64 input channels within one round of row groups, and dense masks
with about a thousand rows or more per CU): Eqs. 4-5 against the oracle on
sampled rows, with and without bias and ReLU, rows past N' untouched.  The
bit-for-bit agreement with the weight-stationary kernel is checked where both
run on the same inputs (the planned conv of the plan tests at 64 channels).
Every input is seeded and synthetic.
"""
import numpy as np
import pytest
import torch

from oracle import shc_oracle as O
from paper_2608_09388_amd import binding as shc
from paper_2608_09388_amd import synth
from tests.gpu_util import Compaction, assert_scaled_close, down, require_gpu, up

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


def rand_nbr(V, K, rng, p_missing=0.1):
    nbr = rng.integers(0, V, size=(V, K)).astype(np.int32)
    nbr[rng.random((V, K)) < p_missing] = -1
    nbr[:, 0] = np.arange(V)
    return nbr


@pytest.mark.parametrize("B,V,K,Cin,Cout,p,mesh", [
    (64, 655, 9, 64, 64, 0.1, False),      # the encoder's 64 -> 64 layer
    (64, 655, 9, 64, 128, 0.1, False),     # and its 64 -> 128 layer
    (3, 700, 5, 64, 64, 0.4, False),       # K other than nine (a loop over the slots)
    (2, 300, 1, 64, 128, 0.6, False),      # one slot
    (4, 400, 32, 64, 64, 0.3, False),      # 32 slots
    (1, 40, 9, 64, 64, 0.5, False),        # one partial row group
    (128, 10475, 9, 128, 128, 0.2, True),  # the density-sweep batch at 20%
    (256, 10475, 9, 64, 64, 0.18, True),   # the full-mesh batch, cap-like density
])
def test_conv_sm_shapes_against_oracle(dev, B, V, K, Cin, Cout, p, mesh):
    rng = np.random.default_rng(B + V + 7 * K + Cin + Cout)
    if mesh:
        _, nbr = synth.mesh("ellipsoid", V, K, 4)
        nbr = np.ascontiguousarray(nbr, dtype=np.int32)
    else:
        nbr = rand_nbr(V, K, rng)
    m = (rng.random((B, V)) < p).astype(np.uint8)
    c = Compaction(m)
    n = c.run()
    table = torch.full((max(K * n, 1),), -7, dtype=torch.int32, device=dev)
    shc.build_neighbor_table(c.coords, c.inv, n, B, V, up(nbr), table)
    S = synth.as_dtype(rng.standard_normal((n, Cin)).astype(np.float32), "bf16")[1]
    W = synth.as_dtype((rng.standard_normal((K, Cin, Cout)) / np.sqrt(K * Cin))
                       .astype(np.float32), "bf16")[1]
    bias = rng.standard_normal(Cout).astype(np.float32)
    coords, _, _, n_ref = O.compact(m)
    assert n_ref == n
    rows = np.unique(np.concatenate([np.arange(min(n, 200)), np.arange(max(0, n - 200), n),
                                     rng.choice(n, size=min(n, 400), replace=False)]))
    Sd, Wd = up(S, "bf16"), up(W, "bf16")
    for b, act in ((bias, shc.SHC_ACT_RELU), (None, shc.SHC_ACT_NONE)):
        out = torch.full((n + 3, Cout), float("nan"), dtype=torch.bfloat16, device=dev)
        shc.sparse_neighbor_conv_table(Sd, table, n, Wd, None if b is None else up(b), out, act)
        got = down(out)
        assert np.all(np.isnan(got[n:]))
        ref = O.conv_at(S, coords, B, V, nbr, W, rows, b, act=act == shc.SHC_ACT_RELU)
        scale = O.conv_at(S, coords, B, V, nbr, W, rows, b, scale=True)
        assert_scaled_close(got[rows], ref, scale, "bf16",
                            f"conv K={K} {Cin}->{Cout} p={p} act={act}", n_terms=K * Cin)
    torch.cuda.synchronize()
