"""The incremental scatter (shc_scatter_update): from the zero-fill scatter of
one active set, the zero-fill scatter of the next (the dense form y (.) m of
Eq. 1 restated for the new mask), bit-identical to shc_scatter with zero fill
and to the oracle after every step of a sequence of masks.  Every input is
seeded and synthetic.
"""
import numpy as np
import pytest
import torch

from oracle import shc_oracle as O
from paper_2608_09388_amd import binding as shc
from paper_2608_09388_amd import synth
from tests.gpu_util import TORCH, Compaction, down, require_gpu, up

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


def mask_sequence(B, V, rng):
    """Random masks of several densities, an empty one, a full one, a repeat
    (no row changes) and one disjoint from its predecessor."""
    ms = [rng.random((B, V)) < p for p in (0.05, 0.3, 0.01)]
    ms.append(np.zeros((B, V), bool))
    ms.append(rng.random((B, V)) < 0.2)
    ms.append(ms[-1].copy())
    ms.append(np.ones((B, V), bool))
    ms.append(rng.random((B, V)) < 0.1)
    ms.append(~ms[-1] & (rng.random((B, V)) < 0.15))
    ms.append(np.zeros((B, V), bool))
    return [m.astype(np.uint8) for m in ms]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("C,B,V", [(16, 9, 1000), (48, 5, 777), (128, 9, 1000),
                                   (256, 3, 500), (2048, 2, 300)])
def test_update_sequence_equals_zero_fill(dev, dtype, C, B, V):
    rng = np.random.default_rng(C + V)
    D = torch.zeros((B * V, C), dtype=TORCH[dtype], device=dev)
    prev = torch.empty((B * V, 2), dtype=torch.int32, device=dev)
    prev_n = 0
    for step, m in enumerate(mask_sequence(B, V, rng)):
        c = Compaction(m)
        n = c.run()
        S_host = synth.as_dtype(rng.standard_normal((max(n, 1), C)).astype(np.float32),
                                dtype)[1][:n]
        S = up(S_host, dtype) if n else torch.empty((1, C), dtype=D.dtype, device=dev)
        shc.scatter_update(S, c.inv, c.coords, n, prev, prev_n, B, V, D)
        ref = torch.full_like(D, float("nan"))
        if n:
            shc.scatter(S, c.inv, c.coords, n, B, V, ref, zero_fill=True)
        else:
            ref.zero_()
        assert torch.equal(D, ref), (step, n, prev_n)
        _, ref_inv, _, _ = O.compact(m)
        exp = O.scatter(S_host.astype(np.float64).reshape(n, C), ref_inv, zero_fill=True)
        assert np.array_equal(down(D), exp), (step, n)
        prev[:n].copy_(c.coords[:n])
        prev_n = n
    torch.cuda.synchronize()


def test_update_leaves_other_rows_alone(dev):
    """Rows that neither set holds keep whatever they held (here a sentinel):
    the update writes only the previous set's rows that are inactive now and
    the current set's rows."""
    B, V, C = 4, 900, 64
    rng = np.random.default_rng(5)
    m0 = (rng.random((B, V)) < 0.2).astype(np.uint8)
    m1 = (rng.random((B, V)) < 0.2).astype(np.uint8)
    c0, c1 = Compaction(m0), Compaction(m1)
    n0, n1 = c0.run(), c1.run()
    S1 = up(rng.standard_normal((n1, C)).astype(np.float32), "f32")
    D = torch.full((B * V, C), 3.5, dtype=torch.float32, device=dev)
    shc.scatter_update(S1, c1.inv, c1.coords, n1, c0.coords, n0, B, V, D)
    got = down(D)
    a0, a1 = m0.reshape(-1) > 0, m1.reshape(-1) > 0
    assert np.all(got[a0 & ~a1] == 0)
    assert np.all(got[~a0 & ~a1] == 3.5)
    _, inv1, _, _ = O.compact(m1)
    rows = np.flatnonzero(a1)
    assert np.array_equal(got[rows], down(S1)[inv1[rows]])
    torch.cuda.synchronize()


def test_update_prepared_and_errors(dev):
    B, V, C = 3, 400, 32
    rng = np.random.default_rng(8)
    m0 = (rng.random((B, V)) < 0.3).astype(np.uint8)
    m1 = (rng.random((B, V)) < 0.1).astype(np.uint8)
    c0, c1 = Compaction(m0), Compaction(m1)
    n0, n1 = c0.run(), c1.run()
    S0 = up(rng.standard_normal((n0, C)).astype(np.float32), "bf16")
    S1 = up(rng.standard_normal((n0, C)).astype(np.float32), "bf16")
    D = torch.zeros((B * V, C), dtype=torch.bfloat16, device=dev)
    prev = torch.empty((B * V, 2), dtype=torch.int32, device=dev)
    shc.scatter(S0, c0.inv, c0.coords, n0, B, V, D, zero_fill=True)
    prev[:n0].copy_(c0.coords[:n0])
    upd = shc.prepare_scatter_update(S1, c1.inv, c1.coords, prev, B, V, D)
    upd(n1, n0)
    ref = torch.empty_like(D)
    shc.scatter(S1, c1.inv, c1.coords, n1, B, V, ref, zero_fill=True)
    assert torch.equal(D, ref)
    with pytest.raises(ValueError):
        upd(n0 + 1, 0)
    with pytest.raises(ValueError):
        upd(0, B * V + 1)
    # the same buffer as both coordinate lists is refused
    with pytest.raises(shc.ShcError, match="INVALID"):
        shc.scatter_update(S1, c1.inv, c1.coords, n1, c1.coords, n1, B, V, D)
    # nothing to do: no launch, D untouched
    shc.scatter_update(S1, c1.inv, c1.coords, 0, prev, 0, B, V, D)
    assert torch.equal(D, ref)
    torch.cuda.synchronize()


@pytest.mark.parametrize("side", [False, True])
def test_stack_incremental_scatter(dev, side):
    """The density-sweep stack at 5% on 24 bodies with incremental_scatter:
    the dense output after every batch identical to the zero-fill stack's,
    batch by batch (one run() each) and over a pipelined run of four."""
    from paper_2608_09388_amd.pipeline import SparseStack
    w = synth.workload_c4(0.05, B=24)
    masks = [np.random.default_rng(90 + k).random(w.B * w.V) < p
             for k, p in enumerate((0.05, 0.02, 0.0, 0.08, 0.05))]
    stacks = {inc: SparseStack(w, device=dev, side_stream=side, incremental_scatter=inc)
              for inc in (False, True)}
    assert stacks[True].incremental_scatter and not stacks[False].incremental_scatter
    for k, m in enumerate(masks):
        outs = {}
        for inc, st in stacks.items():
            st.mask.copy_(torch.from_numpy(m.astype(np.uint8)).to(dev))
            n = st.run(1)
            torch.cuda.synchronize()
            outs[inc] = (n, st.dense_out.clone(), st.pooled.clone())
        assert outs[False][0] == outs[True][0], k
        assert torch.equal(outs[False][1], outs[True][1]), k
        assert torch.equal(outs[False][2], outs[True][2]), k
    outs = {}
    for inc, st in stacks.items():
        def feed(k, st=st):
            st.mask.copy_(torch.from_numpy(masks[(k + 2) % 5].astype(np.uint8)).to(dev))

        n = st.run(4, feed=feed)
        torch.cuda.synchronize()
        outs[inc] = (n, st.dense_out.clone())
    assert outs[False][0] == outs[True][0]
    assert torch.equal(outs[False][1], outs[True][1])
