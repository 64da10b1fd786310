"""The stack executor (shc_stack_create / shc_stack_run): the whole path over
consecutive batches issued from the library's native loop must leave exactly
the outputs of the same calls issued one by one from Python (pipeline.py's
own schedules), on every workload shape the stack takes: linear-first and
conv-first stacks, fp32 and bf16, fused and separate neighbour tables, conv
plans, the split conv (256-channel layers), zero-fill and incremental
scatter, pool only, serial and pipelined.
The per-call results themselves are checked against the oracle by the layer
tests; the stack's against the oracle by test_stack_outputs_match_oracle.
Every input is seeded and synthetic.
"""
import numpy as np
import pytest
import torch

from oracle import shc_oracle as O
from paper_2608_09388_amd import binding as shc
from paper_2608_09388_amd import synth
from paper_2608_09388_amd.pipeline import SparseStack
from tests.gpu_util import assert_scaled_close, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


def wide_body_workload():
    """V = 20000 (above what the compaction's on-chip row numbering holds,
    so the table is a call of its own), random 9-neighbour lists, bf16
    conv 64 -> 64 -> 64 with a bias, scatter and pool."""
    B, V, K, C = 3, 20000, 9, 64
    rng = np.random.default_rng(77)
    nbr = rng.integers(0, V, size=(V, K)).astype(np.int32)
    nbr[rng.random((V, K)) < 0.1] = -1
    nbr[:, 0] = np.arange(V)
    m = synth.bernoulli_mask(B, V, 0.05, rng)
    x = synth.as_dtype(synth.features(B * V, C, rng), "bf16")[1]
    layers = []
    for _ in range(2):
        W = synth.as_dtype(synth.conv_weights(K, C, C, rng).reshape(-1), "bf16")[1]
        layers.append(synth.Layer("conv", C, C, W.reshape(K, C, C),
                                  rng.standard_normal(C).astype(np.float32), True))
    return synth.Workload("wide bodies", B, V, K, "bf16", np.zeros((V, 3)), nbr, m, x, layers,
                          pool=True, scatter=True)


WORKLOADS = {
    "c4_5pct_b24": lambda: synth.workload_c4(0.05, B=24),
    "c1_fp32": synth.workload_c1,
    "c2_encoder": synth.workload_c2,
    "c5_sequences": lambda: synth.workload_c5(4, 8),
    "wide_bodies": wide_body_workload,
}


def masks_for(w, k0, n=4):
    """Batch masks: the workload's own, then Bernoulli masks of 0.5x to 2x
    its density, and an empty one."""
    p = float(np.mean(w.mask))
    out = [w.mask.reshape(-1)]
    for k in range(1, n - 1):
        rng = np.random.default_rng(1000 * k0 + k)
        out.append(rng.random(w.B * w.V) < p * (0.5 + 0.5 * k))
    out.append(np.zeros(w.B * w.V, bool))
    return [m.astype(np.uint8) for m in out]


def run_stack(w, dev, executor, side, inc, plans, masks, batched):
    # plans are taken by shapes the packed conv does not run
    st = SparseStack(w, device=dev, side_stream=side, conv_plans=plans,
                     incremental_scatter=inc, executor=executor,
                     packed_conv=False if plans else None)
    assert st.executor == executor
    md = [torch.from_numpy(m).to(dev) for m in masks]
    snaps = []

    def snap(n):
        torch.cuda.synchronize()
        snaps.append((n, [a[:n].clone() for a in st.acts[1:]],
                      st.dense_out.clone() if st.dense_out is not None else None,
                      st.pooled.clone() if st.pooled is not None else None))

    if batched:
        # all batches in one run, fed batch by batch; outputs of the last
        def feed(k):
            st.mask.copy_(md[k])

        snap(st.run(len(masks), feed=feed))
        # and one more run of two batches over the last mask, same buffers
        snap(st.run(2))
    else:
        for m in md:
            st.mask.copy_(m)
            snap(st.run(1))
    return snaps


def assert_same(a, b, what):
    assert len(a) == len(b)
    for k, (x, y) in enumerate(zip(a, b)):
        assert x[0] == y[0], (what, k, x[0], y[0])
        for l, (u, v) in enumerate(zip(x[1], y[1])):
            assert torch.equal(u, v), (what, k, "layer", l)
        for name, u, v in (("dense", x[2], y[2]), ("pool", x[3], y[3])):
            assert (u is None) == (v is None)
            if u is not None:
                assert torch.equal(u, v), (what, k, name)


@pytest.mark.parametrize("name", list(WORKLOADS))
@pytest.mark.parametrize("side", [False, True])
def test_native_matches_python_schedule(dev, name, side):
    w = WORKLOADS[name]()
    masks = masks_for(w, list(WORKLOADS).index(name))
    incs = (False, True) if w.scatter else (False,)
    for inc in incs:
        for plans in ((None, True) if w.dtype == "bf16" else (None,)):
            for batched in (False, True):
                ref = run_stack(w, dev, "python", side, inc, plans, masks, batched)
                got = run_stack(w, dev, "native", side, inc, plans, masks, batched)
                assert_same(got, ref, (name, side, inc, plans, batched))


def test_stack_outputs_match_oracle(dev):
    """The native pipelined stack on the density-sweep shape at 5% (24
    bodies): after four fed batches, the last batch's compaction, dense
    output and pool against the oracle's; the layer rows on sampled rows
    at the layer tolerance is covered by the layer tests, here the scatter
    and pool of the kernel's rows must be exact."""
    w = synth.workload_c4(0.05, B=24)
    masks = masks_for(w, 5)[:3]
    st = SparseStack(w, device=dev, side_stream=True, incremental_scatter=True)
    md = [torch.from_numpy(m).to(dev) for m in masks]

    def feed(k):
        st.mask.copy_(md[k])

    n = st.run(3, feed=feed)
    torch.cuda.synchronize()
    coords, inv, row_ptr, n_ref = O.compact(masks[-1].reshape(w.B, w.V))
    assert n == n_ref
    assert np.array_equal(st.coords[:n].cpu().numpy(), coords)
    assert np.array_equal(st.inv.cpu().numpy(), inv)
    rows = st.acts[-1][:n].float().cpu().numpy().astype(np.float64)
    dense = st.dense_out.float().cpu().numpy().astype(np.float64)
    assert np.array_equal(dense, O.scatter(rows, inv, zero_fill=True))
    pooled = st.pooled.float().cpu().numpy().astype(np.float64)
    assert np.array_equal(pooled, O.segment_max(rows, row_ptr, 0.0))


def test_split_conv_layers_in_stack_match_oracle(dev):
    """The sequence workload's stack (256-channel convs, which take the split
    conv by default at this density) on a small batch, pipelined: every
    layer's rows against the oracle's conv of that layer's own input rows,
    on sampled rows at the layer bound."""
    w = synth.workload_c5(4, 8)
    st = SparseStack(w, device=dev, side_stream=True)
    assert sorted(st.split_rows) == [0, 1, 2]
    n = st.run(2)
    torch.cuda.synchronize()
    assert 0 < n <= min(st.split_rows.values())
    coords = st.coords[:n].cpu().numpy()
    rows = np.random.default_rng(3).choice(n, size=min(n, 400), replace=False)
    for l, spec in enumerate(w.layers):
        S = st.acts[l][:n].float().cpu().numpy().astype(np.float64)
        got = st.acts[l + 1][:n].float().cpu().numpy().astype(np.float64)
        ref = O.conv_at(S, coords, w.B, w.V, w.nbr, spec.W, rows, spec.bias, act=spec.relu)
        scale = O.conv_at(S, coords, w.B, w.V, w.nbr, spec.W, rows, spec.bias, scale=True)
        assert_scaled_close(got[rows], ref, scale, "bf16", f"stack layer {l}",
                            n_terms=w.K * spec.Cin)


def test_native_time_events_and_feed_errors(dev):
    w = synth.workload_c4(0.05, B=8)
    st = SparseStack(w, device=dev, side_stream=True)
    steps = 6
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          if k % 2 == 0 else (None, None) for k in range(steps)]
    st.run(steps, around_layer=(1, ev))
    torch.cuda.synchronize()
    for a, b in ev[::2]:
        assert a.elapsed_time(b) > 0

    class Stop(Exception):
        pass

    def feed(k):
        if k == 2:
            raise Stop()

    with pytest.raises(Stop):
        st.run(5, feed=feed)
    torch.cuda.synchronize()
    # the stack still runs afterwards
    n = st.run(2)
    torch.cuda.synchronize()
    assert n == int(np.count_nonzero(w.mask))


def test_create_refuses_plan_misuse(dev):
    """Plan buffers on the device: below a plan's size, shared by layers of
    different shapes, or shared differently in another index set."""
    w = synth.workload_c2()
    st = SparseStack(w, device=dev, side_stream=True, conv_plans=True, packed_conv=False)
    base = st._native._desc
    planned = [l for l in range(len(w.layers)) if base.sets[0].plan[l]]
    assert len(planned) >= 2

    def create(d):
        return shc.StackExecutor(d, ())

    d = shc.StackDesc.from_buffer_copy(base)
    d.sets[1].plan_bytes[planned[0]] = 16
    with pytest.raises(shc.ShcError, match="CAPACITY"):
        create(d)
    d = shc.StackDesc.from_buffer_copy(base)
    for s in range(3):
        d.sets[s].plan[planned[1]] = d.sets[s].plan[planned[0]]
        d.sets[s].plan_bytes[planned[1]] = d.sets[s].plan_bytes[planned[0]]
    if (d.layers[planned[0]].Cin, d.layers[planned[0]].Cout) != \
            (d.layers[planned[1]].Cin, d.layers[planned[1]].Cout):
        with pytest.raises(shc.ShcError, match="share a plan"):
            create(d)
    d = shc.StackDesc.from_buffer_copy(base)
    d.layers[planned[0]].plan_rows = shc.load().shc_conv_plan_max_rows(
        w.K, d.layers[planned[0]].Cin, d.layers[planned[0]].Cout, shc.SHC_BF16) + 1
    with pytest.raises(shc.ShcError, match="UNSUPPORTED"):
        create(d)
    d = shc.StackDesc.from_buffer_copy(base)
    pageable = torch.zeros(1, dtype=torch.int64)
    d.sets[1].host_count = pageable.data_ptr()
    with pytest.raises(shc.ShcError, match="page-locked"):
        create(d)
    torch.cuda.synchronize()
