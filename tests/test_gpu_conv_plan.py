"""The conv plan of an active set (shc_build_conv_plan and
shc_sparse_neighbor_conv_planned): a planned layer must give exactly the
output of the conv from the table on the same inputs (Eqs. 4-5), and the
oracle's values on sampled rows.  Every input is seeded and synthetic.
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


def bf16(a):
    return synth.as_dtype(np.asarray(a, np.float32), "bf16")[1]


def setup(dev, B, V, K, Cin, p, seed):
    """Mask, neighbours, compaction and table on the device, bf16 input rows."""
    rng = np.random.default_rng(seed)
    m = (rng.random((B, V)) < p).astype(np.uint8)
    nbr = rand_nbr(V, K, rng)
    c = Compaction(m)
    n = c.run()
    table = torch.full((max(K * n, 1),), -7, dtype=torch.int32, device=dev)
    shc.build_neighbor_table(c.coords, c.inv, n, B, V, up(nbr), table)
    S = bf16(rng.standard_normal((n, Cin)))
    return rng, m, nbr, n, table, S


def weights(rng, K, Cin, Cout):
    W = bf16(rng.standard_normal((K, Cin, Cout)) / np.sqrt(K * Cin))
    return W, rng.standard_normal(Cout).astype(np.float32)


def plan_for(dev, table, n, K, Cin, Cout, extra=0):
    nb = shc.conv_plan_bytes(n, K, Cin, Cout)
    assert nb > 0, (n, K, Cin, Cout)
    plan = torch.full((nb + extra,), 0xA5, dtype=torch.uint8, device=dev)
    shc.build_conv_plan(table, n, K, Cin, Cout, plan)
    return plan


def both(dev, S, table, plan, n, W, bias, act=shc.SHC_ACT_RELU):
    """(table conv, planned conv) outputs, rows past n checked untouched."""
    K, Cin, Cout = W.shape
    Sd, Wd, bd = up(S, "bf16"), up(W, "bf16"), None if bias is None else up(bias)
    outs = []
    for path in ("table", "planned"):
        out = torch.full((n + 2, Cout), float("nan"), dtype=torch.bfloat16, device=dev)
        if path == "table":
            shc.sparse_neighbor_conv_table(Sd, table, n, Wd, bd, out, act)
        else:
            shc.sparse_neighbor_conv_planned(Sd, plan, n, Wd, bd, out, act)
        got = down(out)
        assert np.all(np.isnan(got[n:])), path
        outs.append(got[:n])
    return outs


@pytest.mark.parametrize("B,V,K,Cin,Cout,p,planned", [
    (3, 200, 9, 128, 128, 0.3, True),    # a few rows per workgroup, ragged tail
    (2, 500, 9, 64, 64, 0.5, True),
    (4, 150, 4, 32, 32, 0.4, True),
    (1, 300, 1, 32, 32, 0.6, True),      # one slot
    (2, 700, 10, 64, 192, 0.7, True),    # ten slots, three column slices of 64
    (6, 2000, 10, 64, 64, 0.3, True),
    (4, 3000, 9, 128, 128, 0.05, True),
    (40, 10475, 9, 128, 128, 0.05, True),
    (128, 10475, 9, 128, 128, 0.05, True),  # the density-sweep batch at 5%
    # shapes without a plan: more slots than the kernel takes, a column slice
    # wider than Cout, Cin of one 32-byte k-step
    (2, 100, 32, 16, 16, 0.7, False),
    (1, 300, 1, 32, 16, 0.6, False),
    (2, 300, 9, 16, 64, 0.5, False),
])
def test_planned_equals_table_and_oracle(dev, B, V, K, Cin, Cout, p, planned):
    rng, m, nbr, n, table, S = setup(dev, B, V, K, Cin, p, B * 31 + V + K * 7 + Cout)
    W, bias = weights(rng, K, Cin, Cout)
    nb = shc.conv_plan_bytes(n, K, Cin, Cout)
    if not planned:
        # a shape the planned kernel does not take: no plan, and the planned
        # call says so
        assert nb == 0
        plan = torch.zeros(4096, dtype=torch.uint8, device=dev)
        out = torch.zeros((n, Cout), dtype=torch.bfloat16, device=dev)
        with pytest.raises(shc.ShcError, match="UNSUPPORTED"):
            shc.sparse_neighbor_conv_planned(up(S, "bf16"), plan, n, up(W, "bf16"), None, out)
        return
    plan = plan_for(dev, table, n, K, Cin, Cout)
    for b, act in ((bias, shc.SHC_ACT_RELU), (None, shc.SHC_ACT_NONE)):
        g_tab, g_plan = both(dev, S, table, plan, n, W, b, act)
        assert np.array_equal(g_tab, g_plan), f"planned != table, K={K} {Cin}->{Cout} p={p}"
    coords, _, _, n_ref = O.compact(m)
    assert n_ref == n
    rows = np.unique(np.concatenate([np.arange(min(n, 300)), np.arange(max(0, n - 300), n),
                                     rng.choice(n, size=min(n, 400), replace=False)]))
    ref = O.conv_at(S, coords, B, V, nbr, W, rows, None, act=False)
    scale = O.conv_at(S, coords, B, V, nbr, W, rows, None, scale=True)
    assert_scaled_close(g_plan[rows], ref, scale, "bf16", f"planned conv K={K} {Cin}->{Cout}",
                        n_terms=K * Cin)


def test_one_plan_serves_a_stack_of_layers(dev):
    """Three conv layers of one shape on one active set, chained, from one
    plan: every layer's output equals the table path's."""
    K, C = 9, 128
    rng, m, nbr, n, table, S = setup(dev, 16, 10475, K, C, 0.05, 5)
    plan = plan_for(dev, table, n, K, C, C)
    x_tab = up(S, "bf16")
    x_plan = x_tab.clone()
    for layer in range(3):
        W, bias = weights(rng, K, C, C)
        Wd, bd = up(W, "bf16"), up(bias)
        y_tab = torch.empty((n, C), dtype=torch.bfloat16, device=dev)
        y_plan = torch.empty_like(y_tab)
        shc.sparse_neighbor_conv_table(x_tab, table, n, Wd, bd, y_tab)
        shc.sparse_neighbor_conv_planned(x_plan, plan, n, Wd, bd, y_plan)
        assert torch.equal(y_tab, y_plan), f"layer {layer}"
        x_tab, x_plan = y_tab, y_plan


def test_plan_buffer_reused_for_a_smaller_set(dev):
    """A plan buffer sized for a larger active set, rebuilt for a smaller one
    (stale bytes past the new plan), and prepared calls with n_rows per call."""
    K, C = 9, 128
    rng, m1, nbr, n1, table1, S1 = setup(dev, 24, 10475, K, C, 0.06, 11)
    nb1 = shc.conv_plan_bytes(n1, K, C, C)
    plan = torch.full((nb1 + 4096,), 0x5A, dtype=torch.uint8, device=dev)
    W, bias = weights(rng, K, C, C)
    for n, table, S in ((n1, table1, S1),):
        shc.build_conv_plan(table, n, K, C, C, plan)
        g_tab, g_plan = both(dev, S, table, plan, n, W, bias)
        assert np.array_equal(g_tab, g_plan)
    # a smaller set: rows drawn at a lower density on fewer bodies
    rng2, m2, nbr2, n2, table2, S2 = setup(dev, 10, 10475, K, C, 0.03, 12)
    assert 0 < n2 < n1 and shc.conv_plan_bytes(n2, K, C, C) <= plan.numel()
    shc.build_conv_plan(table2, n2, K, C, C, plan)
    g_tab, g_plan = both(dev, S2, table2, plan, n2, W, bias)
    assert np.array_equal(g_tab, g_plan)
    # prepared calls, n_rows given per call
    Sd = up(S2, "bf16")
    out_p = torch.full((n1, C), float("nan"), dtype=torch.bfloat16, device=dev)
    out_t = torch.full((n1, C), float("nan"), dtype=torch.bfloat16, device=dev)
    build = shc.prepare_build_conv_plan(table2, K, C, C, plan)
    conv = shc.prepare_sparse_neighbor_conv_planned(Sd, plan, up(W, "bf16"), up(bias), out_p)
    plan.fill_(0)
    build(n2)
    conv(n2)
    shc.sparse_neighbor_conv_table(Sd, table2, n2, up(W, "bf16"), up(bias), out_t)
    assert torch.equal(out_p[:n2], out_t[:n2])
    assert torch.isnan(out_p[n2:].float()).all()


def test_plan_errors(dev):
    K, C = 9, 128
    rng, m, nbr, n, table, S = setup(dev, 3, 2000, K, C, 0.2, 3)
    nb = shc.conv_plan_bytes(n, K, C, C)
    assert nb > 0 and nb % 1024 == 0
    assert shc.conv_plan_bytes(n, K, C, C, shc.SHC_F32) == 0   # bf16 only
    assert shc.conv_plan_bytes(0, K, C, C) == 0
    small = torch.zeros(1024, dtype=torch.uint8, device=dev)
    with pytest.raises(shc.ShcError, match="CAPACITY"):
        shc.build_conv_plan(table, n, K, C, C, small)
    W, _ = weights(rng, K, C, C)
    out = torch.zeros((n, C), dtype=torch.bfloat16, device=dev)
    with pytest.raises(shc.ShcError, match="CAPACITY"):
        shc.sparse_neighbor_conv_planned(up(S, "bf16"), small, n, up(W, "bf16"), None, out)
    plan = torch.zeros(nb, dtype=torch.uint8, device=dev)
    with pytest.raises(shc.ShcError, match="UNSUPPORTED"):
        shc.sparse_neighbor_conv_planned(up(S, "f32"), plan, n, up(W, "f32"), None,
                                         out.float())
    # zero rows: a no-op that touches nothing
    shc.build_conv_plan(table, 0, K, C, C, plan)
    shc.sparse_neighbor_conv_planned(up(S, "bf16"), plan, 0, up(W, "bf16"), None, out)
    torch.cuda.synchronize()
    assert int(plan.sum().item()) == 0


def test_plan_row_limit(dev):
    """A plan exists for every row count up to shc_conv_plan_max_rows and for
    none past it; a buffer of shc_conv_plan_bytes(n) holds the plan of every
    smaller count (checked at the counts where the rows per group step up)."""
    K, C = 9, 128
    n_lim = shc.conv_plan_max_rows(K, C, C)
    assert n_lim > 0
    assert shc.conv_plan_max_rows(K, C, C, shc.SHC_F32) == 0
    assert shc.conv_plan_max_rows(32, C, C) == 0
    table = torch.full((K * (n_lim + 1),), -1, dtype=torch.int32, device=dev)
    nb = shc.conv_plan_bytes(n_lim, K, C, C)
    assert nb == shc.conv_plan_bytes(n_lim + 1000, K, C, C)   # nothing past the limit
    plan = torch.empty(nb, dtype=torch.uint8, device=dev)
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    counts = {1, 2, 17, n_lim - 1, n_lim}
    for r in range(64, 1536 + 1, 16):    # the last count of every rows-per-group step
        counts.update(c for c in (r * cus // 4, r * cus // 4 + 1) if 0 < c <= n_lim)
    sizes = []
    for n in sorted(counts):
        sizes.append(shc.conv_plan_bytes(n, K, C, C))
        shc.build_conv_plan(table, n, K, C, C, plan)      # raises if the plan did not fit
    assert sizes == sorted(sizes)                         # a bound over all smaller counts
    with pytest.raises(shc.ShcError, match="UNSUPPORTED"):
        shc.build_conv_plan(table, n_lim + 1, K, C, C, plan)
    torch.cuda.synchronize()


@pytest.mark.parametrize("side", [False, True])
def test_stack_with_plans_matches_without(dev, side):
    """The density-sweep stack (gather + linear, conv, scatter, pool) at 5% on
    24 bodies, with and without conv plans: every output identical, over
    three batches with a new mask each."""
    from paper_2608_09388_amd.pipeline import SparseStack
    w = synth.workload_c4(0.05, B=24)
    outs = {}
    for use in (False, True):
        st = SparseStack(w, device=dev, side_stream=side, conv_plans=use, packed_conv=False)
        assert bool(st.plan_shapes) == use
        masks = [np.random.default_rng(40 + k).random(w.B * w.V) < 0.03 + 0.02 * k
                 for k in range(3)]

        def feed(k):
            st.mask.copy_(torch.from_numpy(masks[k].astype(np.uint8)).to(dev))

        n = st.run(3, feed=feed)
        torch.cuda.synchronize()
        outs[use] = (n, st.acts[-1][:n].clone(), st.dense_out.clone(), st.pooled.clone())
    assert outs[False][0] == outs[True][0]
    for a, b in zip(outs[False][1:], outs[True][1:]):
        assert torch.equal(a, b)


@pytest.mark.parametrize("side", [False, True])
def test_encoder_stack_mixed_plans(dev, side):
    """The 4-layer encoder (conv 16 -> 64 -> 64 -> 128 -> 128 on 64 small
    bodies, max-pool): with plans forced on, the layers whose shape takes one
    read it and the first (C_in = 16) runs from the table; every output
    identical to the stack without plans, over three batches."""
    from paper_2608_09388_amd.pipeline import SparseStack
    w = synth.workload_c2()
    outs = {}
    for use in (False, True):
        st = SparseStack(w, device=dev, side_stream=side, conv_plans=use, packed_conv=False)
        if use:
            assert (9, 16, 64) not in st.plan_shapes
            assert {(9, 64, 64), (9, 64, 128), (9, 128, 128)} <= set(st.plan_shapes)
        masks = [np.random.default_rng(70 + k).random(w.B * w.V) < 0.06 + 0.04 * k
                 for k in range(3)]

        def feed(k):
            st.mask.copy_(torch.from_numpy(masks[k].astype(np.uint8)).to(dev))

        n = st.run(3, feed=feed)
        torch.cuda.synchronize()
        outs[use] = (n, [a[:n].clone() for a in st.acts[1:]], st.pooled.clone())
    assert outs[False][0] == outs[True][0]
    for a, b in zip(outs[False][1], outs[True][1]):
        assert torch.equal(a, b)
    assert torch.equal(outs[False][2], outs[True][2])
