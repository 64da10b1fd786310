"""The sparse neighbour conv with pre-arranged weights held in registers
(shc_pack_conv_weights + shc_sparse_neighbor_conv_packed): Eqs. 4-5 with
Eq. 10's activation against the oracle on sampled rows, at the derived bf16
bound, with and without bias and ReLU, rows past N' untouched.  Shapes: every
channel pair the call takes (64, 128), one, five and nine slots, a partial
16-row block, sparse and dense masks (dense ones stage their out-of-chunk
neighbour rows in several rounds and walk several chunks per workgroup),
slot 0 the vertex itself, another vertex, or absent, the density-sweep batch
at full size on the ellipsoid k-NN mesh, two calls in a row, and the errors.
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


def rand_nbr(V, K, rng, p_missing=0.1, slot0="self"):
    nbr = rng.integers(0, V, size=(V, K)).astype(np.int32)
    nbr[rng.random((V, K)) < p_missing] = -1
    if slot0 == "self":
        nbr[:, 0] = np.arange(V)
    elif slot0 == "absent":
        nbr[rng.random(V) < 0.3, 0] = -1   # slot 0 missing for some vertices
    return nbr


def packed(W, dev):
    K, Cin, Cout = W.shape
    nb = shc.conv_packed_weights_bytes(K, Cin, Cout)
    assert nb == K * Cin * Cout * 2
    Wp = torch.empty(nb, dtype=torch.uint8, device=dev)
    shc.pack_conv_weights(up(W, "bf16"), Wp)
    return Wp


def check_packed(dev, B, V, K, Cin, Cout, p, nbr, seed, extra_rows=3, n_sample=300,
                 m=None):
    rng = np.random.default_rng(seed)
    if m is None:
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
    rows = np.unique(np.concatenate([np.arange(min(n, 150)), np.arange(max(0, n - 150), n),
                                     rng.choice(n, size=min(n, n_sample), replace=False)]))
    Wp = packed(W, dev)
    Sd = up(S, "bf16")
    for b, act in ((bias, shc.SHC_ACT_RELU), (None, shc.SHC_ACT_NONE)):
        out = torch.full((n + extra_rows, Cout), float("nan"), dtype=torch.bfloat16, device=dev)
        shc.sparse_neighbor_conv_packed(Sd, table, n, Wp, K, Cin, Cout,
                                        None if b is None else up(b), out, act)
        got = down(out)
        assert np.all(np.isnan(got[n:]))
        if n == 0:
            continue
        ref = O.conv_at(S, coords, B, V, nbr, W, rows, b, act=act == shc.SHC_ACT_RELU)
        scale = O.conv_at(S, coords, B, V, nbr, W, rows, b, scale=True)
        assert_scaled_close(got[rows], ref, scale, "bf16",
                            f"packed conv K={K} {Cin}->{Cout} p={p} act={act}", n_terms=K * Cin)
    torch.cuda.synchronize()
    return n


@pytest.mark.parametrize("B,V,K,Cin,Cout,p,slot0", [
    (64, 655, 9, 128, 128, 0.1, "self"),
    (16, 655, 9, 64, 64, 0.1, "self"),
    (16, 655, 9, 64, 128, 0.2, "self"),
    (16, 655, 9, 128, 64, 0.2, "self"),
    (6, 700, 5, 64, 128, 0.4, "self"),       # five slots
    (2, 300, 1, 128, 64, 0.6, "self"),       # one slot
    (1, 40, 9, 128, 128, 0.5, "self"),       # one partial 16-row block
    (8, 655, 9, 128, 128, 0.9, "self"),      # dense: several staging rounds
    (24, 4000, 9, 128, 128, 1.0, "self"),    # full mesh: several chunks per workgroup
    (24, 4000, 9, 64, 64, 1.0, "self"),
    (8, 655, 9, 128, 128, 0.3, "other"),     # slot 0 another vertex: staged or from the chunk
    (8, 655, 9, 64, 64, 0.3, "absent"),      # slot 0 absent for some rows
])
def test_packed_conv_against_oracle(dev, B, V, K, Cin, Cout, p, slot0):
    rng = np.random.default_rng(B * 37 + V + K + Cin + 5 * Cout)
    nbr = rand_nbr(V, K, rng, slot0=slot0)
    check_packed(dev, B, V, K, Cin, Cout, p, nbr, seed=B + V + K + 1)


@pytest.mark.parametrize("p", [0.01, 0.05, 0.2])
def test_packed_conv_density_sweep_batch(dev, p):
    """The density-sweep batch (B = 128, V = 10475, 128 -> 128) on the
    ellipsoid k-NN mesh, Bernoulli masks."""
    _, nbr = synth.mesh("ellipsoid", 10475, 9, 4)
    n = check_packed(dev, 128, 10475, 9, 128, 128, p, np.ascontiguousarray(nbr, np.int32),
                     int(p * 1000) + 3)
    assert n > 0.8 * p * 128 * 10475


def test_packed_conv_full_mesh_contact_mask(dev):
    """The full-resolution body mesh's contact mask (y < -0.6 plus 2% noise,
    about 5% active, B = 256) at 64 -> 64: many rows whose neighbours lie in
    the same chunk."""
    w = synth.workload_c3(dtype="bf16", five_percent=True)
    check_packed(dev, w.B, w.V, 9, 64, 64, None, np.ascontiguousarray(w.nbr, np.int32), 17,
                 m=w.mask)


def test_packed_conv_empty_and_repeat(dev):
    """N' = 0 writes nothing; two calls in a row on one output, the second
    with fewer rows, are each right."""
    rng = np.random.default_rng(6)
    nbr = rand_nbr(300, 9, rng)
    assert check_packed(dev, 2, 300, 9, 128, 128, 0.0, nbr, 5) == 0
    V, K, C = 655, 9, 128
    nbr = rand_nbr(V, K, rng)
    W = synth.as_dtype((rng.standard_normal((K, C, C)) / np.sqrt(K * C)).astype(np.float32),
                       "bf16")[1]
    Wp = packed(W, dev)
    out = torch.empty((20 * V, C), dtype=torch.bfloat16, device=dev)
    for B, p in ((20, 0.3), (6, 0.1)):
        m = (rng.random((B, V)) < p).astype(np.uint8)
        c = Compaction(m)
        n = c.run()
        table = torch.empty(K * n, dtype=torch.int32, device=dev)
        shc.build_neighbor_table(c.coords, c.inv, n, B, V, up(nbr), table)
        S = synth.as_dtype(rng.standard_normal((n, C)).astype(np.float32), "bf16")[1]
        shc.sparse_neighbor_conv_packed(up(S, "bf16"), table, n, Wp, K, C, C, None, out,
                                        shc.SHC_ACT_NONE)
        coords = O.compact(m)[0]
        rows = np.arange(n)
        ref = O.conv_at(S, coords, B, V, nbr, W, rows)
        scale = O.conv_at(S, coords, B, V, nbr, W, rows, scale=True)
        assert_scaled_close(down(out)[:n], ref, scale, "bf16", f"repeat B={B}", n_terms=K * C)
    torch.cuda.synchronize()


def test_packed_conv_errors_on_device(dev):
    """Unsupported shapes and dtypes and a short packed buffer are refused."""
    W = torch.zeros((9, 128, 128), dtype=torch.bfloat16, device=dev)
    small = torch.empty(shc.conv_packed_weights_bytes(9, 128, 128) - 16, dtype=torch.uint8,
                        device=dev)
    with pytest.raises(shc.ShcError, match="CAPACITY"):
        shc.pack_conv_weights(W, small)
    with pytest.raises(shc.ShcError, match="UNSUPPORTED"):
        shc.pack_conv_weights(W.float(), small)
    assert shc.conv_packed_weights_bytes(10, 128, 128) == 0
    assert shc.conv_packed_weights_bytes(9, 256, 128) == 0
    assert shc.conv_packed_weights_bytes(9, 128, 128, shc.SHC_F32) == 0
    S = torch.zeros((10, 256), dtype=torch.bfloat16, device=dev)
    table = torch.zeros(9 * 10, dtype=torch.int32, device=dev)
    out = torch.empty((10, 128), dtype=torch.bfloat16, device=dev)
    with pytest.raises(shc.ShcError, match="UNSUPPORTED"):
        shc.sparse_neighbor_conv_packed(S, table, 10, small, 9, 256, 128, None, out)


@pytest.mark.parametrize("executor", ["native", "python"])
def test_packed_stack_against_oracle(dev, executor):
    """The density-sweep stack (gather + linear, conv, scatter, pool) at 5% on
    24 bodies with the conv layer on the packed conv: the conv output against
    the oracle's stack at the derived bf16 bound, over two batches."""
    from paper_2608_09388_amd.pipeline import SparseStack
    w = synth.workload_c4(0.05, B=24)
    st = SparseStack(w, device=dev, side_stream=True, executor=executor)
    assert 1 in st.packed_rows
    for k in range(2):
        m = (np.random.default_rng(90 + k).random((w.B, w.V)) < 0.04 + 0.02 * k).astype(np.uint8)
        st.mask.copy_(torch.from_numpy(m.reshape(-1)).to(dev))
        n = st.run(1)
        torch.cuda.synchronize()
        coords = O.compact(m)[0]
        assert n == len(coords)
        S = down(st.acts[1][:n])
        rows = np.random.default_rng(k).choice(n, size=min(n, 400), replace=False)
        ref = O.conv_at(S, coords, w.B, w.V, w.nbr, w.layers[1].W, rows, None, act=True)
        scale = O.conv_at(S, coords, w.B, w.V, w.nbr, w.layers[1].W, rows, None, scale=True)
        assert_scaled_close(down(st.acts[2][:n])[rows], ref, scale, "bf16",
                            f"packed stack batch {k}", n_terms=9 * 128)


@pytest.mark.parametrize("B,V,K,Cin,Cout,p,slot0", [
    (64, 655, 9, 128, 128, 0.1, "self"),
    (16, 655, 9, 64, 64, 0.1, "self"),
    (16, 655, 9, 64, 128, 0.2, "self"),
    (6, 700, 5, 128, 64, 0.4, "self"),
    (1, 40, 9, 128, 128, 0.5, "self"),
    (8, 655, 9, 128, 128, 0.9, "self"),      # several staging rounds
    (24, 4000, 9, 128, 128, 1.0, "self"),    # several chunks per workgroup
    (8, 655, 9, 128, 128, 0.3, "other"),
    (8, 655, 9, 64, 64, 0.3, "absent"),
])
def test_packed_plan_matches_packed(dev, B, V, K, Cin, Cout, p, slot0):
    """The planned packed conv (shc_build_conv_packed_plan, then
    shc_sparse_neighbor_conv_packed_planned) writes exactly what the packed
    conv writes from the table, with and without bias and ReLU; and it is
    within the derived bound of the oracle on sampled rows."""
    rng = np.random.default_rng(B * 13 + V + K + Cin + 7 * Cout)
    nbr = rand_nbr(V, K, rng, slot0=slot0)
    m = (rng.random((B, V)) < p).astype(np.uint8)
    c = Compaction(m)
    n = c.run()
    table = torch.empty(K * n, dtype=torch.int32, device=dev)
    shc.build_neighbor_table(c.coords, c.inv, n, B, V, up(nbr), table)
    S = synth.as_dtype(rng.standard_normal((n, Cin)).astype(np.float32), "bf16")[1]
    W = synth.as_dtype((rng.standard_normal((K, Cin, Cout)) / np.sqrt(K * Cin))
                       .astype(np.float32), "bf16")[1]
    bias = up(rng.standard_normal(Cout).astype(np.float32))
    Wp, Sd = packed(W, dev), up(S, "bf16")
    plan = torch.empty(shc.conv_packed_plan_bytes(B * V, K, Cin, Cout), dtype=torch.uint8,
                       device=dev)
    plan.fill_(0xA5)   # garbage before the build
    shc.build_conv_packed_plan(table, n, K, Cin, Cout, plan)
    for b, act in ((bias, shc.SHC_ACT_RELU), (None, shc.SHC_ACT_NONE)):
        o1 = torch.full((n + 2, Cout), float("nan"), dtype=torch.bfloat16, device=dev)
        o2 = o1.clone()
        shc.sparse_neighbor_conv_packed(Sd, table, n, Wp, K, Cin, Cout, b, o1, act)
        shc.sparse_neighbor_conv_packed_planned(Sd, plan, n, Wp, K, Cin, Cout, b, o2, act)
        torch.cuda.synchronize()
        assert torch.equal(o1[:n], o2[:n]), f"planned != packed K={K} {Cin}->{Cout} p={p}"
        assert torch.isnan(o2[n:].float()).all()
    coords = O.compact(m)[0]
    rows = rng.choice(n, size=min(n, 200), replace=False)
    ref = O.conv_at(S, coords, B, V, nbr, W, rows)
    scale = O.conv_at(S, coords, B, V, nbr, W, rows, scale=True)
    assert_scaled_close(down(o2)[rows], ref, scale, "bf16", "planned packed conv",
                        n_terms=K * Cin)


def test_packed_plan_other_row_count_and_errors(dev):
    """A plan of another row count writes nothing (every chunk's header
    disagrees); a plan buffer below the call's size is refused."""
    rng = np.random.default_rng(21)
    B, V, K, C = 8, 655, 9, 128
    nbr = rand_nbr(V, K, rng)
    m = (rng.random((B, V)) < 0.2).astype(np.uint8)
    c = Compaction(m)
    n = c.run()
    table = torch.empty(K * n, dtype=torch.int32, device=dev)
    shc.build_neighbor_table(c.coords, c.inv, n, B, V, up(nbr), table)
    plan = torch.empty(shc.conv_packed_plan_bytes(B * V, K, C, C), dtype=torch.uint8, device=dev)
    shc.build_conv_packed_plan(table, n, K, C, C, plan)
    W = torch.zeros((K, C, C), dtype=torch.bfloat16, device=dev)
    Wp = packed(W.cpu().float().numpy(), dev)
    S = torch.zeros((n, C), dtype=torch.bfloat16, device=dev)
    out = torch.full((n, C), 7.0, dtype=torch.bfloat16, device=dev)
    shc.sparse_neighbor_conv_packed_planned(S, plan, n - 5, Wp, K, C, C, None, out)
    torch.cuda.synchronize()
    assert (out.float() == 7.0).all()
    small = plan[:16]
    with pytest.raises(shc.ShcError, match="CAPACITY"):
        shc.build_conv_packed_plan(table, n, K, C, C, small)
    with pytest.raises(shc.ShcError, match="CAPACITY"):
        shc.sparse_neighbor_conv_packed_planned(S, small, n, Wp, K, C, C, None, out)
