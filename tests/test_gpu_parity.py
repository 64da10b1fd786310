"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Bit-exact: compaction (coords, inv, row_ptr, count), gather, scatter, pool.
Floating point: |gpu - oracle| <= rtol * (abs-sum scale) per element, with
rtol 1e-5 for fp32 and 2e-2 for bf16; stacks are also checked normwise.
Every input is seeded and synthetic; no expected value comes from the GPU.
"""
import numpy as np
import pytest
import torch

from oracle import shc_oracle as O
from paper_2608_09388_amd import binding as shc
from paper_2608_09388_amd import synth
from tests.gpu_util import (TORCH, Compaction, assert_gn_close, assert_normwise_close,
                            assert_scaled_close, down, gn_floor, require_gpu, up)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


def rand_nbr(V, K, rng, p_missing=0.1):
    nbr = rng.integers(0, V, size=(V, K)).astype(np.int32)
    nbr[rng.random((V, K)) < p_missing] = -1
    nbr[:, 0] = np.arange(V)
    return nbr


def check_compaction(mask, cap=None):
    ref_c, ref_inv, ref_rp, ref_n = O.compact(mask)
    c = Compaction(mask, cap)
    n = c.run(want_host=(cap is None))
    torch.cuda.synchronize()
    n_dev = int(c.n_dev[0].item())
    assert n_dev == ref_n
    if cap is None:
        assert n == ref_n
    assert np.array_equal(down(c.inv), ref_inv)
    assert np.array_equal(down(c.row_ptr), ref_rp)
    k = min(ref_n, c.cap)
    got_c = down(c.coords)
    assert np.array_equal(got_c[:k], ref_c[:k])
    assert np.all(got_c[k:] == -7)          # rows past N' (or past cap) untouched
    return c


# ----------------------------------------------------------------------------
# compaction
# ----------------------------------------------------------------------------


def test_compact_exhaustive_v10(dev):
    """All 2^10 masks of one V = 10 body at once: body b carries the bits of b."""
    codes = np.arange(1 << 10)
    mask = ((codes[:, None] >> np.arange(10)[None, :]) & 1).astype(np.uint8)
    check_compaction(mask)


def test_compact_exhaustive_v12(dev):
    codes = np.arange(1 << 12)
    mask = ((codes[:, None] >> np.arange(12)[None, :]) & 1).astype(np.uint8)
    check_compaction(mask)


@pytest.mark.parametrize("B,V,p", [(1, 1, 1.0), (1, 1, 0.0), (3, 1, 0.5), (2, 3, 0.5),
                                   (1, 4095, 0.3), (1, 4096, 0.3), (1, 4097, 0.3),
                                   (7, 655, 0.1), (64, 655, 0.0), (64, 655, 1.0),
                                   (5, 10475, 0.05), (1025, 4096, 0.02), (300, 10475, 0.5)])
def test_compact_shapes(dev, B, V, p):
    rng = np.random.default_rng(B * 7919 + V)
    m = (rng.random((B, V)) < p).astype(np.uint8)
    m[m != 0] = rng.integers(1, 256, size=int(m.sum()))   # any non-zero byte is active
    check_compaction(m)


@pytest.mark.parametrize("pinned", [True, False])
def test_compact_host_count_tensor(dev, pinned):
    """The count lands in a caller's host tensor: written by the kernel itself
    when the tensor is page-locked, copied back when it is pageable; a second
    mask with fewer rows overwrites the first count."""
    rng = np.random.default_rng(91)
    for B, V, p in [(16, 10475, 0.05), (3, 655, 0.01)]:
        m = (rng.random((B, V)) < p).astype(np.uint8)
        ref_c, ref_inv, ref_rp, ref_n = O.compact(m)
        c = Compaction(m)
        hc = torch.full((1,), -1, dtype=torch.int64, pin_memory=pinned)
        n = shc.compact_mask(c.mask, B, V, c.coords, c.inv, c.row_ptr, c.n_dev, c.ws,
                             host_count=hc)
        assert n == ref_n and int(hc[0]) == ref_n
        assert np.array_equal(down(c.inv), ref_inv)
        assert np.array_equal(down(c.coords)[:ref_n], ref_c)


def test_compact_prepared_pinned(dev):
    """The prepared compaction (pinned count, as the pipeline runs it) over
    three masks in a row of decreasing size."""
    rng = np.random.default_rng(92)
    B, V = 32, 10475
    c = Compaction(np.zeros((B, V), np.uint8))
    call = shc.PreparedCompact(c.mask, B, V, c.coords, c.inv, c.row_ptr, c.n_dev, c.ws)
    for p in (0.2, 0.05, 0.0):
        m = (rng.random((B, V)) < p).astype(np.uint8)
        c.mask.copy_(up(m.reshape(-1)))
        ref_c, ref_inv, ref_rp, ref_n = O.compact(m)
        assert call() == ref_n
        assert np.array_equal(down(c.inv), ref_inv)
        assert np.array_equal(down(c.row_ptr), ref_rp)
        assert np.array_equal(down(c.coords)[:ref_n], ref_c)


def test_compact_start_wait(dev):
    """The two halves of the compaction with work enqueued between them (the
    zeros of a dense output): same outputs as the oracle over three masks in a
    row of decreasing size, through the prepared call and the plain wrappers."""
    rng = np.random.default_rng(93)
    B, V, C = 24, 10475, 16
    c = Compaction(np.zeros((B, V), np.uint8))
    call = shc.PreparedCompact(c.mask, B, V, c.coords, c.inv, c.row_ptr, c.n_dev, c.ws)
    D = torch.full((B * V, C), float("nan"), dtype=torch.float32, device=dev)
    hc = torch.full((1,), -5, dtype=torch.int64, pin_memory=True)
    for p in (0.3, 0.05, 0.0):
        m = (rng.random((B, V)) < p).astype(np.uint8)
        c.mask.copy_(up(m.reshape(-1)))
        ref_c, ref_inv, ref_rp, ref_n = O.compact(m)
        call.start()
        shc.clear_inactive_rows(c.inv, B, V, D)
        assert call.wait() == ref_n
        assert np.array_equal(down(c.inv), ref_inv)
        assert np.array_equal(down(c.row_ptr), ref_rp)
        assert np.array_equal(down(c.coords)[:ref_n], ref_c)
        assert int(c.n_dev[0].item()) == ref_n
        got = down(D)
        assert np.all(got[ref_inv < 0] == 0)
        shc.compact_mask_start(c.mask, B, V, c.coords, c.inv, c.row_ptr, c.n_dev, c.ws, hc)
        assert shc.compact_mask_wait(hc, c.cap) == ref_n
    # a count above the capacity given to the wait
    m = (rng.random((B, V)) < 0.1).astype(np.uint8)
    c.mask.copy_(up(m.reshape(-1)))
    shc.compact_mask_start(c.mask, B, V, c.coords, c.inv, c.row_ptr, c.n_dev, c.ws, hc)
    with pytest.raises(shc.ShcError) as e:
        shc.compact_mask_wait(hc, int(m.sum()) - 1)
    assert e.value.status == -2
    torch.cuda.synchronize()
    # pageable host memory is refused by the start call, before any launch
    with pytest.raises(shc.ShcError) as e:
        shc.compact_mask_start(c.mask, B, V, c.coords, c.inv, c.row_ptr, c.n_dev, c.ws,
                               torch.zeros(1, dtype=torch.int64))
    assert e.value.status == -1


def test_compact_paper_workload_masks(dev):
    for w in (synth.workload_c1(), synth.workload_c2(), synth.workload_c5()):
        check_compaction(w.mask)
    check_compaction(synth.workload_c4(0.05).mask)


def test_compact_capacity(dev):
    rng = np.random.default_rng(5)
    m = (rng.random((10, 500)) < 0.2).astype(np.uint8)
    n = int(m.sum())
    check_compaction(m, cap=n // 2)          # coords truncated at cap, inv/row_ptr complete
    check_compaction(m, cap=0)
    c = Compaction(m, cap=n - 1)
    with pytest.raises(shc.ShcError) as e:
        c.run(want_host=True)
    assert e.value.status == -2


def test_compact_deterministic(dev):
    m = synth.workload_c4(0.05).mask
    c1 = Compaction(m)
    c1.run()
    c2 = Compaction(m)
    c2.run()
    assert torch.equal(c1.coords, c2.coords) and torch.equal(c1.inv, c2.inv)


# ----------------------------------------------------------------------------
# gather / scatter / pool (exact)
# ----------------------------------------------------------------------------


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("C", [16, 48, 128, 256])
def test_gather_scatter_exact(dev, dtype, C):
    rng = np.random.default_rng(C)
    B, V = 9, 1000
    m = (rng.random((B, V)) < 0.13).astype(np.uint8)
    x = synth.as_dtype(rng.standard_normal((B * V, C)).astype(np.float32), dtype)[1]
    c = Compaction(m)
    n = c.run()
    xd = up(x, dtype)
    S = torch.full((n + 5, C), float("nan"), dtype=xd.dtype, device=dev)
    shc.gather_rows(xd, c.coords, n, B, V, S)
    ref_c, ref_inv, _, _ = O.compact(m)
    ref_S = O.gather(x, ref_c, V)
    got = down(S)
    assert np.array_equal(got[:n], ref_S) and np.all(np.isnan(got[n:]))
    # zero-fill scatter: D = x (.) m exactly
    D = torch.full((B * V, C), float("nan"), dtype=xd.dtype, device=dev)
    shc.scatter(S, c.inv, c.coords, n, B, V, D, zero_fill=True)
    assert np.array_equal(down(D), O.scatter(ref_S, ref_inv, zero_fill=True))
    # active-only scatter keeps the sentinel in inactive rows
    D2 = torch.full((B * V, C), float("nan"), dtype=xd.dtype, device=dev)
    shc.scatter(S, c.inv, c.coords, n, B, V, D2, zero_fill=False)
    exp = O.scatter(ref_S, ref_inv, zero_fill=False, D=np.full((B * V, C), np.nan))
    got2 = down(D2)
    assert np.array_equal(np.isnan(got2), np.isnan(exp))
    assert np.array_equal(got2[~np.isnan(exp)], exp[~np.isnan(exp)])
    # the zeros alone (inactive rows; active rows keep the sentinel), then the
    # active rows: together the zero-fill scatter's result
    D3 = torch.full((B * V, C), float("nan"), dtype=xd.dtype, device=dev)
    shc.clear_inactive_rows(c.inv, B, V, D3)
    got3 = down(D3)
    act = ref_inv >= 0
    assert np.all(got3[~act] == 0) and np.all(np.isnan(got3[act]))
    shc.scatter(S, c.inv, c.coords, n, B, V, D3, zero_fill=False)
    assert torch.equal(D3, D)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("C,B,V", [(16, 70, 3000), (48, 70, 3000), (128, 70, 3000),
                                   (256, 70, 3000), (2048, 9, 700), (4096, 9, 700)])
def test_segment_maxpool_exact(dev, dtype, C, B, V):
    """Empty, short and long segments (body 5 is full: several batches of rows
    per thread), row widths that do and do not fill a wavefront, and rows
    wider than one block's threads."""
    rng = np.random.default_rng(100 + C)
    m = (rng.random((B, V)) < 0.05).astype(np.uint8)
    m[[0, B // 2 + 1, B - 1]] = 0             # empty bodies, first and last included
    m[5] = 1                                 # a full body
    c = Compaction(m)
    n = c.run()
    S = synth.as_dtype(rng.standard_normal((n, C)).astype(np.float32), dtype)[1]
    S[rng.random(S.shape) < 0.01] = np.nan   # NaN loses to numbers
    Sd = up(S, dtype)
    P = torch.full((B, C), 123.0, dtype=Sd.dtype, device=dev)
    shc.segment_maxpool(Sd, c.row_ptr, n, B, P, empty_value=-2.5)
    ref = O.segment_max(S.astype(np.float64), O.compact(m)[2], -2.5)
    got = down(P)
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    assert np.array_equal(got[~np.isnan(ref)], ref[~np.isnan(ref)])


# ----------------------------------------------------------------------------
# sparse linear (Eq. 6)
# ----------------------------------------------------------------------------


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("Cin,Cout", [(16, 16), (16, 64), (64, 64), (128, 128), (48, 80),
                                      (256, 256), (32, 192)])
def test_sparse_linear(dev, dtype, Cin, Cout):
    rng = np.random.default_rng(Cin * 1000 + Cout)
    n = 1000 + Cin                                   # ragged: not a multiple of the 64-row tile
    S = synth.as_dtype(rng.standard_normal((n, Cin)).astype(np.float32), dtype)[1]
    W = synth.as_dtype((rng.standard_normal((Cin, Cout)) / np.sqrt(Cin)).astype(np.float32),
                       dtype)[1]
    bias = rng.standard_normal(Cout).astype(np.float32)
    rows = np.arange(n)
    for b, act in ((None, shc.SHC_ACT_NONE), (bias, shc.SHC_ACT_RELU)):
        out = torch.full((n + 3, Cout), float("nan"), dtype=synth_dtype(dtype), device=dev)
        shc.sparse_linear(up(S, dtype), n, up(W, dtype), None if b is None else up(b), out, act)
        got = down(out)
        ref = O.linear_at(S, W, rows, b, act == shc.SHC_ACT_RELU)
        scale = O.linear_at(S, W, rows, b, scale=True)
        assert_scaled_close(got[:n], ref, scale, dtype, f"linear {Cin}->{Cout}", n_terms=Cin)
        assert np.all(np.isnan(got[n:]))


def synth_dtype(dtype):
    return torch.float32 if dtype == "f32" else torch.bfloat16


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("Cin,Cout", [(16, 64), (128, 128), (64, 48), (256, 128), (32, 16)])
def test_gather_sparse_linear(dev, dtype, Cin, Cout):
    """The fused gather + linear equals the oracle on the gathered rows and,
    bit for bit, the unfused gather followed by the linear layer."""
    rng = np.random.default_rng(Cin * 31 + Cout)
    B, V = 7, 1531
    m = (rng.random((B, V)) < 0.2).astype(np.uint8)
    x = synth.as_dtype(rng.standard_normal((B * V, Cin)).astype(np.float32), dtype)[1]
    W = synth.as_dtype((rng.standard_normal((Cin, Cout)) / np.sqrt(Cin)).astype(np.float32),
                       dtype)[1]
    bias = rng.standard_normal(Cout).astype(np.float32)
    c = Compaction(m)
    n = c.run()
    xd, Wd, bd = up(x, dtype), up(W, dtype), up(bias)
    fused = torch.full((n + 3, Cout), float("nan"), dtype=xd.dtype, device=dev)
    shc.gather_sparse_linear(xd, c.coords, n, B, V, Wd, bd, fused, shc.SHC_ACT_RELU)
    S = torch.empty((n, Cin), dtype=xd.dtype, device=dev)
    shc.gather_rows(xd, c.coords, n, B, V, S)
    plain = torch.empty((n, Cout), dtype=xd.dtype, device=dev)
    shc.sparse_linear(S, n, Wd, bd, plain, shc.SHC_ACT_RELU)
    got = down(fused)
    assert np.all(np.isnan(got[n:]))
    assert np.array_equal(got[:n], down(plain))
    ref_c = O.compact(m)[0]
    S_ref = O.gather(x, ref_c, V)
    ref = O.linear_at(S_ref, W, np.arange(n), bias, act=True)
    scale = O.linear_at(S_ref, W, np.arange(n), bias, scale=True)
    assert_scaled_close(got[:n], ref, scale, dtype, f"gather+linear {Cin}->{Cout}",
                        n_terms=Cin)


def test_gather_sparse_linear_bad_coords_read_zeros(dev):
    """A coordinate outside the mask's shape contributes a zero input row."""
    rng = np.random.default_rng(8)
    B, V, C = 2, 40, 32
    x = rng.standard_normal((B * V, C)).astype(np.float32)
    W = (rng.standard_normal((C, C)) / 6).astype(np.float32)
    bias = rng.standard_normal(C).astype(np.float32)
    coords = np.array([[0, 3], [1, 39], [2, 0], [0, 40], [-1, 5]], np.int32)
    out = torch.empty((5, C), device=dev)
    shc.gather_sparse_linear(up(x), up(coords), 5, B, V, up(W), up(bias), out,
                             shc.SHC_ACT_NONE)
    got = down(out)
    assert_scaled_close(got[0], x[3].astype(np.float64) @ W + bias,
                        np.abs(x[3]) @ np.abs(W) + np.abs(bias), "f32", "row (0,3)")
    assert_scaled_close(got[1], x[V + 39].astype(np.float64) @ W + bias,
                        np.abs(x[V + 39]) @ np.abs(W) + np.abs(bias), "f32", "row (1,39)")
    for r in (2, 3, 4):
        assert np.array_equal(got[r], bias.astype(np.float64))


def test_sparse_linear_zero_rows_is_noop(dev):
    out = torch.full((4, 16), 7.0, device=dev)
    shc.sparse_linear(torch.zeros(4, 16, device=dev), 0, torch.zeros(16, 16, device=dev), None,
                      out)
    torch.cuda.synchronize()
    assert torch.all(out == 7.0)


# ----------------------------------------------------------------------------
# several masks stacked as a batch axis; per-element masks (Sec. 3.1)
# ----------------------------------------------------------------------------


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("C", [16, 128])
def test_stacked_gather_exact(dev, dtype, C):
    rng = np.random.default_rng(C + 3)
    kappa, B, V = 3, 5, 600
    masks = (rng.random((kappa, B, V)) < 0.2).astype(np.uint8)
    x = synth.as_dtype(rng.standard_normal((B * V, C)).astype(np.float32), dtype)[1]
    st = O.stack_masks(masks)
    c = Compaction(st)
    n = c.run()
    S = torch.full((n + 4, C), float("nan"), dtype=synth_dtype(dtype), device=dev)
    shc.gather_rows_stacked(up(x, dtype), c.coords, n, B, kappa, V, S)
    ref_c, _, _, _ = O.compact(st)
    got = down(S)
    assert np.array_equal(got[:n], O.gather_stacked(x, ref_c, B, V))
    assert np.all(np.isnan(got[n:]))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("op", ["sum", "mean", "max"])
def test_combine_stacked(dev, dtype, op):
    """Max is exact; sum and mean are fp32 sums in k order rounded once:
    |err| <= (kappa + 1) 2^-24 sum_k |y_k| + (half an ulp of the output)."""
    rng = np.random.default_rng(5)
    kappa, R, C = 4, 1000, 48
    Y = synth.as_dtype(rng.standard_normal((kappa * R, C)).astype(np.float32) * 3, dtype)[1]
    out = torch.full((R + 2, C), float("nan"), dtype=synth_dtype(dtype), device=dev)
    shc.combine_stacked(up(Y, dtype), kappa, R, out, op)
    got = down(out)
    assert np.all(np.isnan(got[R:]))
    ref = O.combine_stacked(Y.astype(np.float64), kappa, op)
    if op == "max":
        assert np.array_equal(got[:R], ref)
    else:
        sa = np.abs(Y.astype(np.float64)).reshape(kappa, R, C).sum(0)
        if op == "mean":
            sa = sa / kappa
        half_ulp = 2.0 ** -8 if dtype == "bf16" else 2.0 ** -24
        bound = (kappa + 1) * 2.0 ** -24 * sa + half_ulp * np.abs(ref)
        assert np.all(np.abs(got[:R] - ref) <= bound)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_multi_mask_stack_vs_oracle(dev, dtype):
    """kappa = 3 masks as bodies k * B + b through the whole path (stacked
    gather, linear, conv from the table, zero-fill scatter, pool), then the
    kappa dense and pooled outputs combined; against the oracle run mask by
    mask and combined the same way."""
    rng = np.random.default_rng(31)
    kappa, B, V, K, C = 3, 4, 400, 9, 64
    pts = synth.sphere_points(V, rng)
    nbr = synth.knn(pts, K)
    masks = (rng.random((kappa, B, V)) < 0.15).astype(np.uint8)
    x = synth.as_dtype(rng.standard_normal((B * V, C)).astype(np.float32), dtype)[1]
    Wl = synth.as_dtype((rng.standard_normal((C, C)) / np.sqrt(C)).astype(np.float32), dtype)[1]
    Wc = synth.as_dtype((rng.standard_normal((K, C, C)) / np.sqrt(K * C)).astype(np.float32),
                        dtype)[1]
    st = O.stack_masks(masks)
    Bs = kappa * B
    c = Compaction(st)
    n = c.run()
    td = synth_dtype(dtype)
    S0 = torch.empty((n, C), dtype=td, device=dev)
    shc.gather_rows_stacked(up(x, dtype), c.coords, n, B, kappa, V, S0)
    S1 = torch.empty((n, C), dtype=td, device=dev)
    shc.sparse_linear(S0, n, up(Wl, dtype), None, S1, shc.SHC_ACT_RELU)
    table = torch.empty((K * n,), dtype=torch.int32, device=dev)
    shc.build_neighbor_table(c.coords, c.inv, n, Bs, V, up(nbr), table)
    S2 = torch.empty((n, C), dtype=td, device=dev)
    shc.sparse_neighbor_conv_table(S1, table, n, up(Wc, dtype), None, S2, shc.SHC_ACT_RELU)
    D = torch.empty((Bs * V, C), dtype=td, device=dev)
    shc.scatter(S2, c.inv, c.coords, n, Bs, V, D, zero_fill=True)
    P = torch.empty((Bs, C), dtype=td, device=dev)
    shc.segment_maxpool(S2, c.row_ptr, n, Bs, P, 0.0)
    spec = [("linear", Wl, None, True), ("conv", Wc, None, True)]
    dense_k, pool_k = [], []
    for k in range(kappa):
        r = O.run_stack(x, masks[k], nbr, spec, dtype, pool=True)
        dense_k.append(O.scatter(r["outs"][-1], r["inv"], zero_fill=True))
        pool_k.append(r["pool"])
    for op in ("sum", "mean", "max"):
        Dc = torch.empty((B * V, C), dtype=td, device=dev)
        shc.combine_stacked(D, kappa, B * V, Dc, op)
        Pc = torch.empty((B, C), dtype=td, device=dev)
        shc.combine_stacked(P, kappa, B, Pc, op)
        assert_normwise_close(down(Dc), O.combine_stacked(np.concatenate(dense_k), kappa, op),
                              dtype, f"dense {op}")
        assert_normwise_close(down(Pc), O.combine_stacked(np.concatenate(pool_k), kappa, op),
                              dtype, f"pool {op}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("C", [16, 48, 128, 2048])
def test_element_masks_exact(dev, dtype, C):
    rng = np.random.default_rng(C * 7 + 1)
    B, V = 6, 300
    me = (rng.random((B, V, C)) < 0.01 * (2048 / C) ** 0.5).astype(np.uint8)
    me[0, :5, :] = 0
    me[0, 3, C - 1] = 7                      # only the last channel of (0, 3)
    mdev = torch.full((B * V,), 9, dtype=torch.uint8, device=dev)
    shc.row_mask_from_elements(up(me.reshape(-1)), B, V, mdev)
    m = down(mdev).reshape(B, V)
    assert np.array_equal(m, O.row_mask_from_elements(me))
    assert m[0, 3] == 1 and m[0, 2] == 0
    x = synth.as_dtype(rng.standard_normal((B * V, C)).astype(np.float32), dtype)[1]
    c = Compaction(m)
    n = c.run()
    S = torch.full((n + 1, C), float("nan"), dtype=synth_dtype(dtype), device=dev)
    shc.gather_rows_masked(up(x, dtype), up(me.reshape(-1)), c.coords, n, B, V, S)
    ref_c, _, _, _ = O.compact(m)
    got = down(S)
    assert np.array_equal(got[:n], O.gather_masked(x, me, ref_c, V))
    assert np.all(np.isnan(got[n:]))


# ----------------------------------------------------------------------------
# mask scores (Eq. 3) and top-kappa selection
# ----------------------------------------------------------------------------


def score_case(rng, K, N, C):
    """bf16 outputs with a range of mutual similarities: a shared part with
    mask-dependent weight plus mask-own noise, and one mask on its own rows."""
    common = rng.standard_normal((N, C))
    O_ = np.stack([(k / K) * common + rng.standard_normal((N, C)) * (1 + k % 3)
                   for k in range(K)])
    if K > 2:
        O_[K - 1] = 0
        O_[K - 1, : N // 7] = rng.standard_normal((N // 7, C))
    return synth.as_dtype(O_.astype(np.float32), "bf16")[1].reshape(K, N, C)


def similarity_bound(Y, sim, N):
    """First-order bound of the GPU similarity's error: Gram entries summed in
    fp32 over at most N/32 + 2 sequential MFMA accumulations err by
    gamma |O_i|^T |O_k| entrywise; F = ||G||^2 and the normalisation follow."""
    gamma = (N / 32 + 2) * 2.0 ** -24
    K = Y.shape[0]
    A = np.abs(Y).astype(np.float64)
    F = O.gram_frobenius(Y)
    dF = np.empty((K, K))
    for i in range(K):
        for k in range(K):
            a = np.linalg.norm(A[i].T @ A[k]) * gamma
            dF[i, k] = 2 * np.sqrt(F[i, k]) * a + a * a
    d = np.diag(F)
    rel = np.where(F > 0, dF / np.maximum(F, 1e-300), 0)
    return 2 * (sim * (rel + 0.5 * (dF.diagonal()[:, None] / d[:, None]) +
                       0.5 * (dF.diagonal()[None, :] / d[None, :])) + 1e-12)


# pair tiles: (3, 128), (10, 64), (5, 192), (1, 64); 256-column blocks of the
# concatenated outputs: (10, 128), (4, 256), (11, 128) with a padded last
# block, (16, 64) with four masks per block, (7, 256)
@pytest.mark.parametrize("K,N,C", [(3, 1000, 128), (10, 37, 64), (10, 20000, 128),
                                   (4, 5000, 256), (5, 3000, 192), (1, 500, 64),
                                   (11, 3001, 128), (16, 2500, 64), (7, 777, 256)])
def test_mask_scores_vs_oracle(dev, K, N, C):
    rng = np.random.default_rng(K * 1000 + C)
    Y = score_case(rng, K, N, C)
    alpha_in = rng.standard_normal(K)
    kappa = min(3, K)
    a_out = torch.full((K,), np.nan, dtype=torch.float64, device=dev)
    simd = torch.full((K * K,), np.nan, dtype=torch.float64, device=dev)
    top = torch.full((kappa + 1,), -9, dtype=torch.int32, device=dev)
    ws = shc.mask_scores(up(Y.reshape(K * N, C), "bf16").reshape(K, N, C), up(alpha_in),
                         a_out, kappa, top, simd)
    sim = down(simd).reshape(K, K)
    ref_sim = O.mask_similarity(Y)
    assert np.all(np.abs(sim - ref_sim) <= similarity_bound(Y, ref_sim, N)), \
        f"similarity off by {np.max(np.abs(sim - ref_sim)):.3g}"
    ref_alpha = O.alpha_update(alpha_in, Y)
    bound_a = (similarity_bound(Y, ref_sim, N).sum(0) / max(K - 1, 1))
    assert np.all(np.abs(down(a_out) - ref_alpha) <= bound_a + 1e-12)
    got_top = down(top)
    assert got_top[kappa] == -9
    # the selection is the device's own ranking of its scores; where the
    # reference scores are farther apart than the bound it matches them
    assert list(got_top[:kappa]) == list(O.top_kappa(down(a_out), kappa))
    gap = np.min(np.diff(np.sort(ref_alpha))) if K > 1 else 1.0
    if gap > 2 * bound_a.max():
        assert list(got_top[:kappa]) == list(O.top_kappa(ref_alpha, kappa))
    # bit-for-bit repeat, workspace reused
    a2 = torch.empty_like(a_out)
    shc.mask_scores(up(Y.reshape(K * N, C), "bf16").reshape(K, N, C), up(alpha_in), a2, 0,
                    None, None, ws)
    assert torch.equal(a2, a_out)


def test_mask_scores_special_cases(dev):
    """Disjoint row supports give exact zeros off the diagonal (every score
    + 1); identical outputs give similarity 1 (scores unchanged); K = 1
    leaves the score alone; no alpha_in means zeros."""
    rng = np.random.default_rng(9)
    N, C = 300, 64
    Y = np.zeros((3, N, C), np.float32)
    for k in range(3):
        Y[k, 100 * k:100 * k + 100] = rng.standard_normal((100, C))
    Y = synth.as_dtype(Y, "bf16")[1]
    a = torch.empty(3, dtype=torch.float64, device=dev)
    simd = torch.empty(9, dtype=torch.float64, device=dev)
    shc.mask_scores(up(Y.reshape(-1, C), "bf16").reshape(3, N, C), None, a, 0, None, simd)
    sim = down(simd).reshape(3, 3)
    assert np.all(sim[~np.eye(3, dtype=bool)] == 0)
    assert np.allclose(np.diag(sim), 1, atol=1e-12)
    assert np.allclose(down(a), 1, atol=1e-12)
    X = Y[0]
    Yi = np.stack([X, X])
    a = torch.empty(2, dtype=torch.float64, device=dev)
    shc.mask_scores(up(Yi.reshape(-1, C), "bf16").reshape(2, N, C), up(np.array([0.25, -4.0])),
                    a, 0)
    assert np.allclose(down(a), [0.25, -4.0], atol=1e-9)
    a1 = torch.empty(1, dtype=torch.float64, device=dev)
    top1 = torch.empty(1, dtype=torch.int32, device=dev)
    shc.mask_scores(up(X, "bf16").reshape(1, N, C), up(np.array([3.5])), a1, 1, top1)
    assert float(a1[0]) == 3.5 and int(top1[0]) == 0
    # an all-zero output: similarity 1 with every mask, score unchanged,
    # nothing added to the others, ranked last
    Z = np.stack([Y[0], np.zeros_like(Y[0]), Y[2], Y[0] + Y[1]])
    Z = synth.as_dtype(Z.astype(np.float32), "bf16")[1]
    az = torch.empty(4, dtype=torch.float64, device=dev)
    simz = torch.empty(16, dtype=torch.float64, device=dev)
    topz = torch.empty(4, dtype=torch.int32, device=dev)
    alpha0 = np.full(4, 0.5)
    shc.mask_scores(up(Z.reshape(-1, C), "bf16").reshape(4, N, C), up(alpha0), az, 4, topz,
                    simz)
    sz = down(simz).reshape(4, 4)
    ref = O.mask_similarity(Z)
    assert np.all(sz[1] == 1.0) and np.all(sz[:, 1] == 1.0)
    live = np.ix_([0, 2, 3], [0, 2, 3])
    assert np.all(np.abs(sz - ref)[live] <= similarity_bound(Z[[0, 2, 3]], ref[live], N))
    assert float(az[1]) == 0.5
    assert np.allclose(down(az), O.alpha_update(alpha0, Z), atol=1e-6)
    assert int(down(topz)[-1]) == 1


# ----------------------------------------------------------------------------
# sparse group normalization (Eqs. 7-9)
# ----------------------------------------------------------------------------


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("C,G,B,V,p", [
    (16, 4, 9, 300, 0.3), (128, 32, 12, 2000, 0.05), (128, 1, 12, 2000, 0.05),
    (48, 3, 6, 700, 0.4), (256, 8, 5, 1500, 0.2), (128, 16, 3, 3000, 0.9),
    (4096, 64, 3, 200, 0.5), (2048, 2048, 2, 150, 0.6), (48, 1, 4, 500, 0.3),
    (256, 1, 6, 900, 0.3), (1024, 4, 3, 400, 0.5)])
def test_group_norm_oracle(dev, dtype, C, G, B, V, p):
    """Bodies that are empty, of one row, register-resident and streamed (p =
    0.9: 2700 rows, beyond the resident 1024), channel vectors that span
    groups (C/G = 4) and groups that span vectors, G = 1 and G = C."""
    rng = np.random.default_rng(C * 31 + G + B)
    m = (rng.random((B, V)) < p).astype(np.uint8)
    m[1] = 0
    m[2 % B, :] = 0
    m[2 % B, 5] = 1
    coords, inv, rp, n = O.compact(m)
    S = (rng.standard_normal((n, C)) * 2.0 + rng.standard_normal(C) * 3.0).astype(np.float32)
    S = synth.as_dtype(S, dtype)[1]
    Sd = up(S, dtype)
    out = torch.full((n + 3, C), float("nan"), dtype=Sd.dtype, device=dev)
    shc.segment_group_norm(Sd, up(rp), n, B, G, out)
    got = down(out)
    assert np.all(np.isnan(got[n:]))
    ref = O.group_norm(S.astype(np.float64), rp, G)
    assert_gn_close(got[:n], ref, dtype, gn_floor(S, rp, G), f"group norm C={C} G={G} {dtype}")


def test_group_norm_deterministic_and_edge_cases(dev):
    rng = np.random.default_rng(77)
    B, V, C, G = 8, 1000, 128, 32
    m = (rng.random((B, V)) < 0.2).astype(np.uint8)
    coords, inv, rp, n = O.compact(m)
    S = up(rng.standard_normal((n, C)).astype(np.float32), "bf16")
    o1 = torch.empty_like(S)
    o2 = torch.empty_like(S)
    shc.segment_group_norm(S, up(rp), n, B, G, o1)
    shc.segment_group_norm(S, up(rp), n, B, G, o2)
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    # a constant body: zero deviation everywhere, outputs exactly zero
    Sc = torch.full((n, C), 3.25, dtype=torch.float32, device=dev)
    oc = torch.empty_like(Sc)
    shc.segment_group_norm(Sc, up(rp), n, B, G, oc)
    assert torch.all(oc == 0)
    # N' = 0 is a no-op; bad arguments are refused before any launch
    shc.segment_group_norm(S[:0], up(np.zeros(B + 1, np.int32)), 0, B, G, o1[:0])
    for kw, status in ((dict(G=3), -1), (dict(eps=0.0), -1), (dict(eps=float("inf")), -1)):
        a = dict(G=G, eps=1e-5)
        a.update(kw)
        with pytest.raises(shc.ShcError) as e:
            shc.segment_group_norm(S, up(rp), n, B, a["G"], o1, eps=a["eps"])
        assert e.value.status == status


# ----------------------------------------------------------------------------
# sparse neighbourhood conv (Eqs. 4-5)
# ----------------------------------------------------------------------------


def table_reference(m, nbr):
    """table[j][i] = inv[b_i, nbr[v_i][j]] or -1, from the oracle's compaction
    (the definition of the neighbour rows of Eqs. 4-5, written out)."""
    B, V = m.shape
    coords, inv, _, n = O.compact(m)
    K = nbr.shape[1]
    t = np.full((K, n), -1, np.int64)
    for j in range(K):
        u = nbr[coords[:, 1], j].astype(np.int64)
        ok = (u >= 0) & (u < V)
        r = inv[coords[:, 0] * V + np.where(ok, u, 0)]
        t[j] = np.where(ok, r, -1)
    return t


def run_conv(dev, m, nbr, S_vals, W, bias, dtype, act=shc.SHC_ACT_RELU, path="direct"):
    """One conv through the C ABI: `direct` (coords, inv, nbr) or `table`
    (neighbour-row table built by the library, checked exactly first)."""
    B, V = m.shape
    c = Compaction(m)
    n = c.run()
    K, Cin, Cout = W.shape
    out = torch.full((n + 2, Cout), float("nan"), dtype=synth_dtype(dtype), device=dev)
    Sd = up(S_vals, dtype)
    Wd = up(W, dtype)
    bd = None if bias is None else up(bias)
    if path == "direct":
        shc.sparse_neighbor_conv(Sd, c.coords, c.inv, n, B, V, up(nbr), Wd, bd, out, act)
    else:
        table = torch.full((K * n + 3,), -7, dtype=torch.int32, device=dev)
        shc.build_neighbor_table(c.coords, c.inv, n, B, V, up(nbr), table)
        got_t = down(table)
        assert np.array_equal(got_t[:K * n].reshape(K, n), table_reference(m, nbr))
        assert np.all(got_t[K * n:] == -7)
        shc.sparse_neighbor_conv_table(Sd, table, n, Wd, bd, out, act)
    got = down(out)
    assert np.all(np.isnan(got[n:]))
    return got[:n], n


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("B,V,K,Cin,Cout,p", [
    (3, 200, 9, 16, 64, 0.3), (2, 333, 9, 64, 64, 0.5), (4, 150, 4, 48, 32, 0.4),
    (2, 500, 9, 128, 128, 0.1), (1, 300, 1, 32, 16, 0.6), (2, 100, 32, 16, 16, 0.7),
    (2, 257, 9, 256, 256, 0.2), (3, 211, 5, 32, 192, 0.9)])
@pytest.mark.parametrize("path", ["direct", "table"])
def test_sparse_conv_full_oracle(dev, dtype, B, V, K, Cin, Cout, p, path):
    rng = np.random.default_rng(B * V + K * 7 + Cin)
    m = (rng.random((B, V)) < p).astype(np.uint8)
    nbr = rand_nbr(V, K, rng)
    coords, inv, rp, n = O.compact(m)
    S = synth.as_dtype(rng.standard_normal((n, Cin)).astype(np.float32), dtype)[1]
    W = synth.as_dtype((rng.standard_normal((K, Cin, Cout)) / np.sqrt(K * Cin))
                       .astype(np.float32), dtype)[1]
    bias = rng.standard_normal(Cout).astype(np.float32)
    for b, act in ((None, shc.SHC_ACT_NONE), (bias, shc.SHC_ACT_RELU)):
        got, n2 = run_conv(dev, m, nbr, S, W, b, dtype, act, path)
        assert n2 == n
        ref = O.sparse_conv(S, coords, B, V, nbr, W, b, act == shc.SHC_ACT_RELU)
        scale = O.sparse_conv_scale(S, coords, B, V, nbr, W, b)
        assert_scaled_close(got, ref, scale, dtype, f"conv K={K} {Cin}->{Cout} p={p}",
                            n_terms=K * Cin)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("kind,K,Cin,Cout", [("linear", 1, 4096, 4096), ("linear", 1, 4096, 16),
                                             ("conv", 9, 1024, 512), ("conv", 3, 4096, 64)])
def test_max_channels(dev, dtype, kind, K, Cin, Cout):
    """Channel counts at the library's limit (4096) and wide convs whose weight
    slices do not fit in LDS, on a few dozen rows (a ragged last tile)."""
    rng = np.random.default_rng(Cin + Cout + K)
    B, V = 2, 40
    m = (rng.random((B, V)) < 0.6).astype(np.uint8)
    coords, inv, rp, n = O.compact(m)
    S = synth.as_dtype(rng.standard_normal((n, Cin)).astype(np.float32), dtype)[1]
    W = synth.as_dtype((rng.standard_normal((K, Cin, Cout)) / np.sqrt(K * Cin))
                       .astype(np.float32), dtype)[1]
    bias = rng.standard_normal(Cout).astype(np.float32)
    if kind == "linear":
        out = torch.full((n, Cout), float("nan"), dtype=TORCH[dtype], device=dev)
        shc.sparse_linear(up(S, dtype), n, up(W[0], dtype), up(bias), out, shc.SHC_ACT_RELU)
        torch.cuda.synchronize()
        ref = O.relu(np.asarray(S, np.float64) @ W[0] + bias)
        scale = np.abs(np.asarray(S, np.float64)) @ np.abs(W[0]) + np.abs(bias)
        assert_scaled_close(down(out), ref, scale, dtype, f"linear {Cin}->{Cout}", n_terms=Cin)
    else:
        nbr = rand_nbr(V, K, rng)
        got, n2 = run_conv(dev, m, nbr, S, W, bias, dtype, shc.SHC_ACT_RELU, "table")
        assert n2 == n
        ref = O.sparse_conv(S, coords, B, V, nbr, W, bias, True)
        scale = O.sparse_conv_scale(S, coords, B, V, nbr, W, bias)
        assert_scaled_close(got, ref, scale, dtype, f"conv K={K} {Cin}->{Cout}", n_terms=K * Cin)


@pytest.mark.parametrize("path", ["direct", "table"])
def test_sparse_conv_edge_cases(dev, path):
    rng = np.random.default_rng(3)
    V, K, C = 50, 9, 16
    nbr = rand_nbr(V, K, rng)
    nbr[7, 4] = 7
    W = (rng.standard_normal((K, C, C)) / 12).astype(np.float32)
    b = rng.standard_normal(C).astype(np.float32)
    # a lone active vertex sees only its own slots
    m = np.zeros((2, V), np.uint8)
    m[1, 7] = 1
    S = rng.standard_normal((1, C)).astype(np.float32)
    got, n = run_conv(dev, m, nbr, S, W, b, "f32", shc.SHC_ACT_NONE, path)
    ref = b + sum(S[0].astype(np.float64) @ W[j] for j in range(K) if nbr[7, j] == 7)
    assert_scaled_close(got[0], ref, O.conv_at(S, O.compact(m)[0], 2, V, nbr, W, [0], b,
                                                scale=True)[0], "f32", "lone vertex")
    # out-of-range neighbour entries count as absent
    nbr_bad = nbr.copy()
    nbr_bad[:, 3] = V + 5
    nbr_bad[:, 5] = -9
    nbr_ok = nbr.copy()
    nbr_ok[:, 3] = -1
    nbr_ok[:, 5] = -1
    m = (rng.random((2, V)) < 0.6).astype(np.uint8)
    n = int(m.sum())
    S = rng.standard_normal((n, C)).astype(np.float32)
    g_bad, _ = run_conv(dev, m, nbr_bad, S, W, b, "f32", path=path)
    g_ok, _ = run_conv(dev, m, nbr_ok, S, W, b, "f32", path=path)
    assert np.array_equal(g_bad, g_ok)
    # K = 1 self-neighbour conv is the linear layer
    self_nbr = np.arange(V, dtype=np.int32)[:, None]
    g_c, _ = run_conv(dev, m, self_nbr, S, W[:1], b, "f32", path=path)
    out = torch.empty((n, C), device=dev)
    shc.sparse_linear(up(S, "f32"), n, up(W[0], "f32"), up(b), out, shc.SHC_ACT_RELU)
    assert np.array_equal(g_c, down(out))


def test_sparse_conv_deterministic(dev):
    """Repeated calls give identical bits, and the table path gives the same
    bits as the direct path (same kernel, same row blocks)."""
    w = synth.workload_c4(0.05)
    rng = np.random.default_rng(1)
    m = w.mask[:16]
    n = int(m.sum())
    S = synth.as_dtype(rng.standard_normal((n, 128)).astype(np.float32), "bf16")[1]
    W = w.layers[1].W
    g1, _ = run_conv(dev, m, w.nbr, S, W, None, "bf16")
    g2, _ = run_conv(dev, m, w.nbr, S, W, None, "bf16")
    g3, _ = run_conv(dev, m, w.nbr, S, W, None, "bf16", path="table")
    g4, _ = run_conv(dev, m, w.nbr, S, W, None, "bf16", path="table")
    assert np.array_equal(g1, g2)
    assert np.array_equal(g3, g4)
    assert np.array_equal(g1, g3)


def test_neighbor_table_zero_rows(dev):
    """N' = 0: building the table and the table conv are no-ops."""
    V, K = 20, 9
    nbr = up(rand_nbr(V, K, np.random.default_rng(5)))
    c = Compaction(np.zeros((2, V), np.uint8))
    assert c.run() == 0
    table = torch.full((8,), -7, dtype=torch.int32, device=dev)
    shc.build_neighbor_table(c.coords, c.inv, 0, 2, V, nbr, table)
    S = torch.zeros((1, 16), device=dev)
    out = torch.full((1, 16), 3.0, device=dev)
    shc.sparse_neighbor_conv_table(S, table, 0, torch.zeros((K, 16, 16), device=dev), None, out)
    torch.cuda.synchronize()
    assert np.all(down(table) == -7) and np.all(down(out) == 3.0)


# ----------------------------------------------------------------------------
# workloads at their full sizes (sampled rows) and whole stacks
# ----------------------------------------------------------------------------


def test_c1_full_stack(dev):
    from paper_2608_09388_amd.pipeline import SparseStack
    w = synth.workload_c1()
    st = SparseStack(w, device=str(dev))
    st.step()
    res = st.results()
    ref = O.run_stack(w.x, w.mask, w.nbr, [(l.kind, l.W, l.bias, l.relu) for l in w.layers],
                      w.dtype)
    assert res["n"] == ref["n"] == res["n_dev"]
    assert np.array_equal(res["coords"], ref["coords"])
    S0 = O.gather(w.x, ref["coords"], w.V)
    scale = O.sparse_conv_scale(S0, ref["coords"], w.B, w.V, w.nbr, w.layers[0].W)
    assert_scaled_close(res["outs"][0], ref["outs"][0], scale, "f32", "C1 conv")
    dense_ref = O.scatter(res["outs"][0], ref["inv"], zero_fill=True)
    assert np.array_equal(res["dense"], dense_ref)


def test_c2_full_stack_bf16(dev):
    from paper_2608_09388_amd.pipeline import SparseStack
    w = synth.workload_c2()
    st = SparseStack(w, device=str(dev))
    st.step()
    res = st.results()
    ref = O.run_stack(w.x, w.mask, w.nbr, [(l.kind, l.W, l.bias, l.relu) for l in w.layers],
                      w.dtype, pool=True)
    assert res["n"] == ref["n"]
    # first layer: identical inputs, per-element bound
    S0 = O.gather(w.x, ref["coords"], w.V)
    scale = O.sparse_conv_scale(S0, ref["coords"], w.B, w.V, w.nbr, w.layers[0].W)
    ref0 = O.sparse_conv(S0, ref["coords"], w.B, w.V, w.nbr, w.layers[0].W, None, True)
    assert_scaled_close(res["outs"][0], ref0, scale, "bf16", "C2 layer 0",
                        n_terms=w.K * w.layers[0].W.shape[1])
    for l in range(len(w.layers)):
        assert_normwise_close(res["outs"][l], ref["outs"][l], "bf16", f"C2 layer {l}")
    assert_normwise_close(res["pool"], ref["pool"], "bf16", "C2 pool")
    # the pool is exactly the per-body max of the GPU's own last layer
    rp = res["row_ptr"]
    last = res["outs"][-1]
    for b in range(w.B):
        seg = last[rp[b]:rp[b + 1]]
        assert np.array_equal(res["pool"][b], seg.max(0) if len(seg) else np.zeros(seg.shape[1]))


def sampled_layer_check(res_rows_in, got, w, layer, coords, rows, dtype, what):
    """Check sampled output rows of one layer against the oracle's by-row definition."""
    if layer.kind == "conv":
        ref = O.conv_at(res_rows_in, coords, w.B, w.V, w.nbr, layer.W, rows, layer.bias,
                        layer.relu)
        sc = O.conv_at(res_rows_in, coords, w.B, w.V, w.nbr, layer.W, rows, layer.bias,
                       scale=True)
        n_terms = layer.W.shape[0] * layer.W.shape[1]
    else:
        ref = O.linear_at(res_rows_in, layer.W, rows, layer.bias, layer.relu)
        sc = O.linear_at(res_rows_in, layer.W, rows, layer.bias, scale=True)
        n_terms = layer.W.shape[0]
    assert_scaled_close(got[rows], ref, sc, dtype, what, n_terms=n_terms)


@pytest.mark.parametrize("name", ["c3_f32", "c3_bf16", "c3_5pct_bf16", "c4_0.01", "c4_0.05",
                                  "c4_0.2", "c4_0.5", "c4_1.0"])
def test_full_size_workloads_sampled(dev, name):
    from paper_2608_09388_amd.pipeline import SparseStack
    if name.startswith("c3"):
        w = synth.workload_c3("f32" if "f32" in name else "bf16", five_percent="5pct" in name)
    else:
        w = synth.workload_c4(float(name.split("_")[1]))
    st = SparseStack(w, device=str(dev))
    st.step()
    res = st.results()
    coords, inv, rp, n = O.compact(w.mask)
    assert res["n"] == n and np.array_equal(res["coords"], coords)
    assert np.array_equal(res["inv"], inv) and np.array_equal(res["row_ptr"], rp)
    rng = np.random.default_rng(17)
    rows = np.unique(np.concatenate([rng.choice(n, size=min(n, 1500), replace=False),
                                     [0, n - 1]]))
    # layer 0 input is the exact gather; later layers take the oracle's own
    # previous layer at every row the sampled rows read (computed in full)
    S_in = O.gather(w.x, coords, w.V)
    for l, layer in enumerate(w.layers):
        sampled_layer_check(S_in, res["outs"][l], w, layer, coords, rows, w.dtype,
                            f"{name} layer {l}")
        if l + 1 < len(w.layers):
            full_rows = np.arange(n)
            if layer.kind == "conv":
                y = O.conv_at(S_in, coords, w.B, w.V, w.nbr, layer.W, full_rows, layer.bias,
                              layer.relu)
            else:
                y = O.linear_at(S_in, layer.W, full_rows, layer.bias, layer.relu)
            S_in = O.store(y, w.dtype)
            assert_normwise_close(res["outs"][l], S_in, w.dtype, f"{name} layer {l} full")
    if w.scatter:
        dense = res["dense"]
        act_rows = inv >= 0
        assert np.all(dense[~act_rows] == 0)
        assert np.array_equal(dense[act_rows], res["outs"][-1][inv[act_rows]])
    if w.pool:
        last = res["outs"][-1]
        P = res["pool"]
        for b in rng.choice(w.B, size=min(w.B, 40), replace=False):
            seg = last[rp[b]:rp[b + 1]]
            assert np.array_equal(P[b], seg.max(0) if len(seg) else np.zeros(last.shape[1]))


@pytest.mark.parametrize("side", [False, True])
@pytest.mark.parametrize("steps", [1, 2, 3, 5])
def test_overlapped_run_new_mask_per_batch(dev, steps, side):
    """SparseStack.run: each batch's compaction (into another index set) is
    enqueued before the previous batch's scatter and pool -- with ``side``, on
    a second stream beside them, ordered by events and, for an index set's
    reuse, by a host-side check of its last reader (five batches rotate the
    three sets past it).  Every batch gets its own mask and features; the
    outputs left behind must be the oracle's for the last batch, with index
    sets that last held another mask."""
    from paper_2608_09388_amd.pipeline import SparseStack, to_device
    w = synth.workload_c4(0.05, B=6, V=655)
    rng = np.random.default_rng(400 + steps)
    masks = [(rng.random((w.B, w.V)) < p).astype(np.uint8) for p in (0.3, 0.05, 0.2, 0.6, 0.1)][:steps]
    xs = [synth.as_dtype(rng.standard_normal(w.x.shape).astype(np.float32), w.dtype)[1]
          for _ in range(steps)]
    st = SparseStack(w, device=str(dev), side_stream=side)
    st.run(2)                               # two index sets hold the workload's own mask

    def feed(k):
        st.mask.copy_(up(masks[k].reshape(-1)))
        st.x.copy_(to_device(xs[k], w.dtype, st.device))

    n = st.run(steps, feed=feed)
    m, x = masks[-1], xs[-1]
    spec = [(l.kind, l.W, l.bias, l.relu) for l in w.layers]
    ref = O.run_stack(x, m, w.nbr, spec, w.dtype, pool=True)
    got = st.results()
    assert n == ref["n"] == got["n"] == got["n_dev"]
    assert np.array_equal(got["coords"], ref["coords"])
    assert np.array_equal(got["inv"], ref["inv"])
    for l in range(len(w.layers)):
        assert_normwise_close(got["outs"][l], ref["outs"][l], w.dtype, f"layer {l}")
    dense_ref = O.scatter(ref["outs"][-1], ref["inv"], zero_fill=True)
    assert_normwise_close(got["dense"], dense_ref, w.dtype, "dense")
    assert np.all(got["dense"][ref["inv"] < 0] == 0)
    assert_normwise_close(got["pool"], ref["pool"], w.dtype, "pool")


@pytest.mark.parametrize("side", [False, True])
def test_run_under_another_stream(dev, side):
    """A stack built on the default stream and run (and stepped) under
    ``torch.cuda.stream(other)``: the inputs are written on the other stream
    just before, the results read on it just after, and they must be bit for
    bit those of the same run on the default stream."""
    from paper_2608_09388_amd.pipeline import SparseStack, to_device
    w = synth.workload_c4(0.05, B=6, V=655)
    rng = np.random.default_rng(77)
    masks = [(rng.random((w.B, w.V)) < p).astype(np.uint8) for p in (0.2, 0.4, 0.1)]
    xs = [synth.as_dtype(rng.standard_normal(w.x.shape).astype(np.float32), w.dtype)[1]
          for _ in range(3)]

    def go(st, stream):
        def feed(k):
            st.mask.copy_(up(masks[k].reshape(-1)))
            st.x.copy_(to_device(xs[k], w.dtype, st.device))
        with torch.cuda.stream(stream):
            n = st.run(3, feed=feed)
            outs = [a.clone() for a in (st.acts[-1][:n], st.dense_out, st.pooled)]
        torch.cuda.synchronize()
        return [o.view(torch.int16).cpu().numpy() for o in outs]

    ref_st = SparseStack(w, device=str(dev), side_stream=side)
    ref = go(ref_st, torch.cuda.current_stream())
    st = SparseStack(w, device=str(dev), side_stream=side)
    other = torch.cuda.Stream(device=dev)
    got = go(st, other)
    for a, b in zip(got, ref):
        assert np.array_equal(a, b)
    # step() under the other stream, with its input written there just before
    with torch.cuda.stream(other):
        st.mask.copy_(up(masks[0].reshape(-1)))
        st.x.copy_(to_device(xs[0], w.dtype, st.device))
        n = st.step()
        pooled = st.pooled.clone()
    torch.cuda.synchronize()
    spec = [(l.kind, l.W, l.bias, l.relu) for l in w.layers]
    oref = O.run_stack(xs[0], masks[0], w.nbr, spec, w.dtype, pool=True)
    assert n == oref["n"]
    assert_normwise_close(pooled.float().cpu().numpy(), oref["pool"], w.dtype, "pool")


def test_c5_sequences_stack(dev):
    """C5 shape (V=655, C=256 bf16, Markov masks, 3 convs + per-frame pool) on one of
    the 32 sequences end to end against the full oracle stack; all 32 sequences for
    compaction and the pool property."""
    from paper_2608_09388_amd.pipeline import SparseStack
    w_full = synth.workload_c5()
    st = SparseStack(w_full, device=str(dev))
    st.step()
    res = st.results()
    coords, inv, rp, n = O.compact(w_full.mask)
    assert res["n"] == n and np.array_equal(res["row_ptr"], rp)
    last = res["outs"][-1]
    for b in np.random.default_rng(2).choice(w_full.B, 50, replace=False):
        seg = last[rp[b]:rp[b + 1]]
        assert np.array_equal(res["pool"][b], seg.max(0) if len(seg) else np.zeros(256))
    # one sequence (64 frames) through the full oracle
    w = synth.workload_c5(n_seq=1)
    st2 = SparseStack(w, device=str(dev))
    st2.step()
    r2 = st2.results()
    ref = O.run_stack(w.x, w.mask, w.nbr, [(l.kind, l.W, l.bias, l.relu) for l in w.layers],
                      w.dtype, pool=True)
    for l in range(3):
        assert_normwise_close(r2["outs"][l], ref["outs"][l], "bf16", f"C5 layer {l}")
    assert_normwise_close(r2["pool"], ref["pool"], "bf16", "C5 pool")


def test_empty_mask_path(dev):
    from paper_2608_09388_amd.pipeline import SparseStack
    w = synth.workload_c1()
    w.mask = np.zeros_like(w.mask)
    w.pool = True
    st = SparseStack(w, device=str(dev))
    st.dense_out.fill_(float("nan"))
    st.pooled.fill_(float("nan"))
    assert st.step() == 0
    res = st.results()
    assert res["n"] == 0 and np.all(res["row_ptr"] == 0) and np.all(res["inv"] == -1)
    assert np.all(res["dense"] == 0) and np.all(res["pool"] == 0)


def test_stream_events_order_streams(dev):
    """shc_event_*: a wait on the event holds the second stream until the work
    recorded on the first has finished (its device writes visible), a wait on
    a never-recorded event passes, and the host wait returns only after the
    recorded work."""
    a = torch.cuda.Stream(device=dev)
    b = torch.cuda.Stream(device=dev)
    x = torch.zeros(1 << 24, dtype=torch.float32, device=dev)
    y = torch.empty_like(x)
    ev, fresh = shc.StreamEvent(), shc.StreamEvent()
    torch.cuda.synchronize()
    for rep in range(3):
        with torch.cuda.stream(a):
            for _ in range(30):
                x.add_(1.0)
        ev.record(a)
        fresh.wait(b)
        ev.wait(b)
        with torch.cuda.stream(b):
            y.copy_(x)
        torch.cuda.synchronize()
        assert torch.all(y == 30.0 * (rep + 1))
    done = torch.cuda.Event()
    with torch.cuda.stream(a):
        for _ in range(30):
            x.add_(1.0)
        done.record(a)
    ev.record(a)
    ev.synchronize()
    assert done.query()          # everything recorded before the event has finished
    torch.cuda.synchronize()
    assert torch.all(x == 120.0)


@pytest.mark.parametrize("B,V,K,p,cap_delta", [
    (5, 655, 9, 0.1, None),       # 256-thread blocks, one pass
    (3, 4096, 9, 0.3, None),      # 256-thread blocks, two passes
    (4, 4097, 9, 0.05, None),     # 1024-thread blocks, odd body starts
    (3, 10475, 9, 0.05, None),    # 1024-thread blocks, the mesh size of the 10,475-vertex bodies
    (2, 19456, 5, 0.5, None),     # the largest V, two passes
    (7, 333, 32, 0.4, None),      # 32 slots
    (2, 5000, 32, 0.3, None),     # 32 slots, 1024-thread blocks
    (6, 97, 1, 0.9, None),        # one slot
    (9, 211, 9, 0.0, None),       # empty mask
    (4, 300, 9, 1.0, None),       # every vertex active
    (3, 1000, 9, 0.2, 0),         # cap = N' exactly
    (3, 1000, 9, 0.2, -5),        # cap below N': capacity error, table untouched
    (1, 5, 3, 0.6, None),         # tiny body, last bytes of the mask
    (128, 10475, 9, 0.05, None),  # the density-sweep batch
    (200, 655, 9, 0.1, None),     # 200 small bodies
    (3000, 40, 9, 0.3, None),     # many tiny bodies
])
def test_compact_table_start(dev, B, V, K, p, cap_delta):
    """shc_compact_mask_table_start: the lists of the compaction (Eq. 2), bit
    for bit as the oracle's, and the neighbour-row table of its active set
    (the rows each slot of Eqs. 4-5 reads, written out from the oracle's
    compaction), with row stride N'."""
    rng = np.random.default_rng(B * 1000 + V + K)
    m = (rng.random((B, V)) < p).astype(np.uint8)
    nbr = rand_nbr(V, K, rng)
    nbr[rng.random((V, K)) < 0.05] = V + 3          # out-of-range entries read as absent
    ref_c, ref_inv, ref_rp, ref_n = O.compact(m)
    cap = B * V if cap_delta is None else max(ref_n + cap_delta, 0)
    c = Compaction(m, cap)
    table = torch.full((K * max(cap, 1) + 5,), -7, dtype=torch.int32, device=dev)
    pc = shc.PreparedCompact(c.mask, B, V, c.coords, c.inv, c.row_ptr, c.n_dev, c.ws,
                             nbr=up(nbr), table=table)
    pc.start()
    if cap < ref_n:
        with pytest.raises(shc.ShcError, match="exceed"):
            pc.wait()
        torch.cuda.synchronize()
        assert np.all(down(table) == -7)
        assert np.array_equal(down(c.inv), ref_inv)
        assert np.array_equal(down(c.coords)[:cap], ref_c[:cap])
        return
    n = pc.wait()
    torch.cuda.synchronize()
    assert n == ref_n == int(down(c.n_dev)[0])
    assert np.array_equal(down(c.coords)[:n], ref_c)
    assert np.array_equal(down(c.inv), ref_inv)
    assert np.array_equal(down(c.row_ptr), ref_rp)
    got_t = down(table)
    assert np.array_equal(got_t[:K * n].reshape(K, n), table_reference(m, nbr))
    assert np.all(got_t[K * n:] == -7)


@pytest.mark.parametrize("B,V", [(128, 10475), (300, 655)])
def test_compact_table_start_any_workspace(dev, B, V):
    """The compaction with its table: exact whatever the workspace held
    before (random bytes, then the counts of earlier calls on other masks),
    over calls in a row."""
    K = 9
    rng = np.random.default_rng(B + V)
    nbr = rand_nbr(V, K, rng)
    masks = [(rng.random((B, V)) < p).astype(np.uint8) for p in (0.05, 0.3, 0.0, 0.05)]
    c = Compaction(masks[0])
    table = torch.full((K * B * V,), -7, dtype=torch.int32, device=dev)
    c.ws.copy_(torch.from_numpy(rng.integers(0, 256, c.ws.numel(), dtype=np.uint8)).to(dev))
    pc = shc.PreparedCompact(c.mask, B, V, c.coords, c.inv, c.row_ptr, c.n_dev, c.ws,
                             nbr=up(nbr), table=table)
    for m in masks:
        c.mask.copy_(up(m.reshape(-1)))
        ref_c, ref_inv, ref_rp, ref_n = O.compact(m)
        pc.start()
        n = pc.wait()
        torch.cuda.synchronize()
        assert n == ref_n
        assert np.array_equal(down(c.coords)[:n], ref_c)
        assert np.array_equal(down(c.inv), ref_inv)
        assert np.array_equal(down(c.row_ptr), ref_rp)
        assert np.array_equal(down(table)[:K * n].reshape(K, n), table_reference(m, nbr))


@pytest.mark.parametrize("steps", [1, 4])
def test_overlapped_run_conv_only_stack(dev, steps):
    """SparseStack.run with a side stream on a stack of four convs that ends in
    the pool (no fused gather, several layers before the double-buffered last
    one): a new mask and new features per batch; the outputs left behind must
    be the oracle's for the last batch."""
    from paper_2608_09388_amd.pipeline import SparseStack, to_device
    w = synth.workload_c2()
    w.B = 12
    w.mask = w.mask[:12]
    w.x = w.x[: 12 * w.V]
    rng = np.random.default_rng(700 + steps)
    masks = [(rng.random((w.B, w.V)) < p).astype(np.uint8) for p in (0.1, 0.3, 0.05, 0.2)][:steps]
    xs = [synth.as_dtype(rng.standard_normal(w.x.shape).astype(np.float32), w.dtype)[1]
          for _ in range(steps)]
    st = SparseStack(w, device=str(dev), side_stream=True)
    st.run(3)

    def feed(k):
        st.mask.copy_(up(masks[k].reshape(-1)))
        st.x.copy_(to_device(xs[k], w.dtype, st.device))

    n = st.run(steps, feed=feed)
    spec = [(l.kind, l.W, l.bias, l.relu) for l in w.layers]
    ref = O.run_stack(xs[-1], masks[-1], w.nbr, spec, w.dtype, pool=True)
    got = st.results()
    assert n == ref["n"] == got["n"]
    for l in range(len(w.layers)):
        assert_normwise_close(got["outs"][l], ref["outs"][l], w.dtype, f"layer {l}")
    assert_normwise_close(got["pool"], ref["pool"], w.dtype, "pool")


def test_overlapped_run_table_on_its_own(dev):
    """Bodies of more vertices than the compaction keeps on chip (V = 20000):
    the side stream builds the neighbour-row table with its own call after the
    compaction.  A new mask and new features per batch over three batches;
    the outputs left behind must be the oracle's for the last batch."""
    from paper_2608_09388_amd.pipeline import SparseStack, to_device
    w = synth.workload_c4(0.05, B=2, V=20000)
    rng = np.random.default_rng(901)
    masks = [(rng.random((w.B, w.V)) < p).astype(np.uint8) for p in (0.05, 0.2, 0.1)]
    xs = [synth.as_dtype(rng.standard_normal(w.x.shape).astype(np.float32), w.dtype)[1]
          for _ in range(3)]
    st = SparseStack(w, device=str(dev), side_stream=True)
    assert not st._set.fused and st._set.table_side is not None
    st.run(2)

    def feed(k):
        st.mask.copy_(up(masks[k].reshape(-1)))
        st.x.copy_(to_device(xs[k], w.dtype, st.device))

    n = st.run(3, feed=feed)
    spec = [(l.kind, l.W, l.bias, l.relu) for l in w.layers]
    ref = O.run_stack(xs[-1], masks[-1], w.nbr, spec, w.dtype, pool=True)
    got = st.results()
    assert n == ref["n"] == got["n"]
    assert np.array_equal(got["coords"], ref["coords"])
    for l in range(len(w.layers)):
        assert_normwise_close(got["outs"][l], ref["outs"][l], w.dtype, f"layer {l}")
    assert_normwise_close(got["dense"], O.scatter(ref["outs"][-1], ref["inv"], zero_fill=True),
                          w.dtype, "dense")
    assert_normwise_close(got["pool"], ref["pool"], w.dtype, "pool")


@pytest.mark.parametrize("B,V,K,Cout,p", [
    (4, 3000, 9, 128, 0.05),     # few rows per workgroup
    (6, 2000, 10, 64, 0.3),      # ten slots, Cout 64
    (3, 1000, 1, 128, 0.5),      # one slot
    (5, 1500, 4, 16, 0.9),       # four slots, Cout 16, dense mask
    (90, 10475, 9, 128, 0.1),    # about 94 K rows
    (128, 10475, 9, 128, 0.05),  # the density-sweep batch at 5%
])
def test_conv_cin128_table_parity(dev, B, V, K, Cout, p):
    """The bf16 conv from a table with C_in = 128, at row counts from one small
    workgroup per CU to the density-sweep batch, against the oracle on sampled
    rows plus the first and last 400 rows, and bit for bit against the direct
    path (index lists built from coords, inv and nbr inside the kernel)."""
    rng = np.random.default_rng(B * 17 + V + K * 3 + Cout)
    m = (rng.random((B, V)) < p).astype(np.uint8)
    nbr = rand_nbr(V, K, rng)
    coords, inv, rp, n = O.compact(m)
    S = synth.as_dtype(rng.standard_normal((n, 128)).astype(np.float32), "bf16")[1]
    W = synth.as_dtype((rng.standard_normal((K, 128, Cout)) / np.sqrt(K * 128))
                       .astype(np.float32), "bf16")[1]
    bias = rng.standard_normal(Cout).astype(np.float32)
    g_tab, n2 = run_conv(dev, m, nbr, S, W, bias, "bf16", shc.SHC_ACT_RELU, "table")
    g_dir, _ = run_conv(dev, m, nbr, S, W, bias, "bf16", shc.SHC_ACT_RELU, "direct")
    assert n2 == n
    assert np.array_equal(g_tab, g_dir)
    rows = np.unique(np.concatenate([np.arange(min(n, 400)), np.arange(max(0, n - 400), n),
                                     rng.choice(n, size=min(n, 600), replace=False)]))
    ref = O.conv_at(S, coords, B, V, nbr, W, rows, bias, act=True)
    scale = O.conv_at(S, coords, B, V, nbr, W, rows, bias, scale=True)
    assert_scaled_close(g_tab[rows], ref, scale, "bf16", f"conv K={K} 128->{Cout} p={p}",
                        n_terms=K * 128)
