"""Parity of the backward kernels (through the C ABI) with the CPU oracle.

Integer structures (transposed neighbour lists, transposed table) are checked
bit-exactly against a numpy construction.  Gradients against the oracle's
fp64 backward on the same inputs: dS within 2e-2 (bf16) or 1e-5 (fp32) of the
abs-sum scale of its terms, dW and db (fp32) within 1e-5 of theirs.  The stored
output Y that decides the ReLU's derivative is a seeded input on both sides.
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


def expected_transpose(nbr):
    """Senders of u through slot j, ascending, laid out in virtual slots."""
    V, K = nbr.shape
    lists = [[[] for _ in range(K)] for _ in range(V)]
    for v in range(V):
        for j in range(K):
            u = int(nbr[v, j])
            if 0 <= u < V:
                lists[u][j].append(v)
    m = [max(len(lists[u][j]) for u in range(V)) for j in range(K)]
    off = np.concatenate([[0], np.cumsum(m)]).astype(int)
    Kt = int(off[-1])
    tv = np.full((V, Kt), -1, np.int32)
    for u in range(V):
        for j in range(K):
            for c, v in enumerate(sorted(lists[u][j])):
                tv[u, off[j] + c] = v
    slot_of = np.repeat(np.arange(K), m).astype(np.int32)
    return tv, slot_of, Kt


def bf16(a):
    return synth.as_dtype(np.asarray(a, np.float32), "bf16")[1]


def exact(a, dtype):
    """Values exactly representable in dtype ('bf16' or 'f32')."""
    return synth.as_dtype(np.asarray(a, np.float32), dtype)[1]


TDT = {"bf16": torch.bfloat16, "f32": torch.float32}


class ConvSetup:
    """Active set, neighbour-row table and transposed table on the GPU."""

    def __init__(self, mask, nbr):
        self.B, self.V = mask.shape
        self.K = nbr.shape[1]
        self.c = Compaction(mask)
        self.n = self.c.run(want_host=True)
        self.coords = down(self.c.coords)[: self.n]
        self.nbr_d = up(nbr)
        n = max(self.n, 1)
        self.table = torch.empty((self.K, n), dtype=torch.int32, device="cuda")
        if self.n > 0:
            shc.build_neighbor_table(self.c.coords, self.c.inv, self.n, self.B, self.V,
                                     self.nbr_d, self.table)
        self.nbr_t, self.slot_of, self.Kt = shc.transpose_neighbors(self.nbr_d)
        self.table_t = torch.empty((self.Kt, n), dtype=torch.int32, device="cuda")
        self.row_slots = torch.empty(n, dtype=torch.int64, device="cuda")
        if self.n > 0:
            shc.build_transposed_table(self.c.coords, self.c.inv, self.n, self.B, self.V,
                                       self.nbr_t, self.Kt, self.table_t, self.row_slots)


def conv_inputs(rng, n, K, Cin, Cout, dtype="bf16"):
    S = exact(rng.standard_normal((n, Cin)), dtype)
    W = exact(rng.standard_normal((K, Cin, Cout)) / np.sqrt(K * Cin), dtype)
    Y = exact(np.maximum(rng.standard_normal((n, Cout)), 0.0), dtype)   # half exact zeros
    dY = exact(rng.standard_normal((n, Cout)), dtype)
    return S, W, Y, dY


def run_conv_backward(st, S, W, Y, dY, act, want=("dS", "dW", "db"), with_pairs=False,
                      dtype="bf16"):
    n, K = st.n, st.K
    Cin, Cout = W.shape[1], W.shape[2]
    dS = torch.full((max(n, 1), Cin), float("nan"), dtype=TDT[dtype], device="cuda")
    dW = torch.full((K, Cin, Cout), float("nan"), dtype=torch.float32, device="cuda")
    db = torch.full((Cout,), float("nan"), dtype=torch.float32, device="cuda")
    Sd = up(S if n else np.zeros((1, Cin)), dtype)
    Yd = up(Y if n else np.zeros((1, Cout)), dtype)
    dYd = up(dY if n else np.zeros((1, Cout)), dtype)
    pairs = pair_ptr = None
    if with_pairs:
        pairs = torch.full((max(K * n, 1), 2), -7, dtype=torch.int32, device="cuda")
        pair_ptr = torch.full((K + 1,), -7, dtype=torch.int32, device="cuda")
        shc.build_slot_pairs(st.table, n, K, pairs, pair_ptr)
    shc.sparse_neighbor_conv_backward(
        Sd, st.table, st.table_t, st.row_slots, st.slot_of, st.Kt, up(W, dtype), Yd, dYd, n,
        dS if "dS" in want else None, dW if "dW" in want else None,
        db if "db" in want else None, act=shc.SHC_ACT_RELU if act else shc.SHC_ACT_NONE,
        pairs=pairs, pair_ptr=pair_ptr)
    torch.cuda.synchronize()
    return down(dS)[:n], down(dW), down(db)


def check_conv(st, nbr, S, W, Y, dY, act, with_pairs=False, dtype="bf16"):
    B, V = st.B, st.V
    gS, gW, gb = run_conv_backward(st, S, W, Y, dY, act, with_pairs=with_pairs, dtype=dtype)
    rS, rW, rb = O.sparse_conv_backward(S, st.coords, B, V, nbr, W, dY, Y, act)
    dZ = O.relu_backward(dY, Y) if act else np.asarray(dY, np.float64)
    sS, sW, sb = O.sparse_conv_backward(np.abs(S), st.coords, B, V, nbr, np.abs(W), np.abs(dZ))
    # a row receives at most one term per virtual slot and output channel
    assert_scaled_close(gS, rS, sS, dtype, "dS", n_terms=st.Kt * W.shape[2])
    assert_scaled_close(gW, rW, sW, "f32", "dW")
    assert_scaled_close(gb, rb, sb, "f32", "db")
    return gS, gW, gb


# ----------------------------------------------------------------------------
# transposed structures (exact)
# ----------------------------------------------------------------------------


@pytest.mark.parametrize("V,K,seed", [(40, 4, 1), (300, 9, 2), (7, 1, 3)])
def test_transpose_neighbors_exact(dev, V, K, seed):
    rng = np.random.default_rng(seed)
    nbr = rand_nbr(V, K, rng)
    if K > 1:
        nbr[3, 1] = V + 5                  # out of range: no neighbour
    tv, slot_of, Kt = expected_transpose(nbr)
    nbr_t, so, kt = shc.transpose_neighbors(up(nbr))
    assert kt == Kt
    got = down(nbr_t)
    assert np.array_equal(got.reshape(-1)[: V * Kt].reshape(V, Kt), tv)
    assert np.all(got.reshape(-1)[V * Kt:] == -1)
    assert np.array_equal(down(so)[:Kt], slot_of) and np.all(down(so)[Kt:] == -1)


def test_transpose_neighbors_knn_mesh(dev):
    w = synth.workload_c4(0.05, B=2)
    tv, slot_of, Kt = expected_transpose(w.nbr)
    nbr_t, so, kt = shc.transpose_neighbors(up(np.ascontiguousarray(w.nbr, np.int32)))
    assert kt == Kt <= shc.SHC_MAX_VIRTUAL_SLOTS
    assert np.array_equal(down(nbr_t).reshape(-1)[: w.V * Kt].reshape(w.V, Kt), tv)


def test_transposed_table_exact(dev):
    rng = np.random.default_rng(5)
    B, V, K = 3, 60, 5
    nbr = rand_nbr(V, K, rng)
    mask = (rng.random((B, V)) < 0.4).astype(np.uint8)
    st = ConvSetup(mask, nbr)
    tv, slot_of, Kt = expected_transpose(nbr)
    coords, inv, rp, n = O.compact(mask)
    want = np.full((Kt, n), -1, np.int64)
    bits = np.zeros(n, np.uint64)
    for r in range(n):
        b, u = coords[r]
        for s in range(Kt):
            v = tv[u, s]
            if v >= 0 and inv[b * V + v] >= 0:
                want[s, r] = inv[b * V + v]
                bits[r] |= np.uint64(1) << np.uint64(s)
    assert np.array_equal(down(st.table_t)[:, :n], want)
    assert np.array_equal(st.row_slots[:n].cpu().numpy().view(np.uint64), bits)


# ----------------------------------------------------------------------------
# conv and linear gradients against the oracle
# ----------------------------------------------------------------------------


@pytest.mark.parametrize("B,V,K,Cin,Cout,p,act,dtype", [
    (3, 200, 9, 128, 128, 0.3, True, "bf16"),      # both tile edges at 128
    (4, 150, 9, 64, 128, 0.5, True, "bf16"),
    (2, 333, 5, 16, 64, 0.2, False, "bf16"),       # narrow input, no activation
    (5, 97, 3, 48, 32, 0.7, True, "bf16"),         # ragged channel tiles
    (2, 700, 9, 128, 256, 0.05, True, "bf16"),     # sparse, wide output
    (1, 50, 9, 32, 16, 1.0, True, "bf16"),         # every vertex active
    (3, 200, 9, 128, 128, 0.3, True, "f32"),
    (2, 333, 5, 16, 64, 0.2, False, "f32"),
    (2, 400, 9, 64, 192, 0.1, True, "f32"),        # 12 fp32 k-steps (the 16-step path)
    (5, 97, 3, 48, 32, 0.7, True, "f32"),
])
def test_conv_backward_vs_oracle(dev, B, V, K, Cin, Cout, p, act, dtype):
    rng = np.random.default_rng(B * 1000 + V + K + Cin)
    nbr = rand_nbr(V, K, rng)
    mask = (rng.random((B, V)) < p).astype(np.uint8)
    st = ConvSetup(mask, nbr)
    assert st.n > 0
    S, W, Y, dY = conv_inputs(rng, st.n, K, Cin, Cout, dtype)
    # half of the cases take slot pairs built once beforehand, as a stack would
    check_conv(st, nbr, S, W, Y, dY, act, with_pairs=(Cin + Cout) % 3 == 0, dtype=dtype)


@pytest.mark.parametrize("n,Cin,Cout,act,dtype", [
    (1000, 128, 128, True, "bf16"), (37, 64, 32, False, "bf16"), (5000, 16, 256, True, "bf16"),
    (1, 128, 64, True, "bf16"), (1000, 128, 128, True, "f32"), (37, 64, 32, False, "f32"),
    (3000, 48, 256, True, "f32"),
    # the one-pass bf16 kernel (C_in, C_out in {64, 128}): several workgroups
    # with a ragged last one, a single short one, no ReLU
    (70001, 128, 128, True, "bf16"), (300, 64, 64, False, "bf16"), (2049, 64, 128, True, "bf16"),
    (513, 128, 64, False, "bf16"), (31, 64, 64, True, "bf16")])
def test_linear_backward_vs_oracle(dev, n, Cin, Cout, act, dtype):
    rng = np.random.default_rng(n + Cin + Cout)
    S = exact(rng.standard_normal((n, Cin)), dtype)
    W = exact(rng.standard_normal((Cin, Cout)) / np.sqrt(Cin), dtype)
    Y = exact(np.maximum(rng.standard_normal((n, Cout)), 0.0), dtype)
    dY = exact(rng.standard_normal((n, Cout)), dtype)
    dS = torch.empty((n, Cin), dtype=TDT[dtype], device="cuda")
    dW = torch.empty((Cin, Cout), dtype=torch.float32, device="cuda")
    db = torch.empty(Cout, dtype=torch.float32, device="cuda")
    shc.sparse_linear_backward(up(S, dtype), up(W, dtype), up(Y, dtype), up(dY, dtype), n,
                               dS, dW, db, act=shc.SHC_ACT_RELU if act else shc.SHC_ACT_NONE)
    torch.cuda.synchronize()
    rS, rW, rb = O.sparse_linear_backward(S, W, dY, Y, act)
    dZ = O.relu_backward(dY, Y) if act else np.asarray(dY, np.float64)
    sS, sW, sb = O.sparse_linear_backward(np.abs(S), np.abs(W), np.abs(dZ))
    assert_scaled_close(down(dS), rS, sS, dtype, "dS", n_terms=Cout)
    assert_scaled_close(down(dW), rW, sW, "f32", "dW")
    assert_scaled_close(down(db), rb, sb, "f32", "db")


@pytest.mark.parametrize("Cin,Cout", [(128, 128), (64, 128)])
def test_linear_backward_outputs_one_at_a_time(dev, Cin, Cout):
    """Each output of the linear backward asked for alone equals the same
    output of the call that asks for all three, bit for bit, and the outputs
    not asked for stay untouched; two full calls agree bit for bit."""
    rng = np.random.default_rng(Cin + 3 * Cout)
    n = 9001
    S = bf16(rng.standard_normal((n, Cin)))
    W = bf16(rng.standard_normal((Cin, Cout)) / np.sqrt(Cin))
    Y = bf16(np.maximum(rng.standard_normal((n, Cout)), 0.0))
    dY = bf16(rng.standard_normal((n, Cout)))
    args = [up(S, "bf16"), up(W, "bf16"), up(Y, "bf16"), up(dY, "bf16"), n]

    def run(want):
        dS = torch.full((n, Cin), float("nan"), dtype=torch.bfloat16, device="cuda")
        dW = torch.full((Cin, Cout), float("nan"), dtype=torch.float32, device="cuda")
        db = torch.full((Cout,), float("nan"), dtype=torch.float32, device="cuda")
        shc.sparse_linear_backward(*args, dS if "dS" in want else None,
                                   dW if "dW" in want else None, db if "db" in want else None)
        torch.cuda.synchronize()
        return down(dS), down(dW), down(db)

    full = run(("dS", "dW", "db"))
    again = run(("dS", "dW", "db"))
    for x, y in zip(full, again):
        assert np.array_equal(x, y)
    for k, name in enumerate(("dS", "dW", "db")):
        got = run((name,))
        assert np.array_equal(got[k], full[k]), name
        for m in range(3):
            if m != k:
                assert np.all(np.isnan(got[m])), (name, m)


def test_conv_backward_self_slot_is_linear_and_repeats(dev):
    """K = 1 self slot gives the linear layer's gradients; two runs agree bit for bit;
    asking for one output leaves the others untouched."""
    rng = np.random.default_rng(11)
    B, V = 2, 400
    nbr = np.arange(V, dtype=np.int32)[:, None]
    mask = (rng.random((B, V)) < 0.5).astype(np.uint8)
    st = ConvSetup(mask, nbr)
    S, W, Y, dY = conv_inputs(rng, st.n, 1, 64, 128)
    a = run_conv_backward(st, S, W, Y, dY, True)
    b = run_conv_backward(st, S, W, Y, dY, True)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    n = st.n
    dS = torch.empty((n, 64), dtype=torch.bfloat16, device="cuda")
    dW = torch.empty((64, 128), dtype=torch.float32, device="cuda")
    db = torch.empty(128, dtype=torch.float32, device="cuda")
    shc.sparse_linear_backward(up(S, "bf16"), up(W[0], "bf16"), up(Y, "bf16"), up(dY, "bf16"),
                               n, dS, dW, db)
    torch.cuda.synchronize()
    assert np.array_equal(down(dS), a[0])
    # the linear layer's one-pass kernel sums dW and db over its own row
    # chunks: the same values up to the order of the fp32 partial sums
    np.testing.assert_allclose(down(dW), a[1][0], rtol=0, atol=1e-6 * np.abs(a[1]).max())
    np.testing.assert_allclose(down(db), a[2], rtol=0, atol=1e-6 * np.abs(a[2]).max())
    only = run_conv_backward(st, S, W, Y, dY, True, want=("db",))
    assert np.all(np.isnan(only[0])) and np.all(np.isnan(only[1]))
    assert np.array_equal(only[2], a[2])


def test_slot_pairs_exact_and_shared(dev):
    """Slot pair lists are the slot-major (j, i) of every present table entry;
    a conv backward given them equals one that builds its own, bit for bit."""
    rng = np.random.default_rng(13)
    B, V, K = 3, 90, 6
    nbr = rand_nbr(V, K, rng)
    mask = (rng.random((B, V)) < 0.35).astype(np.uint8)
    st = ConvSetup(mask, nbr)
    n = st.n
    pairs = torch.full((K * n, 2), -7, dtype=torch.int32, device="cuda")
    pair_ptr = torch.full((K + 1,), -7, dtype=torch.int32, device="cuda")
    shc.build_slot_pairs(st.table, n, K, pairs, pair_ptr)
    torch.cuda.synchronize()
    tab = down(st.table).reshape(-1)[: K * n].reshape(K, n)
    want = np.array([(j, i) for j in range(K) for i in range(n) if tab[j, i] >= 0], np.int32)
    ptr = down(pair_ptr)
    assert ptr[0] == 0 and ptr[-1] == len(want)
    assert np.array_equal(down(pairs)[: len(want)], want)
    assert np.array_equal(np.diff(ptr), [(tab[j] >= 0).sum() for j in range(K)])
    S, W, Y, dY = conv_inputs(rng, n, K, 64, 64)
    a = run_conv_backward(st, S, W, Y, dY, True)
    b = run_conv_backward(st, S, W, Y, dY, True, with_pairs=True)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_conv_backward_empty_active_set(dev):
    rng = np.random.default_rng(12)
    nbr = rand_nbr(30, 4, rng)
    st = ConvSetup(np.zeros((2, 30), np.uint8), nbr)
    assert st.n == 0
    S, W, Y, dY = conv_inputs(rng, 0, 4, 32, 32)
    gS, gW, gb = run_conv_backward(st, S, W, Y, dY, True)
    assert gS.shape == (0, 32)
    assert np.all(gW == 0) and np.all(gb == 0)


def test_conv_backward_c4_full_size(dev):
    """The density-sweep workload at 5% (B = 128, V = 10475 kNN mesh, K = 9,
    C = 128 bf16): dW and db in full, dS on sampled rows, all against the
    oracle on the oracle's own compaction of the mask."""
    w = synth.workload_c4(0.05)
    nbr = np.ascontiguousarray(w.nbr, np.int32)
    st = ConvSetup(w.mask, nbr)
    coords, inv, rp, n = O.compact(w.mask)
    assert st.n == n and np.array_equal(st.coords, coords)
    rng = np.random.default_rng(99)
    S, W, Y, dY = conv_inputs(rng, n, w.K, 128, 128)
    gS, gW, gb = run_conv_backward(st, S, W, Y, dY, True)
    dZ = O.relu_backward(dY, Y)
    B, V = w.B, w.V
    rW, rb = O.conv_backward_weight_bias(S, coords, B, V, nbr, dZ, w.K)
    sW, sb = O.conv_backward_weight_bias(S, coords, B, V, nbr, dZ, w.K, scale=True)
    assert_scaled_close(gW, rW, sW, "f32", "dW")
    assert_scaled_close(gb, rb, sb, "f32", "db")
    rows = np.unique(np.concatenate([rng.choice(n, 48, replace=False), [0, n - 1]]))
    rS = O.conv_backward_input_at(coords, B, V, nbr, W, dZ, rows)
    sS = O.conv_backward_input_at(coords, B, V, nbr, W, dZ, rows, scale=True)
    assert_scaled_close(gS[rows], rS, sS, "bf16", "dS rows", n_terms=st.Kt * 128)
