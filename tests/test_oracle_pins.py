"""Pins of the CPU oracle against facts other than its own formulas.

Each operator of the oracle is checked against something that does not reuse
its code: a library routine that computes the same thing by another route
(numpy.flatnonzero, scipy.sparse products, numpy.maximum.reduceat, torch's
bfloat16 conversion), exact rational arithmetic, closed forms and special
cases the paper's definitions reduce to, invariants (linearity, relabelling
equivariance, masking), and pure-Python brute force on tiny meshes.  The
cases are chosen so that a dropped term, a wrong sign, a wrong index or a
transposed operand in the oracle makes at least one of them fail.
"""
import itertools
from fractions import Fraction

import numpy as np
import pytest
import scipy.sparse as sp
import torch

from oracle import shc_oracle as O

RNG = np.random.default_rng(20240611)


def rand_nbr(V, K, rng, p_missing=0.15, self_first=True):
    """Random neighbour lists with -1 holes (not a geometric kNN on purpose)."""
    nbr = rng.integers(0, V, size=(V, K)).astype(np.int32)
    nbr[rng.random((V, K)) < p_missing] = -1
    if self_first:
        nbr[:, 0] = np.arange(V)
    return nbr


# ----------------------------------------------------------------------------
# compaction (Eq. 2)
# ----------------------------------------------------------------------------


def brute_compact(m):
    B, V = len(m), len(m[0])
    coords, inv, row_ptr = [], [-1] * (B * V), []
    for b in range(B):
        row_ptr.append(len(coords))
        for v in range(V):
            if m[b][v] != 0:
                inv[b * V + v] = len(coords)
                coords.append((b, v))
    row_ptr.append(len(coords))
    return coords, inv, row_ptr


@pytest.mark.parametrize("B,V", [(1, 10), (3, 4)])
def test_compact_exhaustive_tiny(B, V):
    n_bits = B * V
    for code in range(1 << n_bits):
        m = np.array([(code >> k) & 1 for k in range(n_bits)], dtype=np.uint8).reshape(B, V)
        coords, inv, row_ptr, n = O.compact(m)
        bc, binv, brp = brute_compact(m.tolist())
        assert n == len(bc)
        assert [tuple(r) for r in coords.tolist()] == bc
        assert inv.tolist() == binv
        assert row_ptr.tolist() == brp


@pytest.mark.parametrize("B,V,p", [(5, 655, 0.1), (2, 10475, 0.05), (7, 33, 0.0),
                                   (4, 17, 1.0), (1, 1, 1.0), (300, 3, 0.5)])
def test_compact_vs_flatnonzero(B, V, p):
    m = (RNG.random((B, V)) < p).astype(np.uint8)
    m[m != 0] = RNG.integers(1, 256, size=int(m.sum()))     # any non-zero byte is active
    coords, inv, row_ptr, n = O.compact(m)
    nz = np.flatnonzero(m.ravel())
    b, v = np.divmod(nz, V)
    assert n == nz.size
    assert np.array_equal(coords[:, 0], b) and np.array_equal(coords[:, 1], v)
    expect_rp = np.concatenate([[0], np.cumsum((m != 0).sum(1))])
    assert np.array_equal(row_ptr, expect_rp)
    # invariants
    assert np.array_equal(inv[nz], np.arange(n))
    assert np.all(inv[m.ravel() == 0] == -1)
    assert np.all(np.diff(row_ptr) == (m != 0).sum(1))


# ----------------------------------------------------------------------------
# gather / scatter
# ----------------------------------------------------------------------------


def test_scatter_gather_roundtrip():
    B, V, C = 3, 50, 8
    m = (RNG.random((B, V)) < 0.3).astype(np.uint8)
    x = RNG.standard_normal((B * V, C)).astype(np.float32)
    coords, inv, row_ptr, n = O.compact(m)
    S = O.gather(x, coords, V)
    D = O.scatter(S, inv, zero_fill=True)
    assert np.array_equal(D, x * m.reshape(-1, 1))               # scatter o gather = x (.) m
    assert np.array_equal(O.gather(D, coords, V), S)             # gather o scatter = id
    # active-only scatter leaves inactive rows untouched
    sentinel = np.full_like(x, np.nan)
    D2 = O.scatter(S, inv, zero_fill=False, D=sentinel)
    assert np.all(np.isnan(D2[inv < 0])) and np.array_equal(D2[inv >= 0], S)
    assert np.array_equal(O.densify(S, coords, B, V), D)


# ----------------------------------------------------------------------------
# linear layer (Eq. 6)
# ----------------------------------------------------------------------------


def test_linear_density_one_is_library_linear():
    B, V, Ci, Co = 2, 30, 16, 24
    x = RNG.standard_normal((B * V, Ci))
    W = RNG.standard_normal((Ci, Co))
    b = RNG.standard_normal(Co)
    m = np.ones((B, V), np.uint8)
    coords, inv, rp, n = O.compact(m)
    got = O.sparse_linear(O.gather(x, coords, V), coords, B, V, W, b)
    ref = torch.nn.functional.linear(torch.from_numpy(x), torch.from_numpy(W.T.copy()),
                                     torch.from_numpy(b)).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-13)


def test_linear_rows_are_independent_and_masked():
    B, V, Ci, Co = 2, 40, 8, 8
    m = (RNG.random((B, V)) < 0.3).astype(np.uint8)
    coords, inv, rp, n = O.compact(m)
    S = RNG.standard_normal((n, Ci))
    W = RNG.standard_normal((Ci, Co))
    b = RNG.standard_normal(Co)
    got = O.sparse_linear(S, coords, B, V, W, b, act=True)
    # closed form per row, in pure Python
    for i in range(n):
        for c in range(Co):
            acc = b[c] + sum(float(S[i, k]) * float(W[k, c]) for k in range(Ci))
            assert got[i, c] == pytest.approx(max(acc, 0.0), rel=1e-12, abs=1e-12)


# ----------------------------------------------------------------------------
# convolution (Eqs. 4-5)
# ----------------------------------------------------------------------------


def brute_conv(x, m, nbr, W, bias, B, V, act):
    """Pure-Python loops: output at active (b, v) only, neighbours present in C."""
    K, Ci, Co = W.shape
    rows = []
    for b in range(B):
        for v in range(V):
            if not m[b][v]:
                continue
            out = []
            for c in range(Co):
                acc = 0.0 if bias is None else float(bias[c])
                for j in range(K):
                    u = int(nbr[v][j])
                    if u < 0 or not m[b][u]:
                        continue
                    for k in range(Ci):
                        acc += float(x[b * V + u][k]) * float(W[j][k][c])
                out.append(max(acc, 0.0) if act else acc)
            rows.append(out)
    return np.array(rows, dtype=np.float64).reshape(-1, Co)


@pytest.mark.parametrize("B,V,K,Ci,Co,p", [(1, 6, 3, 2, 3, 0.6), (3, 11, 9, 4, 2, 0.5),
                                           (2, 24, 5, 8, 3, 0.3), (2, 9, 1, 3, 5, 1.0)])
def test_conv_brute_force_tiny(B, V, K, Ci, Co, p):
    rng = np.random.default_rng(B * 100 + V)
    m = (rng.random((B, V)) < p).astype(np.uint8)
    nbr = rand_nbr(V, K, rng)
    x = rng.standard_normal((B * V, Ci))
    W = rng.standard_normal((K, Ci, Co))
    bias = rng.standard_normal(Co)
    coords, inv, rp, n = O.compact(m)
    for act in (False, True):
        got = O.sparse_conv(O.gather(x, coords, V), coords, B, V, nbr, W, bias, act)
        ref = brute_conv(x, m, nbr, W, bias, B, V, act)
        np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_conv_equals_scipy_sparse_adjacency_products():
    """y_b = sum_j A_j (x_b (.) m_b) W_j with A_j[v, nbr[v,j]] = 1 (scipy sparse)."""
    B, V, K, Ci, Co = 3, 200, 9, 6, 7
    m = (RNG.random((B, V)) < 0.25).astype(np.uint8)
    nbr = rand_nbr(V, K, RNG)
    x = RNG.standard_normal((B * V, Ci))
    W = RNG.standard_normal((K, Ci, Co))
    coords, inv, rp, n = O.compact(m)
    got = O.sparse_conv(O.gather(x, coords, V), coords, B, V, nbr, W)
    ref_rows = []
    for b in range(B):
        xb = x[b * V:(b + 1) * V] * m[b][:, None]
        yb = np.zeros((V, Co))
        for j in range(K):
            valid = nbr[:, j] >= 0
            A = sp.csr_matrix((np.ones(valid.sum()), (np.flatnonzero(valid), nbr[valid, j])),
                              shape=(V, V))
            yb += A @ xb @ W[j]
        ref_rows.append(yb[m[b] != 0])
    np.testing.assert_allclose(got, np.concatenate(ref_rows), rtol=1e-12, atol=1e-12)


def test_conv_density_one_is_concatenated_spiral_conv():
    """At density 1 the conv equals concat_j(x[nbr(v, j)]) @ W.reshape(K*Ci, Co)."""
    B, V, K, Ci, Co = 2, 64, 9, 5, 3
    nbr = rand_nbr(V, K, RNG)
    x = RNG.standard_normal((B * V, Ci))
    W = RNG.standard_normal((K, Ci, Co))
    m = np.ones((B, V), np.uint8)
    coords, inv, rp, n = O.compact(m)
    got = O.sparse_conv(O.gather(x, coords, V), coords, B, V, nbr, W)
    xpad = np.concatenate([x.reshape(B, V, Ci), np.zeros((B, 1, Ci))], axis=1)
    idx = np.where(nbr >= 0, nbr, V)                   # -1 -> the zero row
    cat = xpad[:, idx, :].reshape(B * V, K * Ci)
    np.testing.assert_allclose(got, cat @ W.reshape(K * Ci, Co), rtol=1e-12, atol=1e-12)


def test_conv_single_self_slot_is_linear():
    B, V, Ci, Co = 2, 40, 6, 4
    m = (RNG.random((B, V)) < 0.5).astype(np.uint8)
    coords, inv, rp, n = O.compact(m)
    S = RNG.standard_normal((n, Ci))
    W = RNG.standard_normal((Ci, Co))
    b = RNG.standard_normal(Co)
    self_nbr = np.arange(V, dtype=np.int32)[:, None]
    got = O.sparse_conv(S, coords, B, V, self_nbr, W[None], b, act=True)
    ref = np.maximum(S @ W + b, 0.0)
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-13)


def test_conv_lone_active_vertex_sees_only_itself():
    V, K, Ci, Co = 30, 9, 4, 3
    nbr = rand_nbr(V, K, RNG, p_missing=0.0)
    nbr[7, 3] = 7                                   # self also in a second slot
    m = np.zeros((1, V), np.uint8)
    m[0, 7] = 1
    x = RNG.standard_normal((V, Ci))
    W = RNG.standard_normal((K, Ci, Co))
    b = RNG.standard_normal(Co)
    coords, inv, rp, n = O.compact(m)
    got = O.sparse_conv(O.gather(x, coords, V), coords, 1, V, nbr, W, b)
    selfslots = [j for j in range(K) if nbr[7, j] == 7]
    ref = b + sum(x[7] @ W[j] for j in selfslots)
    np.testing.assert_allclose(got[0], ref, rtol=1e-13, atol=1e-13)


def test_conv_is_linear_in_features():
    B, V, K, Ci, Co = 2, 50, 9, 4, 5
    m = (RNG.random((B, V)) < 0.4).astype(np.uint8)
    nbr = rand_nbr(V, K, RNG)
    coords, inv, rp, n = O.compact(m)
    W = RNG.standard_normal((K, Ci, Co))
    S1, S2 = RNG.standard_normal((n, Ci)), RNG.standard_normal((n, Ci))
    a = -1.75
    lhs = O.sparse_conv(a * S1 + S2, coords, B, V, nbr, W)
    rhs = a * O.sparse_conv(S1, coords, B, V, nbr, W) + O.sparse_conv(S2, coords, B, V, nbr, W)
    np.testing.assert_allclose(lhs, rhs, rtol=1e-11, atol=1e-11)


def test_conv_relabelling_equivariance():
    """Renumbering the vertices renumbers the outputs and nothing else."""
    B, V, K, Ci, Co = 2, 45, 9, 3, 4
    rng = np.random.default_rng(5)
    m = (rng.random((B, V)) < 0.5).astype(np.uint8)
    nbr = rand_nbr(V, K, rng)
    x = rng.standard_normal((B * V, Ci))
    W = rng.standard_normal((K, Ci, Co))
    perm = rng.permutation(V)                      # new label of old vertex u is perm[u]
    inv_perm = np.argsort(perm)
    nbr2 = np.where(nbr[inv_perm] >= 0, perm[np.maximum(nbr[inv_perm], 0)], -1).astype(np.int32)
    m2 = m[:, inv_perm]
    x2 = x.reshape(B, V, Ci)[:, inv_perm].reshape(B * V, Ci)
    c1, _, _, _ = O.compact(m)
    c2, _, _, _ = O.compact(m2)
    y1 = O.sparse_conv(O.gather(x, c1, V), c1, B, V, nbr, W)
    y2 = O.sparse_conv(O.gather(x2, c2, V), c2, B, V, nbr2, W)
    d1 = O.densify(y1, c1, B, V).reshape(B, V, Co)
    d2 = O.densify(y2, c2, B, V).reshape(B, V, Co)
    np.testing.assert_allclose(d2, d1[:, inv_perm], rtol=1e-12, atol=1e-12)


def test_conv_scalar_slot_weights_match_paper_eq5_literal():
    """W[j] = w_j * I gives the paper's scalar form: sum_j w_j * s[idx(nbr(v, j))]."""
    B, V, K, C = 2, 40, 9, 6
    rng = np.random.default_rng(9)
    m = (rng.random((B, V)) < 0.35).astype(np.uint8)
    nbr = rand_nbr(V, K, rng)
    w = rng.standard_normal(K)
    x = rng.standard_normal((B * V, C))
    coords, inv, rp, n = O.compact(m)
    S = O.gather(x, coords, V)
    got = O.sparse_conv(S, coords, B, V, nbr, w[:, None, None] * np.eye(C)[None])
    ref = np.zeros_like(S)
    for i, (b, v) in enumerate(coords):
        for j in range(K):
            u = nbr[v, j]
            if u >= 0 and inv[b * V + u] >= 0:
                ref[i] += w[j] * S[inv[b * V + u]]
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_conv_abs_scale_bounds_output():
    B, V, K, Ci, Co = 2, 60, 9, 8, 8
    m = (RNG.random((B, V)) < 0.3).astype(np.uint8)
    nbr = rand_nbr(V, K, RNG)
    coords, inv, rp, n = O.compact(m)
    S = RNG.standard_normal((n, Ci))
    W = RNG.standard_normal((K, Ci, Co))
    b = RNG.standard_normal(Co)
    y = O.sparse_conv(S, coords, B, V, nbr, W, b)
    s = O.sparse_conv_scale(S, coords, B, V, nbr, W, b)
    assert np.all(np.abs(y) <= s * (1 + 1e-12))
    # all-positive data: the scale is the output itself
    yp = O.sparse_conv(np.abs(S), coords, B, V, nbr, np.abs(W), np.abs(b))
    np.testing.assert_allclose(yp, s, rtol=1e-13)


# ----------------------------------------------------------------------------
# pooling
# ----------------------------------------------------------------------------


def test_segment_max_vs_reduceat_and_empty_segments():
    B, V, C = 40, 25, 7
    m = (RNG.random((B, V)) < 0.1).astype(np.uint8)
    m[3] = 0
    m[17] = 0
    coords, inv, rp, n = O.compact(m)
    S = RNG.standard_normal((n, C)).astype(np.float32)
    P = O.segment_max(S, rp, empty_value=-5.0)
    nonempty = np.flatnonzero(np.diff(rp) > 0)
    ref = np.maximum.reduceat(S, rp[nonempty], axis=0)
    assert np.array_equal(P[nonempty], ref)
    empty = np.flatnonzero(np.diff(rp) == 0)
    assert 3 in empty and 17 in empty
    assert np.all(P[empty] == -5.0)


def test_segment_max_ignores_nan_and_equals_dense_pool_after_relu():
    S = np.array([[np.nan, 1.0], [2.0, np.nan], [0.5, 0.25]], np.float32)
    P = O.segment_max(S, np.array([0, 3]))
    assert P.tolist() == [[2.0, 1.0]]
    # after ReLU, the per-body max over active rows equals a dense max over all
    # vertices of relu(y) (.) m, empty bodies included (inactive rows are 0)
    B, V, C = 6, 20, 4
    m = (RNG.random((B, V)) < 0.2).astype(np.uint8)
    m[0] = 0
    coords, inv, rp, n = O.compact(m)
    y = np.maximum(RNG.standard_normal((n, C)), 0)
    dense = O.densify(y, coords, B, V).reshape(B, V, C).max(axis=1)
    assert np.array_equal(O.segment_max(y, rp), dense)


# ----------------------------------------------------------------------------
# several masks stacked as a batch axis; per-element masks (Sec. 3.1)
# ----------------------------------------------------------------------------


def test_stacked_masks_equal_separate_runs():
    """Mask k of body b as body k * B + b: the stacked compaction and gather
    give, block by block, exactly what each mask gives on its own."""
    rng = np.random.default_rng(21)
    kappa, B, V, C = 3, 4, 30, 5
    masks = (rng.random((kappa, B, V)) < 0.3).astype(np.uint8)
    x = rng.standard_normal((B * V, C))
    st = O.stack_masks(masks)
    assert st.shape == (kappa * B, V)
    coords, inv, rp, n = O.compact(st)
    S = O.gather_stacked(x, coords, B, V)
    for k in range(kappa):
        ck, _, _, nk = O.compact(masks[k])
        lo, hi = rp[k * B], rp[(k + 1) * B]
        assert hi - lo == nk
        np.testing.assert_array_equal(coords[lo:hi, 0] - k * B, ck[:, 0])
        np.testing.assert_array_equal(coords[lo:hi, 1], ck[:, 1])
        np.testing.assert_array_equal(S[lo:hi], O.gather(x, ck, V))
    # brute force: every stacked row is the masked input of its body
    for i in range(n):
        bp, v = coords[i]
        assert masks[bp // B, bp % B, v] == 1
        np.testing.assert_array_equal(S[i], x[(bp % B) * V + v])


def test_combine_stacked_brute_force_and_invariants():
    rng = np.random.default_rng(22)
    kappa, R, C = 3, 4, 3
    Y = rng.standard_normal((kappa * R, C))
    for op in ("sum", "mean", "max"):
        got = O.combine_stacked(Y, kappa, op)
        for r in range(R):
            for c in range(C):
                vals = [float(Y[k * R + r, c]) for k in range(kappa)]
                exp = {"sum": sum(vals), "mean": sum(vals) / kappa, "max": max(vals)}[op]
                assert abs(got[r, c] - exp) < 1e-12
    Z = np.tile(Y[:R], (kappa, 1))       # kappa identical copies
    np.testing.assert_allclose(O.combine_stacked(Z, kappa, "sum"), kappa * Y[:R], rtol=1e-15)
    np.testing.assert_allclose(O.combine_stacked(Z, kappa, "mean"), Y[:R], rtol=1e-15)
    np.testing.assert_array_equal(O.combine_stacked(Z, kappa, "max"), Y[:R])
    np.testing.assert_array_equal(O.combine_stacked(Y, 1, "max"), Y)


def test_element_masks_brute_force_and_broadcast_case():
    rng = np.random.default_rng(23)
    B, V, C = 3, 7, 4
    me = (rng.random((B, V, C)) < 0.3).astype(np.uint8)
    x = rng.standard_normal((B * V, C))
    m = O.row_mask_from_elements(me)
    for b in range(B):
        for v in range(V):
            assert m[b, v] == (1 if any(me[b, v, c] for c in range(C)) else 0)
    coords, inv, rp, n = O.compact(m)
    S = O.gather_masked(x, me, coords, V)
    for i in range(n):
        b, v = coords[i]
        for c in range(C):
            assert S[i, c] == (x[b * V + v, c] if me[b, v, c] else 0.0)
    # a mask drawn per vertex and broadcast over channels is the vertex path
    mv = (rng.random((B, V)) < 0.4).astype(np.uint8)
    meb = np.repeat(mv[:, :, None], C, axis=2)
    np.testing.assert_array_equal(O.row_mask_from_elements(meb), mv)
    cv, _, _, _ = O.compact(mv)
    np.testing.assert_array_equal(O.gather_masked(x, meb, cv, V), O.gather(x, cv, V))


# ----------------------------------------------------------------------------
# mask scores (Eq. 3)
# ----------------------------------------------------------------------------


def test_mask_similarity_rank_one_closed_form():
    """Y_k = u_k w_k^T: Y_i^T Y_k = (u_i . u_k) w_i w_k^T, so the similarity is
    cos^2 of the row factors, whatever the channel factors."""
    rng = np.random.default_rng(31)
    K, N, C = 4, 50, 6
    U = rng.standard_normal((K, N))
    Wc = rng.standard_normal((K, C))
    Y = np.einsum("kn,kc->knc", U, Wc)
    sim = O.mask_similarity(Y)
    for i in range(K):
        for k in range(K):
            cos = U[i] @ U[k] / (np.linalg.norm(U[i]) * np.linalg.norm(U[k]))
            assert abs(sim[i, k] - cos * cos) < 1e-12


def test_mask_scores_orthogonal_identical_and_invariances():
    rng = np.random.default_rng(32)
    N, C = 40, 5
    # disjoint row supports: Y_i^T Y_k = 0, similarity 0, every score + 1
    Y = np.zeros((3, N, C))
    for k in range(3):
        Y[k, 10 * k:10 * k + 10] = rng.standard_normal((10, C))
    np.testing.assert_allclose(O.mask_similarity(Y), np.eye(3), atol=1e-15)
    np.testing.assert_allclose(O.alpha_update(np.zeros(3), Y), np.ones(3), atol=1e-15)
    # identical outputs: similarity 1, scores unchanged
    X = rng.standard_normal((N, C))
    np.testing.assert_allclose(O.alpha_update(np.array([0.5, -1.0, 2.0]), np.stack([X, X, X])),
                               [0.5, -1.0, 2.0], atol=1e-12)
    # scaling one output changes nothing; relabelling permutes; 0 <= sim <= 1
    R = rng.standard_normal((4, N, C))
    base = O.mask_similarity(R)
    R2 = R.copy()
    R2[2] *= -7.5
    np.testing.assert_allclose(O.mask_similarity(R2), base, rtol=1e-12)
    perm = [2, 0, 3, 1]
    np.testing.assert_allclose(O.mask_similarity(R[perm]), base[np.ix_(perm, perm)], rtol=1e-12)
    assert np.all(base <= 1 + 1e-12) and np.all(base >= 0)   # Cauchy-Schwarz


def test_mask_scores_zero_output_earns_no_credit():
    """Eq. 3 divides by the Frobenius norms of the two Gram matrices, which
    vanish for an all-zero output.  Reading: such a pair counts as similar
    (sim = 1), so the zero mask's score is unchanged, it adds nothing to the
    others' scores, and it ranks after every mask whose score grew."""
    rng = np.random.default_rng(34)
    N, C = 30, 4
    Y = rng.standard_normal((4, N, C))
    Y[1] = 0.0
    sim = O.mask_similarity(Y)
    assert np.all(np.isfinite(sim))
    np.testing.assert_array_equal(sim[1], np.ones(4))
    np.testing.assert_array_equal(sim[:, 1], np.ones(4))
    live = [0, 2, 3]
    np.testing.assert_allclose(sim[np.ix_(live, live)], O.mask_similarity(Y[live]),
                               rtol=1e-14)
    a0 = np.array([0.25, 0.25, 0.25, 0.25])
    a1 = O.alpha_update(a0, Y)
    assert a1[1] == a0[1]
    # the live masks' increments are those of the three-mask problem scaled by
    # (3 - 1) / (4 - 1): the zero mask contributes 1 - 1 = 0 to each sum
    inc3 = O.alpha_update(np.zeros(3), Y[live])
    np.testing.assert_allclose(a1[live] - 0.25, inc3 * 2.0 / 3.0, rtol=1e-13)
    assert O.top_kappa(a1, 4)[-1] == 1
    # every output zero: all pairs similar, nothing changes
    np.testing.assert_array_equal(O.alpha_update(a0, np.zeros((4, N, C))), a0)


def test_gram_frobenius_brute_force_and_top_kappa():
    rng = np.random.default_rng(33)
    K, N, C = 3, 4, 2
    Y = rng.standard_normal((K, N, C))
    F = O.gram_frobenius(Y)
    for i in range(K):
        for k in range(K):
            tot = 0.0
            for a in range(C):
                for b in range(C):
                    g = sum(float(Y[i, n, a]) * float(Y[k, n, b]) for n in range(N))
                    tot += g * g
            assert abs(F[i, k] - tot) < 1e-12 * max(1.0, tot)
    assert list(O.top_kappa(np.array([0.3, 0.9, 0.3, 0.1, 0.9]), 3)) == [1, 4, 0]
    np.testing.assert_array_equal(O.alpha_update(np.array([1.25]), Y[:1]), [1.25])  # K = 1
    assert list(O.top_kappa(np.array([2.0]), 1)) == [0]


# ----------------------------------------------------------------------------
# backward of the sparse linear and conv layers
# ----------------------------------------------------------------------------


def bwd_case(rng, B=3, V=11, K=4, Ci=5, Co=6, p=0.5):
    m = (rng.random((B, V)) < p).astype(np.uint8)
    m[0, 0] = 1
    coords, inv, rp, n = O.compact(m)
    S = rng.standard_normal((n, Ci))
    nbr = rand_nbr(V, K, rng)
    nbr[1, 2] = nbr[2, 2] = 4                # two rows sending to one neighbour by one slot
    W = rng.standard_normal((K, Ci, Co))
    bias = rng.standard_normal(Co)
    return m, coords, n, S, nbr, W, bias


def torch_sparse_conv(S, coords, B, V, nbr, W, bias, act):
    """The dense conv of x (.) m read at the active rows, written with torch
    ops (an index_select per slot) so that autograd differentiates it."""
    n = S.shape[0]
    flat = torch.as_tensor(coords[:, 0].astype(np.int64) * V + coords[:, 1])
    xd = torch.zeros((B * V, S.shape[1]), dtype=torch.float64).index_copy(0, flat, S)
    xd = xd.view(B, V, -1)
    y = torch.zeros((B, V, W.shape[2]), dtype=torch.float64)
    for j in range(W.shape[0]):
        idx = torch.as_tensor(np.maximum(nbr[:, j], 0).astype(np.int64))
        has = torch.as_tensor(nbr[:, j] >= 0, dtype=torch.float64).view(1, V, 1)
        y = y + has * (xd.index_select(1, idx) @ W[j])
    y = y + bias
    if act:
        y = torch.relu(y)
    return y.view(B * V, -1).index_select(0, flat)


@pytest.mark.parametrize("act", [False, True])
def test_conv_backward_matches_torch_autograd(act):
    """dS, dW, db against autograd of an independently written dense conv."""
    rng = np.random.default_rng(41 + act)
    m, coords, n, S, nbr, W, bias = bwd_case(rng)
    B, V = m.shape
    St = torch.tensor(S, requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    bt = torch.tensor(bias, requires_grad=True)
    Y = torch_sparse_conv(St, coords, B, V, nbr, Wt, bt, act)
    dY = rng.standard_normal(Y.shape)
    (Y * torch.as_tensor(dY)).sum().backward()
    dS, dW, db = O.sparse_conv_backward(S, coords, B, V, nbr, W, dY,
                                        Y.detach().numpy(), act)
    np.testing.assert_allclose(dS, St.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dW, Wt.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-12, atol=1e-12)
    if act:
        assert np.any(Y.detach().numpy() == 0)   # the mask cut something


@pytest.mark.parametrize("act", [False, True])
def test_linear_backward_matches_torch_autograd(act):
    rng = np.random.default_rng(43 + act)
    S = rng.standard_normal((9, 5))
    W = rng.standard_normal((5, 7))
    bias = rng.standard_normal(7)
    St, Wt, bt = (torch.tensor(a, requires_grad=True) for a in (S, W, bias))
    Y = torch.nn.functional.linear(St, Wt.T, bt)
    if act:
        Y = torch.relu(Y)
    dY = rng.standard_normal(Y.shape)
    (Y * torch.as_tensor(dY)).sum().backward()
    dS, dW, db = O.sparse_linear_backward(S, W, dY, Y.detach().numpy(), act)
    np.testing.assert_allclose(dS, St.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dW, Wt.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_conv_backward_finite_differences_and_adjoint():
    """Central differences of <dY, conv(S)> in a few entries of S and W, and
    the dot-product test <conv(S), G> = <S, dS(G)> (no bias, no activation)."""
    rng = np.random.default_rng(45)
    m, coords, n, S, nbr, W, bias = bwd_case(rng)
    B, V = m.shape
    dY = rng.standard_normal((n, W.shape[2]))
    dS, dW, db = O.sparse_conv_backward(S, coords, B, V, nbr, W, dY)

    def loss(S_, W_, b_):
        return float((O.sparse_conv(S_, coords, B, V, nbr, W_, b_) * dY).sum())

    h = 1e-6
    for (r, c) in [(0, 0), (n - 1, 3), (n // 2, 1)]:
        Sp, Sm = S.copy(), S.copy()
        Sp[r, c] += h
        Sm[r, c] -= h
        assert abs((loss(Sp, W, bias) - loss(Sm, W, bias)) / (2 * h) - dS[r, c]) < 1e-6
    for (j, c, o) in [(0, 0, 0), (2, 4, 5), (3, 1, 2)]:
        Wp, Wm = W.copy(), W.copy()
        Wp[j, c, o] += h
        Wm[j, c, o] -= h
        assert abs((loss(S, Wp, bias) - loss(S, Wm, bias)) / (2 * h) - dW[j, c, o]) < 1e-6
    bp = bias.copy()
    bp[2] += 1.0
    assert abs(loss(S, W, bp) - loss(S, W, bias) - db[2]) < 1e-9
    G = rng.standard_normal((n, W.shape[2]))
    dSG = O.sparse_conv_backward(S, coords, B, V, nbr, W, G)[0]
    lhs = float((O.sparse_conv(S, coords, B, V, nbr, W) * G).sum())
    assert abs(lhs - float((S * dSG).sum())) < 1e-10 * max(1.0, abs(lhs))


def test_conv_backward_brute_force_tiny():
    """Pure-Python loops over (row, slot) pairs."""
    rng = np.random.default_rng(46)
    m, coords, n, S, nbr, W, bias = bwd_case(rng, B=2, V=7, K=3, Ci=2, Co=3, p=0.6)
    B, V = m.shape
    Y = np.maximum(rng.standard_normal((n, 3)), 0.0)
    dY = rng.standard_normal((n, 3))
    dS, dW, db = O.sparse_conv_backward(S, coords, B, V, nbr, W, dY, Y, act=True)
    row = {(int(b), int(v)): i for i, (b, v) in enumerate(coords)}
    eS = [[0.0] * 2 for _ in range(n)]
    eW = [[[0.0] * 3 for _ in range(2)] for _ in range(3)]
    eb = [0.0] * 3
    for i, (b, v) in enumerate(coords.tolist()):
        for o in range(3):
            g = float(dY[i, o]) if Y[i, o] > 0 else 0.0
            eb[o] += g
            for j in range(3):
                u = int(nbr[v, j])
                if u < 0 or (b, u) not in row:
                    continue
                src = row[(b, u)]
                for c in range(2):
                    eS[src][c] += g * float(W[j, c, o])
                    eW[j][c][o] += float(S[src, c]) * g
    np.testing.assert_allclose(dS, eS, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dW, eW, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, eb, rtol=1e-12, atol=1e-12)


def test_conv_backward_special_cases_and_rows_at():
    """A single self slot is the linear layer's backward; an inactive
    neighbour receives nothing; the per-row evaluation agrees."""
    rng = np.random.default_rng(47)
    m, coords, n, S, nbr, W, bias = bwd_case(rng)
    B, V = m.shape
    dY = rng.standard_normal((n, W.shape[2]))
    self_nbr = np.arange(V, dtype=np.int32)[:, None]
    got = O.sparse_conv_backward(S, coords, B, V, self_nbr, W[:1], dY)
    want = O.sparse_linear_backward(S, W[0], dY)
    for a, b in zip(got, want):
        np.testing.assert_allclose(a, np.reshape(b, a.shape), rtol=1e-12, atol=1e-12)
    dS = O.sparse_conv_backward(S, coords, B, V, nbr, W, dY)[0]
    rows = np.array([0, n // 3, n - 1])
    np.testing.assert_allclose(O.conv_backward_input_at(coords, B, V, nbr, W, dY, rows),
                               dS[rows], rtol=1e-12, atol=1e-12)
    # a lone active vertex whose slots point elsewhere gets only its self term
    m1 = np.zeros((1, V), np.uint8)
    m1[0, 5] = 1
    c1 = O.compact(m1)[0]
    d1 = O.sparse_conv_backward(S[:1], c1, 1, V, nbr, W, dY[:1])
    np.testing.assert_allclose(d1[0], dY[:1] @ W[0].T, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed,p", [(48, 0.5), (49, 0.15), (50, 1.0)])
def test_conv_backward_weight_bias_matches_full_backward(seed, p):
    """The slot-by-slot weight and bias gradient from dZ equals the full
    backward's dW and db (no activation, so dZ = dY), and its scale form
    equals the full backward of the absolute values."""
    rng = np.random.default_rng(seed)
    m, coords, n, S, nbr, W, bias = bwd_case(rng, B=3, V=23, K=5, Ci=4, Co=6, p=p)
    B, V = m.shape
    dZ = rng.standard_normal((n, W.shape[2]))
    _, dW, db = O.sparse_conv_backward(S, coords, B, V, nbr, W, dZ)
    gW, gb = O.conv_backward_weight_bias(S, coords, B, V, nbr, dZ, W.shape[0])
    np.testing.assert_allclose(gW, dW, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(gb, db, rtol=1e-12, atol=1e-12)
    _, aW, ab = O.sparse_conv_backward(np.abs(S), coords, B, V, nbr, np.abs(W), np.abs(dZ))
    sW, sb = O.conv_backward_weight_bias(S, coords, B, V, nbr, dZ, W.shape[0], scale=True)
    np.testing.assert_allclose(sW, aW, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(sb, ab, rtol=1e-12, atol=1e-12)
    # brute force of one slot's gradient: rows whose slot-j neighbour is active
    row = {(int(b), int(v)): i for i, (b, v) in enumerate(coords)}
    j = 2
    e = np.zeros((S.shape[1], dZ.shape[1]))
    for i, (b, v) in enumerate(coords.tolist()):
        u = int(nbr[v, j])
        if u >= 0 and (b, u) in row:
            e += np.outer(S[row[(b, u)]], dZ[i])
    np.testing.assert_allclose(gW[j], e, rtol=1e-12, atol=1e-12)


# ----------------------------------------------------------------------------
# group normalization (Eqs. 7-9)
# ----------------------------------------------------------------------------


def gn_case(rng, B=5, V=40, C=12, p=0.4):
    m = (rng.random((B, V)) < p).astype(np.uint8)
    m[2] = 0                                # one body without rows
    m[3] = 0
    m[3, 7] = 1                             # one body with a single row
    coords, inv, rp, n = O.compact(m)
    x = rng.standard_normal((B * V, C)) * 3.0 + rng.standard_normal(C)
    return m, coords, rp, O.gather(x, coords, V), x


@pytest.mark.parametrize("G", [1, 3, 4, 12])
def test_group_norm_full_mask_is_torch_group_norm(G):
    """All rows active: each body's statistics cover all V rows, which is
    torch's group_norm on the body's [C, V] feature map."""
    rng = np.random.default_rng(G)
    B, V, C = 3, 30, 12
    m = np.ones((B, V), np.uint8)
    coords, inv, rp, n = O.compact(m)
    x = rng.standard_normal((B * V, C)) * 2 + 1
    S = O.gather(x, coords, V)
    got = O.group_norm(S, rp, G)
    xt = torch.from_numpy(x.reshape(B, V, C).transpose(0, 2, 1).copy())   # [B][C][V]
    ref = torch.nn.functional.group_norm(xt, G, eps=1e-5).numpy().transpose(0, 2, 1).reshape(-1, C)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_group_norm_one_group_is_torch_layer_norm_per_body():
    """G = 1 (the paper's layer-normalization case): per body, torch's
    layer_norm over all of its active rows and channels at once."""
    rng = np.random.default_rng(11)
    m, coords, rp, S, _ = gn_case(rng)
    got = O.group_norm(S, rp, 1)
    for b in range(len(rp) - 1):
        lo, hi = rp[b], rp[b + 1]
        if hi > lo:
            blk = torch.from_numpy(S[lo:hi])
            ref = torch.nn.functional.layer_norm(blk, blk.shape, eps=1e-5).numpy()
            np.testing.assert_allclose(got[lo:hi], ref, rtol=1e-12, atol=1e-12)


def test_group_norm_two_rows_closed_form():
    """Two rows, one channel per group: mu = (a + c) / 2, biased variance
    ((a - c) / 2)^2, so the outputs are +-d / sqrt(d^2 + eps), d = (a - c) / 2."""
    a = np.array([[1.5, -2.0, 7.0], [-0.5, 4.0, 7.0]])
    got = O.group_norm(a, np.array([0, 2]), 3, eps=0.25)
    d = (a[0] - a[1]) / 2
    exp = np.stack([d, -d]) / np.sqrt(d * d + 0.25)
    np.testing.assert_allclose(got, exp, rtol=1e-15, atol=0)
    assert np.all(got[:, 2] == 0)           # equal values: zero deviation


def test_group_norm_single_row_and_empty_bodies():
    rng = np.random.default_rng(12)
    m, coords, rp, S, _ = gn_case(rng, C=8)
    got = O.group_norm(S, rp, 8)            # one channel per group
    lo = rp[3]
    assert rp[4] - lo == 1
    assert np.all(got[lo] == 0)             # a lone value has zero deviation
    assert rp[3] == rp[2]                   # body 2 contributes no row


def test_group_norm_invariants():
    """Per (body, group): the output has mean 0 and mean square var/(var+eps);
    a constant added to a (body, group) block changes nothing; scaling the
    input by s and eps by s^2 changes nothing; bodies do not interact; and
    the statistics use the body's ACTIVE rows only (a dense normalization of
    x (.) m over all V rows differs)."""
    rng = np.random.default_rng(13)
    m, coords, rp, S, x = gn_case(rng, C=12)
    G, eps = 3, 1e-5
    out = O.group_norm(S, rp, G, eps)
    for b in range(len(rp) - 1):
        lo, hi = rp[b], rp[b + 1]
        if hi - lo < 2:
            continue
        for g in range(G):
            blk = out[lo:hi, 4 * g:4 * g + 4]
            v = S[lo:hi, 4 * g:4 * g + 4]
            var = v.var()
            assert abs(blk.mean()) < 1e-12
            assert abs((blk ** 2).mean() - var / (var + eps)) < 1e-12
    S2 = S.copy()
    S2[rp[1]:rp[2], 4:8] += 123.0
    np.testing.assert_allclose(O.group_norm(S2, rp, G, eps), out, atol=1e-9)
    np.testing.assert_allclose(O.group_norm(S * 7.0, rp, G, eps * 49.0), out, atol=1e-12)
    S3 = S.copy()
    S3[rp[0]:rp[1]] *= -5.0
    o3 = O.group_norm(S3, rp, G, eps)
    np.testing.assert_array_equal(o3[rp[1]:], out[rp[1]:])
    # dense group norm of x (.) m over all V rows of body 0 is a different thing
    V = m.shape[1]
    xm = (x * m.reshape(-1, 1))[:V]
    dense = torch.nn.functional.group_norm(torch.from_numpy(xm.T[None].copy()), G).numpy()[0].T
    assert not np.allclose(dense[m[0] != 0], out[rp[0]:rp[1]], atol=1e-3)


# ----------------------------------------------------------------------------
# bfloat16 round-to-nearest-even
# ----------------------------------------------------------------------------


def bf16_exact_rne(x: float) -> float:
    """Nearest bf16 by exact rational comparison of the two bracketing values."""
    if x == 0 or not np.isfinite(x):
        return x
    fx = Fraction(x)
    ax = abs(fx)
    e = 0
    while ax >= 2:
        ax /= 2
        e += 1
    while ax < 1:
        ax *= 2
        e -= 1
    e = max(e, -126)
    spacing = Fraction(2) ** (e - 7)
    lo = (abs(fx) // spacing) * spacing
    hi = lo + spacing
    dlo, dhi = abs(fx) - lo, hi - abs(fx)
    if dlo < dhi:
        r = lo
    elif dhi < dlo:
        r = hi
    else:
        r = lo if (lo / spacing) % 2 == 0 else hi
    maxf = (2 - Fraction(1, 128)) * Fraction(2) ** 127
    if r > maxf:
        return float(np.copysign(np.inf, x))
    return float(r) if x > 0 else -float(r)


def test_round_bf16_matches_torch_on_fp32_inputs():
    vals = np.concatenate([
        RNG.standard_normal(200000).astype(np.float32) * np.float32(7.0),
        (RNG.standard_normal(20000) * 1e-39).astype(np.float32),          # subnormals
        np.array([3.3895e38, 3.39e38, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.0 - 2 ** -8,
                  2 ** -133, 3 * 2 ** -134, 0.0, -0.0, np.inf, -np.inf], np.float32),
    ])
    ref = torch.from_numpy(vals).to(torch.bfloat16).to(torch.float64).numpy()
    got = O.round_bf16(vals.astype(np.float64))
    assert np.array_equal(got, ref)


def test_round_bf16_exact_rational_on_fp64_inputs():
    vals = list(RNG.standard_normal(3000) * 10.0 ** RNG.integers(-40, 38, 3000))
    # exact ties of the bf16 grid in fp64, and near-ties one fp64 ulp away
    for k in range(200):
        base = float(np.float32(RNG.standard_normal()))
        t = float(torch.tensor(base).to(torch.bfloat16).double())
        spacing = 2.0 ** (np.frexp(abs(t))[1] - 1 - 7) if t != 0 else 2.0 ** -133
        tie = t + spacing / 2
        vals += [tie, np.nextafter(tie, np.inf), np.nextafter(tie, -np.inf)]
    got = O.round_bf16(np.array(vals))
    ref = np.array([bf16_exact_rne(v) for v in vals])
    assert np.array_equal(got, ref)
    assert np.isnan(O.round_bf16(np.array([np.nan]))[0])


# ----------------------------------------------------------------------------
# stacks and the paper's density reading
# ----------------------------------------------------------------------------


def test_stack_matches_chained_brute_force_bf16():
    B, V, K = 2, 14, 4
    rng = np.random.default_rng(77)
    m = (rng.random((B, V)) < 0.6).astype(np.uint8)
    nbr = rand_nbr(V, K, rng)
    x = torch.from_numpy(rng.standard_normal((B * V, 3))).to(torch.bfloat16).double().numpy()
    W1 = rng.standard_normal((K, 3, 4))
    W2 = rng.standard_normal((4, 2))
    layers = [("conv", W1, None, True), ("linear", W2, None, True)]
    res = O.run_stack(x, m, nbr, layers, "bf16", pool=True)
    # chained brute force with torch's conversion between layers
    h = brute_conv(x, m, nbr, W1, None, B, V, True)
    h = torch.from_numpy(h).to(torch.bfloat16).double().numpy()
    h2 = np.maximum(h @ W2, 0)
    h2 = torch.from_numpy(h2).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(res["outs"][1], h2)
    rp = res["row_ptr"]
    for b in range(B):
        seg = h2[rp[b]:rp[b + 1]]
        ref = seg.max(0) if len(seg) else np.zeros(2)
        np.testing.assert_array_equal(res["pool"][b], ref)


def f32_exact_rne(x: float) -> float:
    """Nearest binary32 value (24 significant bits, exponents from -126,
    largest finite (2 - 2^-23) 2^127), ties to even, by exact rational
    comparison of the two bracketing values."""
    if x == 0 or not np.isfinite(x):
        return x
    fx = abs(Fraction(x))
    e = 0
    ax = fx
    while ax >= 2:
        ax /= 2
        e += 1
    while ax < 1:
        ax *= 2
        e -= 1
    spacing = Fraction(2) ** (max(e, -126) - 23)
    lo = (fx // spacing) * spacing
    hi = lo + spacing
    if fx - lo < hi - fx:
        r = lo
    elif hi - fx < fx - lo:
        r = hi
    else:
        r = lo if (lo / spacing) % 2 == 0 else hi
    if r > (2 - Fraction(1, 2 ** 23)) * Fraction(2) ** 127:
        return float(np.copysign(np.inf, x))
    return float(r) if x > 0 else -float(r)


def test_round_f32_exact_rational_and_store():
    vals = list(RNG.standard_normal(3000) * 10.0 ** RNG.integers(-45, 38, 3000))
    for k in range(200):
        t = float(np.float32(RNG.standard_normal() * 10.0 ** RNG.integers(-30, 30)))
        spacing = 2.0 ** (max(np.frexp(abs(t))[1] - 1, -126) - 23)
        tie = t + spacing / 2
        vals += [tie, np.nextafter(tie, np.inf), np.nextafter(tie, -np.inf)]
    vals += [3.4028235677973366e38, 3.4028235e38 * 1.0000001, 2.0 ** -149, 2.0 ** -150,
             1.5 * 2.0 ** -149, -0.0]
    got = O.round_f32(np.array(vals))
    ref = np.array([f32_exact_rne(v) for v in vals])
    assert np.array_equal(got, ref)
    np.testing.assert_array_equal(O.store(np.array(vals), "f32"), ref)
    np.testing.assert_array_equal(O.store(np.array(vals[:50]), "bf16"),
                                  [bf16_exact_rne(v) for v in vals[:50]])
    with pytest.raises(ValueError):
        O.store(np.zeros(2), "f16")


def test_stack_matches_chained_brute_force_f32():
    """An fp32 stack: every layer's output is rounded to binary32 (torch's
    conversion here) before it feeds the next layer."""
    B, V, K = 2, 16, 5
    rng = np.random.default_rng(78)
    m = (rng.random((B, V)) < 0.55).astype(np.uint8)
    nbr = rand_nbr(V, K, rng)
    x = rng.standard_normal((B * V, 3)).astype(np.float32).astype(np.float64)
    W1 = rng.standard_normal((K, 3, 4))
    b1 = rng.standard_normal(4)
    W2 = rng.standard_normal((K, 4, 4))
    W3 = rng.standard_normal((4, 2))
    layers = [("conv", W1, b1, True), ("conv", W2, None, False), ("linear", W3, None, True)]
    res = O.run_stack(x, m, nbr, layers, "f32", pool=True)
    to32 = lambda a: torch.from_numpy(a).to(torch.float32).double().numpy()   # noqa: E731
    h1 = to32(brute_conv(x, m, nbr, W1, b1, B, V, True))
    # the second conv reads the first layer's rows scattered back (x (.) m)
    coords = res["coords"]
    d1 = np.zeros((B * V, 4))
    d1[coords[:, 0] * V + coords[:, 1]] = h1
    h2 = to32(brute_conv(d1, m, nbr, W2, None, B, V, False))
    h3 = to32(np.maximum(h2 @ W3, 0))
    for got, want in zip(res["outs"], (h1, h2, h3)):
        np.testing.assert_array_equal(got, want)
    rp = res["row_ptr"]
    for b in range(B):
        seg = h3[rp[b]:rp[b + 1]]
        np.testing.assert_array_equal(res["pool"][b], seg.max(0) if len(seg) else np.zeros(2))
    # the rounding matters: the same stack in fp64 storage differs somewhere
    assert not np.array_equal(to32(h2), brute_conv(d1, m, nbr, W2, None, B, V, False))


def test_density_reading_matches_table4(request):
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "table4_vertex_counts.txt")
    kv = {}
    for line in open(path):
        if line.strip() and not line.startswith("#"):
            k, v = line.split()
            kv[k] = float(v)
    density = 1.0 - kv["sparsity_ratio"]
    expected = kv["vertices_dense"] * density
    assert abs(expected - kv["vertices_processed_one_mask"]) < 1.0
    B = 4000
    m = (np.random.default_rng(3).random((B, int(kv["vertices_dense"]))) < density)
    _, _, rp, n = O.compact(m.astype(np.uint8))
    sigma = np.sqrt(kv["vertices_dense"] * density * (1 - density) / B)
    assert abs(n / B - expected) < 4 * sigma


def test_conv_at_and_linear_at_agree_with_full_layers():
    B, V, K, Ci, Co = 3, 70, 9, 8, 5
    rng = np.random.default_rng(13)
    m = (rng.random((B, V)) < 0.3).astype(np.uint8)
    nbr = rand_nbr(V, K, rng)
    coords, inv, rp, n = O.compact(m)
    S = rng.standard_normal((n, Ci))
    W = rng.standard_normal((K, Ci, Co))
    b = rng.standard_normal(Co)
    rows = rng.choice(n, size=min(n, 25), replace=False)
    for act in (False, True):
        full = O.sparse_conv(S, coords, B, V, nbr, W, b, act)
        np.testing.assert_allclose(O.conv_at(S, coords, B, V, nbr, W, rows, b, act), full[rows],
                                   rtol=1e-12, atol=1e-12)
        fl = O.sparse_linear(S, coords, B, V, W[0], b, act)
        np.testing.assert_allclose(O.linear_at(S, W[0], rows, b, act), fl[rows],
                                   rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(O.conv_at(S, coords, B, V, nbr, W, rows, b, scale=True),
                               O.sparse_conv_scale(S, coords, B, V, nbr, W, b)[rows], rtol=1e-12)
