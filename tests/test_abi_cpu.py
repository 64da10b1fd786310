"""The C ABI without a GPU: the library loads, exports what shc.h declares, and
rejects bad arguments on the host before any HIP call.

Only validation failures are exercised here (no call below reaches a kernel
launch), so no device is touched.  Fake "device pointers" are plain integers
with the alignment each case needs; validation never dereferences them.
"""
import ctypes
import os
import subprocess

import pytest

from paper_2608_09388_amd import binding as shc

A = 0x10000          # a 16-byte aligned fake address
MIS = 0x10004        # a misaligned one


@pytest.fixture(scope="module")
def lib():
    return shc.load()


def test_exports_every_declared_symbol(lib):
    declared = shc.header_symbols()
    assert len(declared) >= 9
    out = subprocess.run(["nm", "-D", "--defined-only", shc.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    for name in declared:
        assert name in exported, name
        assert getattr(lib, name) is not None


def test_status_strings(lib):
    for code, name in shc.STATUS.items():
        assert lib.shc_status_string(code).decode() == name
    assert lib.shc_status_string(-99).decode() == "SHC_ERR_UNKNOWN"


def test_workspace_query(lib):
    assert lib.shc_compact_mask_workspace(0, 5) == 0
    ws = lib.shc_compact_mask_workspace(128, 10475)
    assert ws > 0 and ws % 256 == 0
    assert lib.shc_compact_mask_workspace(1, 1) >= 4


def err(lib):
    return lib.shc_last_error().decode()


def test_compact_mask_validation(lib):
    ws = lib.shc_compact_mask_workspace(4, 655)
    ok = dict(mask=A, B=4, V=655, coords=A, inv=A, row_ptr=A, n_dev=A, n_host=None, cap=2620,
              ws=A, ws_bytes=ws)

    def call(**kw):
        a = dict(ok, **kw)
        return lib.shc_compact_mask(a["mask"], a["B"], a["V"], a["coords"], a["inv"], a["row_ptr"],
                                    a["n_dev"], a["n_host"], a["cap"], a["ws"], a["ws_bytes"], None)

    assert call(B=0) == -1 and "B = 0" in err(lib)
    assert call(V=-3) == -1
    assert call(B=1 << 16, V=1 << 16) == -4
    assert call(mask=None) == -1 and "mask" in err(lib)
    assert call(inv=MIS) == -3 and "inv" in err(lib)
    assert call(row_ptr=None) == -1
    assert call(n_dev=MIS) == -3
    assert call(ws=None) == -1
    assert call(cap=-1) == -1
    assert call(coords=None) == -1            # cap > 0 needs coords
    assert call(ws_bytes=ws - 1) == -2 and "workspace" in err(lib)


def test_compact_mask_noalloc_validation(lib):
    """The allocation-free compaction checks its arguments before it looks up
    its scratch array, so none of these touches a device."""
    ok = dict(mask=A, B=4, V=655, coords=A, inv=A, row_ptr=A, n_dev=A, n_host=None, cap=2620)

    def call(**kw):
        a = dict(ok, **kw)
        return lib.shc_compact_mask_noalloc(a["mask"], a["B"], a["V"], a["coords"], a["inv"],
                                            a["row_ptr"], a["n_dev"], a["n_host"], a["cap"], None)

    assert call(B=0) == -1 and "B = 0" in err(lib)
    assert call(B=1 << 16, V=1 << 16) == -4
    assert call(mask=None) == -1 and "mask" in err(lib)
    assert call(inv=MIS) == -3 and "inv" in err(lib)
    assert call(row_ptr=None) == -1
    assert call(n_dev=MIS) == -3
    assert call(cap=-1) == -1
    assert call(coords=None) == -1
    # the largest mask the library takes needs 4 KB of the 64 KB scratch
    assert lib.shc_compact_mask_workspace(1 << 15, (1 << 16) - 1) <= 4096


def test_compact_mask_start_wait_validation(lib):
    ws = lib.shc_compact_mask_workspace(4, 655)

    def start(n_host=None, **kw):
        a = dict(dict(mask=A, B=4, V=655, coords=A, inv=A, row_ptr=A, n_dev=A, cap=2620, ws=A,
                      ws_bytes=ws), **kw)
        return lib.shc_compact_mask_start(a["mask"], a["B"], a["V"], a["coords"], a["inv"],
                                          a["row_ptr"], a["n_dev"], n_host, a["cap"], a["ws"],
                                          a["ws_bytes"], None)

    assert start() == -1 and "n_active_host" in err(lib)   # the host count is required
    assert lib.shc_compact_mask_wait(None, 10, None) == -1 and "n_active_host" in err(lib)


def test_clear_inactive_rows_validation(lib):
    def call(inv=A, B=4, V=655, C=16, dtype=0, D=A):
        return lib.shc_clear_inactive_rows(inv, B, V, C, dtype, D, None)

    assert call(inv=None) == -1 and "inv" in err(lib)
    assert call(D=MIS) == -3 and "D" in err(lib)
    assert call(C=8) == -4
    assert call(dtype=5) < 0
    assert call(B=0) == -1


def test_group_norm_validation(lib):
    def call(S=A, rp=A, n=100, B=4, C=128, G=32, eps=1e-5, dt=1, out=A):
        return lib.shc_segment_group_norm(S, rp, n, B, C, G, eps, dt, out, None)

    assert call(B=0) == -1
    assert call(n=-1) == -1
    assert call(C=8) == -4
    assert call(dt=9) < 0
    assert call(G=0) == -1 and "G = 0" in err(lib)
    assert call(G=3) == -1 and "divide" in err(lib)
    assert call(eps=0.0) == -1 and "eps" in err(lib)
    assert call(eps=float("nan")) == -1
    assert call(n=0, S=None, out=None) == 0        # no-op
    assert call(S=None) == -1
    assert call(rp=MIS) == -3
    assert call(out=MIS) == -3


def test_multi_mask_validation(lib):
    def stacked(x=A, c=A, n=10, B=4, kappa=3, V=655, C=128, dt=1, S=A):
        return lib.shc_gather_rows_stacked(x, c, n, B, kappa, V, C, dt, S, None)

    assert stacked(kappa=0) == -1 and "kappa" in err(lib)
    assert stacked(B=0) == -1
    assert stacked(kappa=1 << 20, B=1 << 12) == -4
    assert stacked(C=8) == -4
    assert stacked(n=0, x=None, c=None, S=None) == 0
    assert stacked(x=None) == -1
    assert stacked(S=MIS) == -3

    def combine(Y=A, kappa=3, rows=100, C=128, dt=1, op=1, out=A):
        return lib.shc_combine_stacked(Y, kappa, rows, C, dt, op, out, None)

    assert combine(kappa=0) == -1
    assert combine(op=3) == -4 and "combination" in err(lib)
    assert combine(rows=-1) == -1
    assert combine(rows=0, Y=None, out=None) == 0
    assert combine(Y=MIS) == -3

    assert lib.shc_row_mask_from_elements(None, 4, 655, 128, A, None) == -1
    assert lib.shc_row_mask_from_elements(A, 4, 655, 24, A, None) == -4
    assert lib.shc_row_mask_from_elements(A, 0, 655, 128, A, None) == -1

    def masked(x=A, me=A, c=A, n=10, B=4, V=655, C=128, dt=1, S=A):
        return lib.shc_gather_rows_masked(x, me, c, n, B, V, C, dt, S, None)

    assert masked(me=None) == -1 and "me" in err(lib)
    assert masked(me=MIS) == -3
    assert masked(n=0, x=None, me=None, c=None, S=None) == 0


def test_mask_scores_validation(lib):
    assert lib.shc_mask_scores_workspace(10, 1000, 128) > 0
    assert lib.shc_mask_scores_workspace(65, 1000, 128) == 0
    assert lib.shc_mask_scores_workspace(10, 1000, 96) == 0
    assert lib.shc_mask_scores_workspace(0, 1000, 128) == 0
    need = lib.shc_mask_scores_workspace(4, 100, 128)

    def call(O=A, K=4, N=100, C=128, dt=1, ain=None, aout=A, sim=None, kappa=0, top=None,
             ws=A, nbytes=need):
        return lib.shc_mask_scores(O, K, N, C, dt, ain, aout, sim, kappa, top, ws, nbytes, None)

    assert call(K=0) == -4 and call(K=65) == -4
    assert call(N=0) == -1
    assert call(dt=0) == -4 and "bf16" in err(lib)
    assert call(C=96) == -4
    assert call(kappa=5) == -1
    assert call(kappa=2) == -1 and "top" in err(lib)
    assert call(O=None) == -1
    assert call(aout=None) == -1
    assert call(sim=MIS) == -3
    assert call(nbytes=need - 1) == -2 and "workspace" in err(lib)


def test_backward_validation(lib):
    """The transposed lists, the transposed table and both layer backward
    calls reject bad arguments before any launch."""
    assert lib.shc_transpose_neighbors_workspace(100, 9) > 0
    assert lib.shc_transpose_neighbors_workspace(100, 33) == 0
    kt = ctypes.c_int32(0)
    tn = lib.shc_transpose_neighbors
    need_t = lib.shc_transpose_neighbors_workspace(100, 9)
    assert tn(A, 0, 9, A, A, ctypes.addressof(kt), A, need_t, None) == -1
    assert tn(A, 100, 33, A, A, ctypes.addressof(kt), A, need_t, None) == -4
    assert tn(A, 100, 9, A, A, None, A, need_t, None) == -1
    assert tn(MIS, 100, 9, A, A, ctypes.addressof(kt), A, need_t, None) == -3
    assert tn(A, 100, 9, A, A, ctypes.addressof(kt), A, need_t - 1, None) == -2
    tt = lib.shc_build_transposed_table
    assert tt(A, A, 10, 4, 100, A, 0, A, A, None) == -1
    assert tt(A, A, 10, 4, 100, A, 65, A, A, None) == -1
    assert tt(A, A, 10, 4, 100, A, 20, A, MIS, None) == -3
    assert tt(A, A, 10, 0, 100, A, 20, A, A, None) == -1

    assert lib.shc_sparse_linear_backward_workspace(1000, 128, 128, 1) > 0
    assert lib.shc_sparse_linear_backward_workspace(1000, 128, 128, 0) > 0     # fp32
    assert lib.shc_sparse_linear_backward_workspace(1000, 128, 128, 7) == 0
    need = lib.shc_sparse_linear_backward_workspace(1000, 128, 128, 1)

    def lin(S=A, W=A, Y=A, dY=A, n=1000, Cin=128, Cout=128, dt=1, act=1, dS=A, dW=A, db=A,
            ws=A, nbytes=need):
        return lib.shc_sparse_linear_backward(S, W, Y, dY, n, Cin, Cout, dt, act, dS, dW, db, ws,
                                              nbytes, None)

    assert lin(dt=7) == -4 and "dtype" in err(lib)
    assert lin(Cin=24) == -4
    assert lin(Cout=512) == -4
    assert lin(act=7) == -4
    assert lin(n=-1) == -1
    assert lin(Y=None) == -1                       # the ReLU needs the stored output
    assert lin(dY=None) == -1
    assert lin(S=None) == -1                       # dW needs S
    assert lin(W=None) == -1
    assert lin(dS=MIS) == -3
    assert lin(nbytes=need - 1) == -2 and "workspace" in err(lib)

    needc = lib.shc_sparse_neighbor_conv_backward_workspace(1000, 9, 128, 128, 1)
    assert needc > need
    assert lib.shc_sparse_neighbor_conv_backward_workspace(1000, 33, 128, 128, 1) == 0

    def conv(S=A, table=A, pairs=None, pp=None, table_t=A, rs=A, so=A, Kt=56, W=A, Y=A, dY=A,
             n=1000, K=9, Cin=128, Cout=128, dt=1, act=1, dS=A, dW=A, db=A, ws=A, nbytes=needc):
        return lib.shc_sparse_neighbor_conv_backward(S, table, pairs, pp, table_t, rs, so, Kt, W,
                                                     Y, dY, n, K, Cin, Cout, dt, act, dS, dW, db,
                                                     ws, nbytes, None)

    assert conv(K=0) == -1 and conv(K=33) == -4
    assert conv(dt=7) == -4
    # fp32 weight fragments of 9 slots x 256 outputs do not fit in LDS: refused up front
    need_big = lib.shc_sparse_neighbor_conv_backward_workspace(1000, 9, 64, 256, 0)
    assert conv(dt=0, Cin=64, Cout=256, nbytes=need_big) == -4 and "fit" in err(lib)
    assert conv(table=None) == -1                  # dW needs the neighbour-row table
    assert conv(table_t=None) == -1                # dS needs the transposed table
    assert conv(Kt=0) == -1 and conv(Kt=65) == -1
    assert conv(rs=MIS) == -3
    assert conv(nbytes=needc - 1) == -2
    assert conv(pairs=A) == -1 and "together" in err(lib)   # pairs without their offsets
    assert conv(pairs=MIS, pp=A) == -3
    sp = lib.shc_build_slot_pairs
    need_p = lib.shc_build_slot_pairs_workspace(1000, 9)
    assert need_p > 0 and lib.shc_build_slot_pairs_workspace(1000, 33) == 0
    assert sp(A, 1000, 0, A, A, A, need_p, None) == -1
    assert sp(A, 1000, 33, A, A, A, need_p, None) == -4
    assert sp(None, 1000, 9, A, A, A, need_p, None) == -1
    assert sp(A, 1000, 9, A, A, A, need_p - 1, None) == -2


def test_gather_scatter_pool_validation(lib):
    g = lib.shc_gather_rows
    assert g(A, A, 10, 4, 655, 24, 0, A, None) == -4
    assert g(A, A, 10, 4, 655, 16, 7, A, None) == -4
    assert g(A, A, -1, 4, 655, 16, 0, A, None) == -1
    assert g(A, A, 1 << 31, 4, 655, 16, 0, A, None) == -1
    assert g(None, A, 10, 4, 655, 16, 0, A, None) == -1
    assert g(A, MIS, 10, 4, 655, 16, 1, A, None) == -3
    assert g(A, A, 10, 4, 655, 0, 1, A, None) == -1
    assert g(A, A, 10, 4, 655, 4112, 1, A, None) == -4
    s = lib.shc_scatter
    assert s(A, A, A, 10, 4, 655, 16, 0, 2, A, None) == -1
    assert s(A, None, A, 10, 4, 655, 16, 0, 1, A, None) == -1       # zero-fill needs inv
    assert s(A, A, None, 10, 4, 655, 16, 0, 0, A, None) == -1       # active-only needs coords
    assert s(A, A, A, 10, 4, 655, 16, 0, 1, MIS, None) == -3
    u = lib.shc_scatter_update
    A2 = 0x20000         # a second aligned fake address (prev_coords != coords)
    assert u(A, A, A, -1, A2, 0, 4, 655, 16, 0, A, None) == -1
    assert u(A, A, A, 0, A2, -1, 4, 655, 16, 0, A, None) == -1
    assert u(A, A, A, 10, A2, 0, 4, 655, 16, 7, A, None) == -4
    assert u(A, A, A, 10, A2, 0, 4, 655, 24, 0, A, None) == -4
    assert u(A, A, A, 10, A2, 0, 0, 655, 16, 0, A, None) == -1
    assert u(None, None, None, 0, None, 0, 4, 655, 16, 0, None, None) == 0   # nothing to do
    assert u(A, A, A, 10, A2, 0, 4, 655, 16, 0, None, None) == -1 and "D" in err(lib)
    assert u(A, None, A, 10, A2, 0, 4, 655, 16, 0, A, None) == -1 and "inv" in err(lib)
    assert u(None, A, A, 10, A2, 0, 4, 655, 16, 0, A, None) == -1 and "S" in err(lib)
    assert u(A, A, None, 10, A2, 0, 4, 655, 16, 0, A, None) == -1 and "coords" in err(lib)
    assert u(None, A, None, 0, None, 10, 4, 655, 16, 0, A, None) == -1
    assert "prev_coords" in err(lib)
    assert u(A, A, A, 10, A, 10, 4, 655, 16, 0, A, None) == -1 and "same" in err(lib)
    assert u(A, A, A, 10, A2, 0, 4, 655, 16, 0, MIS, None) == -3
    assert u(A, A, A, 10, MIS, 10, 4, 655, 16, 0, A, None) == -3
    assert u(A, A, A, 1 << 31, A2, 0, 4, 655, 16, 0, A, None) == -1
    p = lib.shc_segment_maxpool
    assert p(A, A, 10, 0, 16, 0, 0.0, A, None) == -1
    assert p(A, None, 10, 4, 16, 0, 0.0, A, None) == -1
    assert p(MIS, A, 10, 4, 16, 0, 0.0, A, None) == -3
    assert p(A, A, 10, 4, 20, 0, 0.0, A, None) == -4


def test_layer_validation(lib):
    L = lib.shc_sparse_linear
    assert L(A, 10, A, None, 16, 24, 0, 1, A, None) == -4
    assert L(A, 10, A, None, 16, 16, 0, 5, A, None) == -4
    assert L(None, 10, A, None, 16, 16, 0, 1, A, None) == -1
    assert L(A, 10, A, MIS, 16, 16, 0, 1, A, None) == -3           # bias alignment
    assert L(A, 10, None, None, 16, 16, 1, 0, A, None) == -1
    C = lib.shc_sparse_neighbor_conv

    def conv(**kw):
        a = dict(S=A, coords=A, inv=A, n=10, B=4, V=655, nbr=A, K=9, W=A, bias=None, Cin=16,
                 Cout=64, dt=0, act=1, out=A)
        a.update(kw)
        return C(a["S"], a["coords"], a["inv"], a["n"], a["B"], a["V"], a["nbr"], a["K"], a["W"],
                 a["bias"], a["Cin"], a["Cout"], a["dt"], a["act"], a["out"], None)

    assert conv(K=0) == -1
    assert conv(K=33) == -4 and "K = 33" in err(lib)
    assert conv(nbr=None) == -1
    assert conv(inv=MIS) == -3
    assert conv(Cout=8) == -4
    assert conv(B=0) == -1
    assert conv(dt=2) == -4
    assert conv(out=None) == -1


def test_gather_sparse_linear_validation(lib):
    G = lib.shc_gather_sparse_linear

    def call(**kw):
        a = dict(x=A, coords=A, n=10, B=4, V=655, W=A, bias=None, Cin=128, Cout=128, dt=1, act=1,
                 out=A)
        a.update(kw)
        return G(a["x"], a["coords"], a["n"], a["B"], a["V"], a["W"], a["bias"], a["Cin"],
                 a["Cout"], a["dt"], a["act"], a["out"], None)

    assert call(coords=None) == -1 and "coords" in err(lib)
    assert call(x=MIS) == -3
    assert call(B=0) == -1
    assert call(Cin=40) == -4
    assert call(act=9) == -4
    assert call(n=-2) == -1
    assert call(n=0, x=None, coords=None, W=None, out=None) == 0


def test_neighbor_table_validation(lib):
    T = lib.shc_build_neighbor_table

    def table(**kw):
        a = dict(coords=A, inv=A, n=10, B=4, V=655, nbr=A, K=9, table=A)
        a.update(kw)
        return T(a["coords"], a["inv"], a["n"], a["B"], a["V"], a["nbr"], a["K"], a["table"], None)

    assert table(K=0) == -1
    assert table(K=33) == -4
    assert table(V=0) == -1
    assert table(n=-1) == -1
    assert table(coords=None) == -1 and "coords" in err(lib)
    assert table(table=None) == -1 and "table" in err(lib)
    assert table(nbr=MIS) == -3
    assert table(n=0, coords=None, table=None) == 0     # N' = 0 is a no-op
    C = lib.shc_sparse_neighbor_conv_table

    def conv(**kw):
        a = dict(S=A, table=A, n=10, K=9, W=A, bias=None, Cin=16, Cout=64, dt=1, act=1, out=A)
        a.update(kw)
        return C(a["S"], a["table"], a["n"], a["K"], a["W"], a["bias"], a["Cin"], a["Cout"],
                 a["dt"], a["act"], a["out"], None)

    assert conv(table=None) == -1 and "table" in err(lib)
    assert conv(table=MIS) == -3
    assert conv(K=40) == -4
    assert conv(Cin=20) == -4
    assert conv(act=3) == -4
    assert conv(bias=MIS) == -3
    assert conv(n=0, S=None, table=None, out=None) == 0


def test_conv_split_validation(lib):
    """shc_conv_split_workspace_bytes's closed form and the split conv's
    argument checks, without a device."""
    Q = lib.shc_conv_split_workspace_bytes
    bf = shc.SHC_BF16
    assert Q(1000, 9, 128, 128, bf) == 8 * 1000 * 128 * 4
    assert Q(1000, 9, 256, 64, bf) == 8 * 1000 * 64 * 4
    assert Q(1000, 1, 64, 64, bf) == 16          # no pairs: the minimum
    assert Q(0, 9, 128, 128, bf) == 16
    assert Q(-1, 9, 128, 128, bf) == 0
    assert Q(1000, 9, 128, 128, shc.SHC_F32) == 0
    assert Q(1000, 9, 96, 128, bf) == 0          # channels outside {64, 128, 256}
    assert Q(1000, 9, 128, 512, bf) == 0
    assert Q(1000, 0, 128, 128, bf) == 0
    assert Q(1000, 33, 128, 128, bf) == 0
    n_max = (0x7FFF0000 // (8 * 256 * 4))         # the workspace stays below 2^31 bytes
    assert Q(n_max, 9, 256, 256, bf) > 0 and Q(n_max + 1, 9, 256, 256, bf) == 0
    C = lib.shc_sparse_neighbor_conv_split

    def conv(**kw):
        a = dict(S=A, table=A, n=10, K=9, W=A, bias=None, Cin=128, Cout=128, dt=bf, act=1,
                 out=A, ws=A, nb=8 * 10 * 128 * 4)
        a.update(kw)
        return C(a["S"], a["table"], a["n"], a["K"], a["W"], a["bias"], a["Cin"], a["Cout"],
                 a["dt"], a["act"], a["out"], a["ws"], a["nb"], None)

    assert conv(table=None) == -1 and "table" in err(lib)
    assert conv(S=MIS) == -3
    assert conv(ws=None) == -1 and "workspace" in err(lib)
    assert conv(ws=MIS) == -3
    assert conv(nb=8 * 10 * 128 * 4 - 1) == -2 and "workspace_bytes" in err(lib)
    assert conv(dt=shc.SHC_F32) == -4 and "bf16" in err(lib)
    assert conv(Cin=96) == -4
    assert conv(Cout=512) == -4
    assert conv(K=0) == -1
    assert conv(K=33) == -4
    assert conv(act=3) == -4
    assert conv(n=-1) == -1
    assert conv(bias=MIS) == -3
    assert conv(n=0, S=None, table=None, out=None, ws=None, nb=0) == 0   # N' = 0 is a no-op


def test_conv_plan_validation(lib):
    Q = lib.shc_conv_plan_bytes
    bf = shc.SHC_BF16
    assert Q(0, 9, 128, 128, bf) == 0
    assert Q(-1, 9, 128, 128, bf) == 0
    assert Q(1 << 31, 9, 128, 128, bf) == 0
    assert Q(100, 0, 128, 128, bf) == 0
    assert Q(100, 33, 128, 128, bf) == 0
    assert Q(100, 9, 20, 128, bf) == 0
    assert Q(100, 9, 128, 0, bf) == 0
    assert Q(100, 9, 128, 128, 7) == 0
    P = lib.shc_build_conv_plan

    def plan(**kw):
        a = dict(table=A, n=10, K=9, Cin=128, Cout=128, dt=bf, plan=A, nb=1 << 20)
        a.update(kw)
        return P(a["table"], a["n"], a["K"], a["Cin"], a["Cout"], a["dt"], a["plan"], a["nb"],
                 None)

    assert plan(table=None) == -1 and "table" in err(lib)
    assert plan(table=MIS) == -3
    assert plan(plan=None) == -1 and "plan" in err(lib)
    assert plan(plan=MIS) == -3
    assert plan(K=0) == -1
    assert plan(K=40) == -4
    assert plan(Cout=24) == -4
    assert plan(dt=5) == -4
    assert plan(n=-2) == -1
    assert plan(n=0, table=None, plan=None) == 0     # N' = 0 is a no-op
    C = lib.shc_sparse_neighbor_conv_planned

    def conv(**kw):
        a = dict(S=A, plan=A, nb=1 << 20, n=10, K=9, W=A, bias=None, Cin=128, Cout=128, dt=bf,
                 act=1, out=A)
        a.update(kw)
        return C(a["S"], a["plan"], a["nb"], a["n"], a["K"], a["W"], a["bias"], a["Cin"],
                 a["Cout"], a["dt"], a["act"], a["out"], None)

    assert conv(plan=None) == -1 and "plan" in err(lib)
    assert conv(plan=MIS) == -3
    assert conv(S=None) == -1 and "S" in err(lib)
    assert conv(W=MIS) == -3
    assert conv(out=None) == -1
    assert conv(bias=MIS) == -3
    assert conv(act=3) == -4
    assert conv(K=33) == -4
    assert conv(n=0, S=None, plan=None, out=None) == 0


def test_binding_refuses_cpu_tensors():
    torch = pytest.importorskip("torch")
    x = torch.zeros(4 * 655, 16)
    with pytest.raises(ValueError):
        shc.gather_rows(x, torch.zeros(10, 2, dtype=torch.int32), 10, 4, 655, torch.zeros(10, 16))


def test_event_helpers_validation(lib):
    """The stream-ordering event helpers refuse a NULL event before any HIP
    call (destroy accepts it)."""
    assert lib.shc_event_create(None) == -1 and "event" in err(lib)
    assert lib.shc_event_record(None, None) == -1
    assert lib.shc_stream_wait_event(None, None) == -1
    assert lib.shc_event_synchronize(None) == -1
    assert lib.shc_event_destroy(None) == 0


def test_compact_table_start_validation(lib):
    ws = lib.shc_compact_mask_workspace(4, 655)
    host = ctypes.c_int64(0)
    ok = dict(mask=A, B=4, V=655, coords=A, inv=A, row_ptr=A, n_dev=A,
              n_host=ctypes.addressof(host), cap=2620, nbr=A, K=9, table=A, ws=A, ws_bytes=ws)

    def call(**kw):
        a = dict(ok, **kw)
        return lib.shc_compact_mask_table_start(a["mask"], a["B"], a["V"], a["coords"], a["inv"],
                                                a["row_ptr"], a["n_dev"], a["n_host"], a["cap"],
                                                a["nbr"], a["K"], a["table"], a["ws"],
                                                a["ws_bytes"], None)

    assert call(K=0) == -1 and "K" in err(lib)
    assert call(K=33) == -4
    assert call(V=19457, ws_bytes=1 << 30) == -4 and "19456" in err(lib)
    assert call(nbr=None) == -1 and "nbr" in err(lib)
    assert call(nbr=MIS) == -3
    assert call(table=None) == -1 and "table" in err(lib)
    assert call(n_host=None) == -1
    assert call(ws_bytes=ws - 1) == -2
    # pageable host memory cannot receive the kernel's count
    assert call() == -1 and "page-locked" in err(lib)


def _c_layout(tmp_path, struct, fields):
    """offsetof of each field and sizeof of `struct`, from the C compiler."""
    src = tmp_path / f"{struct}.c"
    lines = ["#include <stddef.h>", "#include <stdio.h>", '#include "shc.h"', "int main(void) {",
             f'  printf("%zu\\n", sizeof({struct}));']
    lines += [f'  printf("%zu\\n", offsetof({struct}, {f}));' for f in fields]
    lines += ["  return 0;", "}"]
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / f"{struct}_layout"
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    subprocess.run(["gcc", "-D__HIP_PLATFORM_AMD__", "-I", os.path.dirname(shc.HEADER), "-I",
                    os.path.join(rocm, "include"), str(src), "-o", str(exe)], check=True,
                   capture_output=True)
    vals = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True,
                                           check=True).stdout.split()]
    return vals[0], vals[1:]


@pytest.mark.parametrize("py,c", [(shc.StackLayer, "shc_stack_layer"),
                                  (shc.StackIndexSet, "shc_stack_index_set"),
                                  (shc.StackDesc, "shc_stack_desc")])
def test_stack_struct_layout_matches_header(tmp_path, py, c):
    """The binding's ctypes mirrors of the stack structs have the header's
    size and field offsets."""
    names = [f[0] for f in py._fields_]
    size, offs = _c_layout(tmp_path, c, names)
    assert ctypes.sizeof(py) == size
    for name, off in zip(names, offs):
        assert getattr(py, name).offset == off, name


def test_stack_validation(lib):
    """shc_stack_create refuses a description the path's calls would refuse,
    before any HIP call; shc_stack_run and _destroy take NULL safely.  (Without
    a device no shape takes a conv plan, so the plan buffers' checks are in
    the GPU tests.)"""
    B, V, K = 4, 655, 9
    ws = lib.shc_compact_mask_workspace(B, V)

    def desc(**kw):
        d = shc.StackDesc()
        d.B, d.V, d.K, d.dtype, d.C0 = B, V, K, shc.SHC_BF16, 64
        d.mask, d.x, d.nbr = A, A + 0x100, A + 0x200
        d.table_in_compaction = 1
        d.n_layers = 2
        for l in range(2):
            L = d.layers[l]
            L.kind, L.Cin, L.Cout, L.act = shc.SHC_LAYER_CONV, 64, 64, shc.SHC_ACT_RELU
            L.W, L.bias, L.plan_rows = A + 0x300 + 0x100 * l, None, 0
        for i in range(3):
            d.acts[i] = A + 0x1000 * (i + 1)
        d.last_alt, d.dense_out, d.pooled = A + 0x5000, A + 0x6000, A + 0x7000
        d.incremental, d.prev_coords = 1, A + 0x8000
        d.n_sets = 3
        for s in range(3):
            S = d.sets[s]
            base = A + 0x100000 * (s + 1)
            S.coords, S.inv, S.row_ptr, S.n_active = base, base + 0x100, base + 0x200, base + 0x300
            S.host_count, S.ws, S.ws_bytes, S.table = base + 0x400, base + 0x500, ws, base + 0x600
        d.side, d.tail = 0x1111, 0x2222
        for k, v in kw.items():
            obj, _, name = k.rpartition("__")
            tgt = d
            for part in filter(None, obj.split("__")):
                tgt = getattr(tgt, part[:-1])[int(part[-1])] if part[-1].isdigit() else \
                    getattr(tgt, part)
            setattr(tgt, name, v)
        return d

    def create(d):
        h = ctypes.c_void_p()
        rc = lib.shc_stack_create(ctypes.byref(d), ctypes.byref(h))
        assert not h.value
        return rc

    assert lib.shc_stack_create(None, ctypes.byref(ctypes.c_void_p())) == -1
    assert lib.shc_stack_create(ctypes.byref(desc()), None) == -1
    assert create(desc(B=0)) == -1
    assert create(desc(dtype=5)) == -4
    assert create(desc(n_layers=0)) == -1
    assert create(desc(n_layers=17)) == -1
    assert create(desc(mask=MIS)) == -3
    assert create(desc(C0=48)) == -1 and "Cin = 64" in err(lib)
    assert create(desc(layers0__Cout=40)) == -4
    assert create(desc(layers1__act=7)) == -4
    assert create(desc(layers0__kind=3)) == -4
    assert create(desc(layers0__plan_rows=1 << 40)) == -4 and "plan_rows" in err(lib)
    assert create(desc(layers1__W=None)) == -1
    assert create(desc(K=0)) == -1
    assert create(desc(K=33)) == -4
    assert create(desc(nbr=None)) == -1
    d = desc()
    d.acts[0] = None                  # layer 0 is a conv: the gathered rows are needed
    assert create(d) == -1 and "acts[0]" in err(lib)
    d = desc()
    d.acts[2] = MIS
    assert create(d) == -3
    assert create(desc(last_alt=None)) == -1 and "last_alt" in err(lib)
    assert create(desc(tail=0)) == -1 and "both" in err(lib)
    assert create(desc(tail=0x1111)) == -1 and "different" in err(lib)
    assert create(desc(n_sets=2)) == -1
    assert create(desc(prev_coords=None)) == -1
    assert create(desc(incremental=1, dense_out=None)) == -1
    assert create(desc(table_in_compaction=2)) == -1
    assert create(desc(V=20000)) == -4 and "table" in err(lib)
    assert create(desc(sets0__ws_bytes=ws - 1)) == -2
    assert create(desc(sets1__table=None)) == -1
    assert create(desc(sets2__host_count=None)) == -1
    assert create(desc(sets1__coords=A + 0x100000)) == -1 and "share" in err(lib)
    d = desc()
    d.sets[1].plan[1] = A + 0x9000    # a plan buffer for a layer without plan rows
    assert create(d) == -1 and "plan_rows = 0" in err(lib)
    # a linear layer with a plan row limit
    d = desc()
    d.layers[0].kind = shc.SHC_LAYER_LINEAR
    d.layers[0].plan_rows = 10
    assert create(d) == -1 and "linear" in err(lib)
    # prev_coords aliasing an index set's coords
    assert create(desc(prev_coords=A + 0x200000)) == -1
    # the split conv: a row limit per conv layer, one shared workspace
    need = lib.shc_conv_split_workspace_bytes(100, K, 64, 64, shc.SHC_BF16)
    assert create(desc(layers0__split_rows=-1)) == -1 and "split_rows" in err(lib)
    assert create(desc(layers0__split_rows=100)) == -1 and "split_ws" in err(lib)
    assert create(desc(layers0__split_rows=100, split_ws=MIS, split_ws_bytes=need)) == -3
    assert create(desc(layers0__split_rows=100, layers1__split_rows=100, split_ws=A + 0x9000,
                       split_ws_bytes=need - 1)) == -2
    assert create(desc(split_ws=A + 0x9000, split_ws_bytes=need)) == -1 and \
        "no layer" in err(lib)
    assert create(desc(layers0__split_rows=100, layers0__plan_rows=100, split_ws=A + 0x9000,
                       split_ws_bytes=need)) == -1 and "both" in err(lib)
    assert create(desc(layers0__split_rows=100, dtype=shc.SHC_F32, split_ws=A + 0x9000,
                       split_ws_bytes=need)) == -4
    d = desc(split_ws=A + 0x9000, split_ws_bytes=need)
    d.layers[0].kind = shc.SHC_LAYER_LINEAR
    d.layers[0].split_rows = 100
    assert create(d) == -1 and "linear" in err(lib)
    assert lib.shc_stack_destroy(None) == 0
    cur, prev, n = ctypes.c_int32(0), ctypes.c_int64(0), ctypes.c_int64(0)
    assert lib.shc_stack_run(None, 1, None, ctypes.cast(None, shc.STACK_FEED_FN), None, 0, None,
                             ctypes.byref(cur), ctypes.byref(prev), ctypes.byref(n)) == -1
