"""A sparse contact-layer stack driven through the C ABI.

``SparseStack`` uploads one workload (mesh neighbour lists, mask, dense
features, layer weights) to the GPU once, allocates every buffer the path
needs at its worst-case size (all B*V rows active), and then runs the path
as a sequence of library calls:

    shc_compact_mask_start -> shc_compact_mask_wait (-> shc_build_neighbor_table)
    -> shc_gather_rows -> (shc_sparse_linear | shc_sparse_neighbor_conv_table)
    per layer -> shc_scatter / shc_segment_maxpool

with the gather fused into the first layer (shc_gather_sparse_linear) when
that layer is linear, and a conv layer's neighbour-row table written by the
compaction itself (shc_compact_mask_table_start) when a body's vertices fit
its on-chip row numbering.

The active set never changes across layers (C'_k = C_k, Sec. 3.2), so the
active count is read back once per mask and passed to every layer call.  For
the same reason the conv's index lists can be built once per mask and conv
shape (shc_build_conv_plan) and read by every layer of that shape
(shc_sparse_neighbor_conv_planned); by default this is done for shapes shared
by two or more conv layers.

The index buffers of a mask (coords, inv, row_ptr, the neighbour-row table)
exist twice (three times with a side stream).  ``run(steps)`` uses this for
consecutive batches: the compaction of batch k + 1 goes into another set and
is enqueued before the scatter and pool of batch k, so the host learns the
next active count while the GPU still has batch k's tail to run, and the
stream never idles on that wait.  With a side stream the compaction runs on
it, and the scatter and pool of batch k run on a third stream beside batch
k + 1's layers (the last layer's output alternates between two buffers).
Every batch still runs the whole path.  ``run`` issues these calls from the
library's own loop (shc_stack_run, one call for all the batches) unless the
stack is made with executor="python", which issues the same calls one by one
from this module.

With ``incremental_scatter`` the dense output is kept from batch to batch and
each scatter is shc_scatter_update: the rows of the previous batch that are
inactive now are zeroed and this batch's rows written, instead of all B*V
rows; the result is the zero-fill scatter's, bit for bit.

This module only moves buffers and issues calls; all arithmetic runs in the
library's kernels.
"""
from __future__ import annotations

from typing import Callable, Dict, Optional, Sequence, Tuple

import numpy as np
import torch

from . import binding as shc
from .synth import Workload

TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}

# Active fraction of the B*V rows up to which a 256-channel conv layer runs as
# the split conv by default.  On the sequence workload's mesh (2048 x 655
# vertices, K = 9, 256 -> 256) the split conv took 61 / 146 / 245 us against
# 130 / 226 / 343 us for the table conv at 5 / 10 / 15% Bernoulli masks; its
# workspace limit (2^31 bytes) ends it near 20% there.
SPLIT_DENSITY = 0.2

# Active fraction of the B*V rows up to which a conv layer of a shape the
# packed conv takes (bf16, 64 or 128 channels, K <= 9) runs as the packed conv
# by default.  On the density-sweep batch (B = 128, V = 10475, K = 9,
# 128 -> 128) it took 10.3 / 21.6 / 109.9 us against 12.6 / 25.9 / 114.9 us
# for the table conv at 1 / 5 / 20% Bernoulli masks.  It runs one workgroup
# of eight wavefronts per CU when C_out = 128 and four when C_out = 64; with
# four (one per SIMD) and on small batches (under PACKED_MIN_ROWS_PER_CU rows
# per CU the weights' load dominates) the other kernels were faster: the
# full-mesh 64 -> 64 layer at its 5% cap took 66 us against 36 us, the
# encoder's step 0.069 ms against 0.052 ms.
PACKED_DENSITY = 0.25
PACKED_MIN_ROWS_PER_CU = 32


def to_device(a: np.ndarray, dtype: str, device) -> torch.Tensor:
    """Upload fp32 values that are exact in `dtype` as a tensor of that dtype."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(device=device, dtype=TORCH_DTYPE[dtype])


class _IndexSet:
    """The compaction outputs of one mask and every call that reads them."""

    def __init__(self, st: "SparseStack"):
        dev, B, V, K = st.device, st.B, st.V, st.K
        BV = B * V
        self.coords = torch.empty((BV, 2), dtype=torch.int32, device=dev)
        self.inv = torch.empty(BV, dtype=torch.int32, device=dev)
        self.row_ptr = torch.empty(B + 1, dtype=torch.int32, device=dev)
        self.n_active = torch.empty(4, dtype=torch.int32, device=dev)
        ws = shc.compact_mask_workspace(B, V)
        self.ws = torch.empty(max(ws, 16), dtype=torch.uint8, device=dev)
        has_conv = any(l.kind == "conv" for l in st.w.layers)
        # neighbour-row table of the active set, shared by every conv layer
        self.table = (torch.empty((K, BV), dtype=torch.int32, device=dev)
                      if has_conv else None)
        self.n: Optional[int] = None
        # every call marshalled once, on the current stream; the buffers are at
        # full capacity, so each call only takes the row count.  compact.start()
        # also writes the neighbour-row table when one is needed and a body's
        # row numbering fits on chip (shc_compact_mask_table_start): `fused`
        self.fused = self.table is not None and V <= shc.COMPACT_TABLE_MAX_V and K <= 32
        tbl = dict(nbr=st.nbr, table=self.table) if self.fused else {}
        self.compact = shc.PreparedCompact(st.mask, B, V, self.coords, self.inv, self.row_ptr,
                                           self.n_active, self.ws, **tbl)
        # the same compaction (and table build) on the side stream (run() with
        # side_stream: they overlap the previous batch's layers, scatter and pool)
        self.compact_side = (shc.PreparedCompact(st.mask, B, V, self.coords, self.inv,
                                                 self.row_ptr, self.n_active, self.ws,
                                                 stream=st.side, **tbl)
                             if st.side is not None else None)
        self.gather = shc.prepare_gather_rows(st.x, self.coords, B, V, st.acts[0])
        self.table_call = (shc.prepare_build_neighbor_table(self.coords, self.inv, B, V, st.nbr,
                                                            self.table)
                           if self.table is not None else None)
        self.table_side = (shc.prepare_build_neighbor_table(self.coords, self.inv, B, V, st.nbr,
                                                            self.table, stream=st.side)
                           if self.table is not None and st.side is not None and not self.fused
                           else None)
        # conv plans (shc_build_conv_plan): one per conv shape that takes one,
        # built after the table, read by every conv layer of that shape while
        # the batch's row count is within the shape's limit
        self.plans = {}
        for key, n_lim in st.plan_shapes.items():
            K_, Cin, Cout = key
            nb = shc.conv_plan_bytes(min(BV, n_lim), K_, Cin, Cout)
            buf = torch.empty(nb, dtype=torch.uint8, device=dev)
            build = shc.prepare_build_conv_plan(self.table, K_, Cin, Cout, buf)
            build_side = (shc.prepare_build_conv_plan(self.table, K_, Cin, Cout, buf,
                                                      stream=st.side)
                          if st.side is not None else None)
            self.plans[key] = (buf, n_lim, build, build_side)
        self.layers = [self._layer_call(st, l, st.acts[l + 1]) for l in range(len(st.w.layers))]
        last = st.acts[-1]
        self.scatter = self._scatter_call(st, last, None)
        self.pool = (shc.prepare_segment_maxpool(last, self.row_ptr, B, st.pooled, 0.0)
                     if st.pooled is not None else None)
        # run() with a side stream: the last layer writes one of two buffers
        # (acts[-1] or st.last_alt), and the scatter and pool of that buffer
        # run on the tail stream
        self.last_into = self.scatter_tail = self.pool_tail = None
        if st.tail is not None and st.w.layers:
            L = (st.acts[-1], st.last_alt)
            self.last_into = [self._layer_call(st, len(st.w.layers) - 1, L[i]) for i in range(2)]
            self.scatter_tail = [self._scatter_call(st, L[i], st.tail) for i in range(2)]
            self.pool_tail = [shc.prepare_segment_maxpool(L[i], self.row_ptr, B, st.pooled, 0.0,
                                                          stream=st.tail)
                              if st.pooled is not None else None for i in range(2)]

    def _scatter_call(self, st: "SparseStack", src: torch.Tensor, stream):
        """The scatter of src into the dense output (on `stream`, None: the
        stack's own): a zero-fill scatter, or with incremental_scatter an
        update of the previous batch's output."""
        if st.dense_out is None:
            return None
        B, V = st.B, st.V
        if not st.incremental_scatter:
            return shc.prepare_scatter(src, self.inv, self.coords, B, V, st.dense_out,
                                       stream=stream)
        upd = shc.prepare_scatter_update(src, self.inv, self.coords, st.prev_coords, B, V,
                                         st.dense_out, stream=stream)
        return _IncrementalScatter(st, upd, self.coords, stream)

    def build_plans(self, n: int, side: bool = False):
        """The conv plans of this set's n rows (on the side stream: side)."""
        for buf, n_lim, build, build_side in self.plans.values():
            if 0 < n <= n_lim:
                (build_side if side else build)(n)

    def _layer_call(self, st: "SparseStack", l: int, dst: torch.Tensor):
        """Layer l of the stack on this index set, writing dst."""
        spec = st.w.layers[l]
        src = st.acts[l]
        a = st.act if spec.relu else shc.SHC_ACT_NONE
        if spec.kind == "conv":
            table = shc.prepare_sparse_neighbor_conv_table(src, self.table, st.weights[l],
                                                           st.biases[l], dst, a)
            if l in st.packed_rows:
                K_, Cin, Cout = st.weights[l].shape
                packed = shc.prepare_sparse_neighbor_conv_packed(src, self.table, st.packed_w[l],
                                                                 K_, Cin, Cout, st.biases[l],
                                                                 dst, a)
                return _SplitConv(table, packed, st.packed_rows[l], st.packed_min_rows)
            if l in st.split_rows:
                split = shc.prepare_sparse_neighbor_conv_split(src, self.table, st.weights[l],
                                                               st.biases[l], dst, st.split_ws, a)
                return _SplitConv(table, split, st.split_rows[l])
            plan = self.plans.get(tuple(st.weights[l].shape))
            if plan is None:
                return table
            planned = shc.prepare_sparse_neighbor_conv_planned(src, plan[0], st.weights[l],
                                                               st.biases[l], dst, a)
            return _PlannedConv(table, planned, plan[1])
        if l == 0 and st.fused_gather:
            return shc.prepare_gather_sparse_linear(st.x, self.coords, st.B, st.V, st.weights[l],
                                                    st.biases[l], dst, a)
        return shc.prepare_sparse_linear(src, st.weights[l], st.biases[l], dst, a)


class _IncrementalScatter:
    """shc_scatter_update from the previous scattered batch's coordinates
    (kept in the stack's prev_coords), then this batch's coordinates copied
    there, both on the scatter's stream."""

    def __init__(self, st: "SparseStack", upd, coords: torch.Tensor, stream):
        self.st, self.upd, self.coords = st, upd, coords
        self.stream = stream if stream is not None else st.main

    def __call__(self, n: int):
        st = self.st
        self.upd(n, st.prev_n)
        with torch.cuda.stream(self.stream):
            st.prev_coords[:n].copy_(self.coords[:n])
        st.prev_n = n


class _SplitConv:
    """A conv layer that runs as the split (or packed) conv when the batch's
    row count is within its limit, else from the table."""

    def __init__(self, table, split, n_lim: int, n_min: int = 0):
        self.table, self.split, self.n_lim, self.n_min = table, split, n_lim, max(n_min, 1)

    def __call__(self, n: int):
        return self.split(n) if self.n_min <= n <= self.n_lim else self.table(n)


def _split_rows_limit(want: int, K: int, Cin: int, Cout: int) -> int:
    """The largest row count up to `want` whose split conv of this shape the
    library takes (0: none)."""
    if want <= 0 or shc.conv_split_workspace_bytes(1, K, Cin, Cout) == 0:
        return 0
    if shc.conv_split_workspace_bytes(want, K, Cin, Cout) > 0:
        return want
    lo, hi = 1, want  # split at lo, none at hi
    while hi - lo > 1:
        mid = (lo + hi) // 2
        if shc.conv_split_workspace_bytes(mid, K, Cin, Cout) > 0:
            lo = mid
        else:
            hi = mid
    return lo


class _PlannedConv:
    """A conv layer that reads its set's plan when the batch's row count has
    one (the plan was built for it), else the table."""

    def __init__(self, table, planned, n_lim: int):
        self.table, self.planned, self.n_lim = table, planned, n_lim

    def __call__(self, n: int):
        return self.planned(n) if 0 < n <= self.n_lim else self.table(n)


class SparseStack:
    def __init__(self, w: Workload, device: str = "cuda", act: int = shc.SHC_ACT_RELU,
                 side_stream: bool = False, conv_plans: Optional[bool] = None,
                 incremental_scatter: bool = False, executor: str = "native",
                 split_conv: Optional[bool] = None, packed_conv: Optional[bool] = None):
        if executor not in ("native", "python"):
            raise ValueError(f"executor = {executor!r}: 'native' or 'python'")
        self.w = w
        self.device = torch.device(device)
        # every prepared call below launches on the stream current now; step()
        # and run() order that stream after the caller's stream when they
        # are called under another one (and the caller's stream after them)
        self.main = torch.cuda.current_stream(self.device)
        self._bracket = None
        # with side_stream, run() uses two more streams (default priority): the
        # side stream for the next batch's compaction and table, the tail stream
        # for each batch's scatter and pool; None: everything on the current one
        self.side = torch.cuda.Stream(device=self.device) if side_stream else None
        self.tail = torch.cuda.Stream(device=self.device) if side_stream else None
        self._events = None
        if side_stream:
            with torch.cuda.device(self.device):
                ev = shc.StreamEvent
                self._events = dict(set_free=[ev() for _ in range(3)], ready=ev(), x_read=ev(),
                                    last_done=[ev() for _ in range(2)],
                                    tail_done=[ev() for _ in range(2)], tail_end=ev())
        self.dtype = TORCH_DTYPE[w.dtype]
        self.B, self.V, self.K = w.B, w.V, w.K
        self.act = act
        dev = self.device
        BV = self.B * self.V
        self.mask = torch.from_numpy(np.ascontiguousarray(w.mask.reshape(-1))).to(dev)
        self.nbr = torch.from_numpy(np.ascontiguousarray(w.nbr, dtype=np.int32)).to(dev)
        self.x = to_device(w.x, w.dtype, dev)
        self.weights = [to_device(l.W, w.dtype, dev) for l in w.layers]
        self.biases = [None if l.bias is None else
                       torch.from_numpy(l.bias.astype(np.float32)).to(dev) for l in w.layers]
        # activations: gathered input + one buffer per layer
        chans = [w.C0] + [l.Cout for l in w.layers]
        self.acts = [torch.empty((BV, c), dtype=self.dtype, device=dev) for c in chans]
        # second buffer of the last layer's output (run() with side_stream)
        self.last_alt = torch.empty_like(self.acts[-1]) if side_stream else None
        Cl = chans[-1]
        # With incremental_scatter the dense output stays resident from batch
        # to batch: it starts as zeros and each scatter only zeroes the rows
        # the previous batch wrote that are inactive now and writes this
        # batch's rows (shc_scatter_update); it then must not be written by
        # anything else.  Otherwise every scatter writes all B*V rows.
        self.incremental_scatter = bool(incremental_scatter and w.scatter)
        self.dense_out = ((torch.zeros if self.incremental_scatter else torch.empty)(
            (BV, Cl), dtype=self.dtype, device=dev) if w.scatter else None)
        self.prev_coords = (torch.empty((BV, 2), dtype=torch.int32, device=dev)
                            if self.incremental_scatter else None)
        self.prev_n = 0
        self.pooled = torch.empty((self.B, Cl), dtype=self.dtype, device=dev) if w.pool else None
        # A first linear layer reads its rows straight from x (gather fused in);
        # otherwise the active rows are gathered into acts[0] first.
        self.fused_gather = len(w.layers) > 0 and w.layers[0].kind == "linear"
        # Conv shapes that read a plan of the active set instead of sorting
        # the table's rows in every layer and column slice.  A plan costs a
        # launch of its own (7.7 us for 67 K rows at K = 9, C = 128, against
        # 4.4 us saved per planned layer), so by default a shape takes one
        # only when two or more conv layers share it; conv_plans = True /
        # False forces plans on / off for every conv shape that can take one.
        # Conv layers that run as shc_sparse_neighbor_conv_split (slot 0 apart
        # from the other slots, through a workspace) for batches of at most
        # split_rows[l] rows.  By default: layers with 256 input or output
        # channels, up to SPLIT_DENSITY of the B*V rows (the table conv runs
        # them on its tiled kernel, which re-reads the weights per row tile);
        # split_conv = True / False forces it on every shape that takes it / off.
        # Conv layers that run as shc_sparse_neighbor_conv_packed (every slot's
        # weights in registers, packed once here) for batches of at most
        # packed_rows[l] rows.  By default: every shape it takes, up to
        # PACKED_DENSITY of the B*V rows; packed_conv = True / False forces it
        # up to all rows / off.
        self.packed_rows: Dict[int, int] = {}
        self.packed_w: Dict[int, torch.Tensor] = {}
        if w.dtype == "bf16" and packed_conv is not False:
            for l, spec in enumerate(w.layers):
                if spec.kind != "conv":
                    continue
                K_, Cin, Cout = self.weights[l].shape
                nb = shc.conv_packed_weights_bytes(K_, Cin, Cout)
                if nb == 0 or (packed_conv is None and Cout != 128):
                    continue
                rows = BV if packed_conv else int(PACKED_DENSITY * BV)
                rows = min(rows, (2 ** 31 - 1) // (4 * K_))
                if rows > 0:
                    Wp = torch.empty(nb, dtype=torch.uint8, device=dev)
                    shc.pack_conv_weights(self.weights[l], Wp)
                    self.packed_w[l], self.packed_rows[l] = Wp, rows
        cus = torch.cuda.get_device_properties(dev).multi_processor_count
        self.packed_min_rows = 0 if packed_conv else PACKED_MIN_ROWS_PER_CU * cus
        self.split_rows: Dict[int, int] = {}
        if w.dtype == "bf16" and split_conv is not False:
            for l, spec in enumerate(w.layers):
                if spec.kind != "conv" or l in self.packed_rows:
                    continue
                K_, Cin, Cout = self.weights[l].shape
                if split_conv is None and max(Cin, Cout) < 256:
                    continue
                want = BV if split_conv else int(SPLIT_DENSITY * BV)
                rows = _split_rows_limit(min(want, BV), K_, Cin, Cout)
                if rows > 0:
                    self.split_rows[l] = rows
        self.split_ws = None
        if self.split_rows:
            need = max(shc.conv_split_workspace_bytes(r, *self.weights[l].shape)
                       for l, r in self.split_rows.items())
            self.split_ws = torch.empty(need, dtype=torch.uint8, device=dev)
        self.plan_shapes: Dict[Tuple[int, int, int], int] = {}
        split_shapes = {tuple(self.weights[l].shape)
                        for l in list(self.split_rows) + list(self.packed_rows)}
        if w.dtype == "bf16":
            shapes: Dict[Tuple[int, int, int], int] = {}
            for l, spec in enumerate(w.layers):
                if spec.kind == "conv":
                    key = tuple(self.weights[l].shape)
                    shapes[key] = shapes.get(key, 0) + 1
            for key, count in shapes.items():
                if key in split_shapes:
                    continue  # a layer takes a plan, the split or the packed conv
                use = conv_plans if conv_plans is not None else count >= 2
                n_lim = shc.conv_plan_max_rows(*key) if use else 0
                if n_lim > 0:
                    self.plan_shapes[key] = n_lim
        # two index sets, or three with a side stream (run() then checks an
        # index set's reuse from the host; see _run_pipelined)
        self._sets = [_IndexSet(self) for _ in range(3 if side_stream else 2)]
        self._cur = 0
        # run() issues its calls from the library's native loop
        # (shc_stack_run) unless executor = "python" (the same calls, issued
        # from this module); a stack without layers always takes the latter
        self.executor = executor if w.layers else "python"
        self._native = self._make_native() if self.executor == "native" else None

    def _make_native(self) -> shc.StackExecutor:
        """The shc_stack_desc of this stack's buffers, and its executor."""
        w = self.w
        d = shc.StackDesc()
        has_conv = any(l.kind == "conv" for l in w.layers)
        d.B, d.V, d.K = self.B, self.V, self.K if has_conv else 0
        d.dtype = shc.SHC_BF16 if w.dtype == "bf16" else shc.SHC_F32
        d.C0 = w.C0
        d.mask, d.x = self.mask.data_ptr(), self.x.data_ptr()
        d.nbr = self.nbr.data_ptr() if has_conv else None
        d.table_in_compaction = int(self._sets[0].fused)
        d.n_layers = len(w.layers)
        BV = self.B * self.V
        for l, spec in enumerate(w.layers):
            L = d.layers[l]
            W = self.weights[l]
            L.kind = shc.SHC_LAYER_CONV if spec.kind == "conv" else shc.SHC_LAYER_LINEAR
            L.Cin, L.Cout = W.shape[-2], W.shape[-1]
            L.act = self.act if spec.relu else shc.SHC_ACT_NONE
            L.W = W.data_ptr()
            L.bias = self.biases[l].data_ptr() if self.biases[l] is not None else None
            n_lim = self.plan_shapes.get(tuple(W.shape), 0) if spec.kind == "conv" else 0
            L.plan_rows = min(BV, n_lim)
            L.split_rows = self.split_rows.get(l, 0)
            L.Wp = self.packed_w[l].data_ptr() if l in self.packed_w else None
            L.packed_rows = self.packed_rows.get(l, 0)
            L.packed_min_rows = self.packed_min_rows if l in self.packed_rows else 0
        for i, a in enumerate(self.acts):
            d.acts[i] = a.data_ptr()
        d.last_alt = self.last_alt.data_ptr() if self.last_alt is not None else None
        d.dense_out = self.dense_out.data_ptr() if self.dense_out is not None else None
        d.incremental = int(self.incremental_scatter)
        d.prev_coords = self.prev_coords.data_ptr() if self.prev_coords is not None else None
        d.pooled = self.pooled.data_ptr() if self.pooled is not None else None
        d.pool_empty = 0.0
        d.n_sets = len(self._sets)
        keep = []
        for i, s in enumerate(self._sets):
            S = d.sets[i]
            host = torch.zeros(1, dtype=torch.int64, pin_memory=True)
            keep.append(host)
            S.coords, S.inv = s.coords.data_ptr(), s.inv.data_ptr()
            S.row_ptr, S.n_active = s.row_ptr.data_ptr(), s.n_active.data_ptr()
            S.host_count = host.data_ptr()
            S.ws, S.ws_bytes = s.ws.data_ptr(), s.ws.numel()
            S.table = s.table.data_ptr() if s.table is not None else None
            for l, spec in enumerate(w.layers):
                plan = s.plans.get(tuple(self.weights[l].shape)) if spec.kind == "conv" else None
                if plan is not None:
                    S.plan[l], S.plan_bytes[l] = plan[0].data_ptr(), plan[0].numel()
        d.side = self.side.cuda_stream if self.side is not None else None
        d.tail = self.tail.cuda_stream if self.tail is not None else None
        if self.split_ws is not None:
            d.split_ws, d.split_ws_bytes = self.split_ws.data_ptr(), self.split_ws.numel()
        return shc.StackExecutor(d, keep)

    # -- the index set of the current mask -------------------------------------
    @property
    def _set(self) -> _IndexSet:
        return self._sets[self._cur]

    @property
    def n(self) -> Optional[int]:
        return self._set.n

    @n.setter
    def n(self, value: Optional[int]):
        self._set.n = value

    coords = property(lambda self: self._set.coords)
    inv = property(lambda self: self._set.inv)
    row_ptr = property(lambda self: self._set.row_ptr)
    n_active = property(lambda self: self._set.n_active)
    ws = property(lambda self: self._set.ws)
    table = property(lambda self: self._set.table)

    # -- individual steps (on the current index set) ---------------------------
    def compact(self) -> int:
        """Compaction; waits for the active count (one host wait per mask),
        then builds the neighbour-row table of the active set if a conv layer
        will read it."""
        s = self._set
        s.n = s.compact()
        if s.table_call is not None:
            s.table_call(s.n)
        s.build_plans(s.n)
        return s.n

    def build_table(self):
        """The neighbour-row table (and the conv plans) of the current set."""
        self._set.table_call(self.n)
        self._set.build_plans(self.n)

    def gather(self):
        """Gather the active rows into acts[0] (not needed by the step when
        the first layer fuses the gather)."""
        self._set.gather(self.n)

    def layer(self, l: int):
        self._set.layers[l](self.n)

    def scatter(self):
        self._set.scatter(self.n)

    def pool(self):
        self._set.pool(self.n)

    def finish(self):
        """Scatter and pool of the current batch."""
        s = self._set
        if s.scatter is not None:
            s.scatter(s.n)
        if s.pool is not None:
            s.pool(s.n)

    def _front(self, s: _IndexSet, around=None, table_done: bool = False,
               plans_done: bool = False):
        """Everything of a batch after its compaction, up to its last layer;
        ``around = (l, ev_a, ev_b)`` records the events around layer l."""
        if s.table_call is not None and not table_done:
            s.table_call(s.n)
        if not plans_done:
            s.build_plans(s.n)
        if not self.fused_gather:
            s.gather(s.n)
        for l, call in enumerate(s.layers):
            if around is not None and around[0] == l:
                around[1].record()
            call(s.n)
            if around is not None and around[0] == l:
                around[2].record()

    def _enter(self):
        """If the caller's current stream is not the stack's own, make the
        stack's stream wait for the caller's work so far; returns the
        caller's stream, or None when they are the same."""
        cur = torch.cuda.current_stream(self.device)
        if cur == self.main:
            return None
        if self._bracket is None:
            with torch.cuda.device(self.device):
                self._bracket = (shc.StreamEvent(), shc.StreamEvent())
        self._bracket[0].record(cur)
        self._bracket[0].wait(self.main)
        return cur

    def _leave(self, cur):
        """The caller's stream waits for the stack's work (see _enter)."""
        if cur is not None:
            self._bracket[1].record(self.main)
            self._bracket[1].wait(cur)

    def step(self) -> int:
        """One pass of the whole path over the workload's batch, on its own."""
        cur = self._enter()
        s = self._set
        s.n = s.compact()
        self._front(s)
        self.finish()
        self._leave(cur)
        return s.n

    def run(self, steps: int, around_layer: Optional[Tuple[int, Sequence]] = None,
            feed: Optional[Callable[[int], None]] = None) -> int:
        """`steps` passes of the whole path over consecutive batches, the
        compaction of each batch overlapped with the scatter and pool of the
        one before (module docstring); with a side stream, each batch's scatter
        and pool also run beside the next batch's layers (_run_pipelined).

        ``feed(k)``, if given, is called just before batch k's compaction is
        enqueued and may write batch k's mask and features into ``mask`` and
        ``x`` with work on the stream current when it is called (the side
        stream in a pipelined run, after the gather of batch k - 1; without
        it every batch reuses them).  ``around_layer = (l, [(ev_a, ev_b), ...])`` records one pair of
        events around layer l of every batch (a pair of None: none for that
        batch).  The outputs left behind are the
        last batch's.  Returns its N'."""
        if steps <= 0:
            return self.n or 0
        cur = self._enter()
        try:
            with torch.cuda.stream(self.main):
                if self._native is not None:
                    return self._run_native(steps, around_layer, feed)
                if self.side is not None and self.w.layers:
                    return self._run_pipelined(steps, around_layer, feed)
                return self._run_serial(steps, around_layer, feed)
        finally:
            self._leave(cur)

    def _run_native(self, steps: int, around_layer, feed) -> int:
        """run() through shc_stack_run: the schedule of _run_serial or
        _run_pipelined, issued from the library."""
        tl, ev = 0, None
        if around_layer is not None:
            tl, pairs = around_layer
            ev = []
            for pair in pairs[:steps]:
                if pair[0] is None:
                    ev += [0, 0]
                    continue
                for e in pair:
                    if not e.cuda_event:    # torch creates the HIP event at its first record
                        e.record(self.main)
                ev += [pair[0].cuda_event, pair[1].cuda_event]
        fd = None
        if feed is not None:
            side_h = self.side.cuda_stream if self.side is not None else None

            def fd(k: int, h: int):
                with torch.cuda.stream(self.side if side_h is not None and h == side_h
                                       else self.main):
                    feed(k)
        n, cur, prev = self._native.run(steps, self.main, fd, tl, ev, self._cur, self.prev_n)
        self._cur = cur
        self._set.n = n
        self.prev_n = prev
        return n

    def _run_serial(self, steps: int, around_layer, feed) -> int:
        """run() on the stack's own stream alone."""
        s = self._set
        if feed is not None:
            feed(0)
        s.compact.start()
        s.n = s.compact.wait()
        for k in range(steps):
            ev = None
            if around_layer is not None and around_layer[1][k][0] is not None:
                ev = (around_layer[0], *around_layer[1][k])
            self._front(s, ev, table_done=s.fused)
            nxt = None
            if k + 1 < steps:
                self._cur = (self._cur + 1) % len(self._sets)
                nxt = self._set
                if feed is not None:
                    feed(k + 1)
                nxt.compact.start()
            if s.scatter is not None:
                s.scatter(s.n)
            if s.pool is not None:
                s.pool(s.n)
            if nxt is not None:
                nxt.n = nxt.compact.wait()
                s = nxt
        return s.n

    def _run_pipelined(self, steps: int, around_layer, feed) -> int:
        """run() over three streams: the current stream runs each batch's
        layers; the side stream the next batch's compaction (which also
        writes its neighbour-row table); the tail stream each batch's scatter
        and pool, beside the next batch's layers.

        The last layer writes one of two buffers (acts[-1], last_alt) in turn,
        the last batch into acts[-1], so the scatter and pool of batch k read
        theirs while batch k + 1's layers write the other.  Three index sets
        rotate: batch k + 1's compaction writes the set last read by batch
        k - 2's scatter and pool, and the host checks that they have finished
        (an event on the tail stream, synchronised from the host; the host
        runs at most about two batches ahead, so it has almost always fired)
        instead of making the side stream wait for it on the GPU.  GPU waits:
        the current stream on the side stream's table before a batch's layers
        and on the tail stream before it overwrites a buffer the tail still
        reads; the tail stream on the current stream's last layer of its
        batch; the side stream on the gather of the batch before (the read
        of ``x``) ahead of ``feed``, which runs with the side stream current
        so that the next batch's inputs are written and compacted beside the
        current batch's later layers.  At the end the current
        stream waits for the tail stream, so work the caller enqueues after
        run() sees the last batch's scatter and pool.  The events carry no
        system-scope fence (shc_event_create): a default event's cache
        write-back at every record costs the step microseconds.  Every batch
        runs the whole path."""
        main = self.main
        side, tail = self.side, self.tail
        ev = self._events
        ns = len(self._sets)
        set_used = [False] * ns
        buf_used = [False, False]
        nl = len(self.w.layers)
        cur = self._cur
        s = self._sets[cur]
        if feed is not None:
            feed(0)
        s.compact.start()
        s.n = s.compact.wait()
        table_done = s.fused
        plans_done = False
        for k in range(steps):
            i = (steps - 1 - k) % 2        # the last batch writes acts[-1]
            around = None
            if around_layer is not None and around_layer[1][k][0] is not None:
                around = (around_layer[0], *around_layer[1][k])
            # layers of batch k (current stream)
            if s.table_call is not None and not table_done:
                s.table_call(s.n)
            if not plans_done:
                s.build_plans(s.n)
            if not self.fused_gather:
                s.gather(s.n)
                if feed is not None:
                    ev["x_read"].record(main)
            for l in range(nl):
                call = s.layers[l]
                if l == nl - 1:
                    if buf_used[i]:
                        ev["tail_done"][i].wait(main)
                    call = s.last_into[i]
                if around is not None and around[0] == l:
                    around[1].record()
                call(s.n)
                if around is not None and around[0] == l:
                    around[2].record()
                if l == 0 and self.fused_gather and feed is not None:
                    ev["x_read"].record(main)
            ev["last_done"][i].record(main)
            buf_used[i] = True
            # compaction of batch k + 1 (side stream)
            nxt_i = (cur + 1) % ns
            nxt = self._sets[nxt_i] if k + 1 < steps else None
            if nxt is not None:
                if feed is not None:
                    # batch k + 1's inputs may be written once batch k's
                    # gather has read x (its compaction read the mask
                    # earlier on the side stream)
                    ev["x_read"].wait(side)
                    with torch.cuda.stream(side):
                        feed(k + 1)
                if set_used[nxt_i]:
                    ev["set_free"][nxt_i].synchronize()
                nxt.compact_side.start()
            # scatter and pool of batch k (tail stream)
            ev["last_done"][i].wait(tail)
            if s.scatter_tail[i] is not None:
                s.scatter_tail[i](s.n)
            if s.pool_tail[i] is not None:
                s.pool_tail[i](s.n)
            ev["tail_done"][i].record(tail)
            ev["set_free"][cur].record(tail)
            set_used[cur] = True
            if nxt is not None:
                nxt.n = nxt.compact_side.wait()
                if nxt.table_side is not None:
                    nxt.table_side(nxt.n)
                nxt.build_plans(nxt.n, side=True)
                table_done = nxt.table is not None    # built on the side stream
                plans_done = True
                ev["ready"].record(side)
                ev["ready"].wait(main)
                cur = nxt_i
                s = nxt
        ev["tail_end"].record(tail)
        ev["tail_end"].wait(main)
        self._cur = cur
        return s.n

    # -- results on the host --------------------------------------------------
    def rows(self, l: int) -> np.ndarray:
        """Active rows of activation l (0 = gathered input) as fp64 numpy."""
        return self.acts[l][: self.n].float().cpu().numpy().astype(np.float64)

    def results(self) -> Dict[str, object]:
        torch.cuda.synchronize(self.device)
        n = self.n
        out = dict(n=n, coords=self.coords[:n].cpu().numpy(), inv=self.inv.cpu().numpy(),
                   row_ptr=self.row_ptr.cpu().numpy(),
                   n_dev=int(self.n_active[0].item()),
                   outs=[self.rows(l + 1) for l in range(len(self.w.layers))])
        if self.pooled is not None:
            out["pool"] = self.pooled.float().cpu().numpy().astype(np.float64)
        if self.dense_out is not None:
            out["dense"] = self.dense_out.float().cpu().numpy().astype(np.float64)
        return out
