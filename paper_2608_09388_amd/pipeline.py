"""A sparse contact-layer stack driven through the C ABI.

``SparseStack`` uploads one workload (mesh neighbour lists, mask, dense
features, layer weights) to the GPU once, allocates every buffer the path
needs at its worst-case size (all B*V rows active), and then runs the path
as a sequence of library calls:

    shc_compact_mask (+ shc_build_neighbor_table) -> shc_gather_rows ->
    (shc_sparse_linear | shc_sparse_neighbor_conv_table) per layer ->
    shc_scatter / shc_segment_maxpool

with the gather fused into the first layer (shc_gather_sparse_linear) when
that layer is linear.

The active set never changes across layers (C'_k = C_k, Sec. 3.2), so the
active count is read back once per mask and passed to every layer call.
This module only moves buffers and issues calls; all arithmetic runs in the
library's kernels.
"""
from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np
import torch

from . import binding as shc
from .synth import BF16, Workload

TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}


def to_device(a: np.ndarray, dtype: str, device) -> torch.Tensor:
    """Upload fp32 values that are exact in `dtype` as a tensor of that dtype."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(device=device, dtype=TORCH_DTYPE[dtype])


class SparseStack:
    def __init__(self, w: Workload, device: str = "cuda", act: int = shc.SHC_ACT_RELU):
        self.w = w
        self.device = torch.device(device)
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
        # compaction outputs (capacity: every row active)
        self.coords = torch.empty((BV, 2), dtype=torch.int32, device=dev)
        self.inv = torch.empty(BV, dtype=torch.int32, device=dev)
        self.row_ptr = torch.empty(self.B + 1, dtype=torch.int32, device=dev)
        self.n_active = torch.empty(4, dtype=torch.int32, device=dev)
        ws = shc.compact_mask_workspace(self.B, self.V)
        self.ws = torch.empty(max(ws, 16), dtype=torch.uint8, device=dev)
        # activations: gathered input + one buffer per layer
        chans = [w.C0] + [l.Cout for l in w.layers]
        self.acts = [torch.empty((BV, c), dtype=self.dtype, device=dev) for c in chans]
        Cl = chans[-1]
        self.dense_out = torch.empty((BV, Cl), dtype=self.dtype, device=dev) if w.scatter else None
        self.pooled = torch.empty((self.B, Cl), dtype=self.dtype, device=dev) if w.pool else None
        self.n = None
        # neighbour-row table of the active set, shared by every conv layer
        has_conv = any(l.kind == "conv" for l in w.layers)
        self.table = (torch.empty((self.K, BV), dtype=torch.int32, device=dev)
                      if has_conv else None)
        # every call of the path marshalled once, on the current stream; the
        # buffers are at full capacity, so each call only takes the row count
        B, V = self.B, self.V
        self._compact = shc.PreparedCompact(self.mask, B, V, self.coords, self.inv, self.row_ptr,
                                            self.n_active, self.ws)
        # A first linear layer reads its rows straight from x (gather fused in);
        # otherwise the active rows are gathered into acts[0] first.
        self.fused_gather = len(w.layers) > 0 and w.layers[0].kind == "linear"
        self._gather = shc.prepare_gather_rows(self.x, self.coords, B, V, self.acts[0])
        self._table = (shc.prepare_build_neighbor_table(self.coords, self.inv, B, V, self.nbr,
                                                        self.table)
                       if self.table is not None else None)
        self._layers = []
        for l, spec in enumerate(w.layers):
            src, dst = self.acts[l], self.acts[l + 1]
            a = act if spec.relu else shc.SHC_ACT_NONE
            if spec.kind == "conv":
                call = shc.prepare_sparse_neighbor_conv_table(src, self.table, self.weights[l],
                                                              self.biases[l], dst, a)
            elif l == 0 and self.fused_gather:
                call = shc.prepare_gather_sparse_linear(self.x, self.coords, B, V,
                                                        self.weights[l], self.biases[l], dst, a)
            else:
                call = shc.prepare_sparse_linear(src, self.weights[l], self.biases[l], dst, a)
            self._layers.append(call)
        last = self.acts[-1]
        self._scatter = (shc.prepare_scatter(last, self.inv, self.coords, B, V, self.dense_out)
                         if self.dense_out is not None else None)
        self._pool = (shc.prepare_segment_maxpool(last, self.row_ptr, B, self.pooled, 0.0)
                      if self.pooled is not None else None)

    # -- individual steps -----------------------------------------------------
    def compact(self) -> int:
        """Compaction; waits for the active count (one host sync per mask),
        then builds the neighbour-row table of the active set if a conv layer
        will read it."""
        self.n = self._compact()
        if self._table is not None:
            self._table(self.n)
        return self.n

    def gather(self):
        """Gather the active rows into acts[0] (not needed by the step when
        the first layer fuses the gather)."""
        self._gather(self.n)

    def layer(self, l: int):
        self._layers[l](self.n)

    def scatter(self):
        self._scatter(self.n)

    def pool(self):
        self._pool(self.n)

    def finish(self):
        if self._scatter is not None:
            self._scatter(self.n)
        if self._pool is not None:
            self._pool(self.n)

    def step(self) -> int:
        """One pass of the whole path over the workload's batch."""
        self.compact()
        if not self.fused_gather:
            self.gather()
        for call in self._layers:
            call(self.n)
        self.finish()
        return self.n

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
