"""Helpers for the GPU parity tests (tolerances, uploads)."""
import numpy as np
import torch

from paper_2608_09388_amd import binding as shc

# per-element tolerance relative to the abs-sum scale sum |a||w| + |b| of each output
RTOL = {"f32": 1e-5, "bf16": 2e-2}
TORCH = {"f32": torch.float32, "bf16": torch.bfloat16}


def require_gpu():
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a visible GPU (torch.cuda.is_available() is False)")
    shc.load()   # fail loudly when the library is missing
    return torch.device("cuda:0")


def up(a, dtype=None, device="cuda:0"):
    """numpy -> device tensor; float arrays go to `dtype` ('f32' / 'bf16')."""
    a = np.ascontiguousarray(a)
    if dtype is None:
        return torch.from_numpy(a).to(device)
    return torch.from_numpy(a.astype(np.float32)).to(device=device, dtype=TORCH[dtype])


def down(t):
    return t.float().cpu().numpy().astype(np.float64) if t.is_floating_point() else t.cpu().numpy()


def assert_scaled_close(got, ref, scale, dtype, what=""):
    """|got - ref| <= rtol * scale elementwise (ref, scale in fp64)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = np.asarray(scale, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = np.abs(got - ref)
    bound = RTOL[dtype] * scale
    bad = err > bound
    if bad.any():
        idx = np.argwhere(bad)[:5]
        worst = np.max(err / np.maximum(scale, 1e-300))
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} outside rtol={RTOL[dtype]}"
                             f" x abs-sum scale; worst rel {worst:.3g}; first at {idx.tolist()}:"
                             f" got {got[tuple(idx[0])]}, ref {ref[tuple(idx[0])]}")


# group normalization: sequential fp32 sums over at most ~280 terms (a
# thread's rows, the threads of a channel, the channels of a group) bound the
# error by about 1e-4 * (1 + |ref|) at these sizes; bf16 adds the output's
# rounding, half an ulp: 2^-8 * |ref|
GN_ATOL = 1e-4
GN_RTOL = {"f32": 1e-4, "bf16": 2.0 ** -8 + 1e-4}


def assert_gn_close(got, ref, dtype, what=""):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = np.abs(got - ref)
    bound = GN_ATOL + GN_RTOL[dtype] * np.abs(ref)
    bad = err > bound
    if bad.any():
        idx = np.argwhere(bad)[:3]
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} outside the bound; worst "
                             f"excess {np.max(err - bound):.3g}; first at {idx.tolist()}")


def assert_normwise_close(got, ref, dtype, what=""):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    num = np.linalg.norm(got - ref)
    den = max(np.linalg.norm(ref), 1e-300)
    assert num / den <= RTOL[dtype], f"{what}: normwise error {num / den:.3g} > {RTOL[dtype]}"


class Compaction:
    """Device buffers for one compaction of a [B][V] mask."""

    def __init__(self, mask: np.ndarray, cap=None, device="cuda:0"):
        B, V = mask.shape
        self.B, self.V = B, V
        self.cap = B * V if cap is None else cap
        self.mask = up(mask.reshape(-1).astype(np.uint8), device=device)
        self.coords = torch.full((max(self.cap, 1), 2), -7, dtype=torch.int32, device=device)
        if self.cap == 0:
            self.coords = self.coords[:0]
        self.inv = torch.full((B * V,), -7, dtype=torch.int32, device=device)
        self.row_ptr = torch.full((B + 1,), -7, dtype=torch.int32, device=device)
        self.n_dev = torch.full((4,), -7, dtype=torch.int32, device=device)
        self.ws = torch.empty(max(shc.compact_mask_workspace(B, V), 16), dtype=torch.uint8,
                              device=device)
        self.n = None

    def run(self, want_host=True):
        self.n = shc.compact_mask(self.mask, self.B, self.V, self.coords, self.inv, self.row_ptr,
                                  self.n_dev, self.ws, want_host_count=want_host)
        return self.n
