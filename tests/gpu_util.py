"""Helpers for the GPU parity tests (tolerances, uploads)."""
import numpy as np
import torch

from paper_2608_09388_amd import binding as shc

# per-element tolerance relative to the abs-sum scale s = sum |a||w| + |b| of
# each output: the benchmark spec's figures, used as they stand for fp32 and as the
# ceiling of the derived bf16 bound below
RTOL = {"f32": 1e-5, "bf16": 2e-2}
TORCH = {"f32": torch.float32, "bf16": torch.bfloat16}


def bf16_layer_bound(ref, scale, n_terms):
    """Per-element bound on |gpu - ref| for a bf16 layer output.

    Both sides take the same bf16 operands, whose products are exact in fp32.
    The GPU sums the n_terms products and the bias in fp32 in some order: the
    error of any summation order is at most (n_terms + 1) * u * s with
    u = 2^-24, or 2^-23 for a unit that truncates; twice the truncating
    figure, (n_terms + 2) * 2^-22 * s, is taken.  The output is then rounded
    once to bf16 (8 significant bits, round to nearest even): at most 2^-8 of
    its magnitude, |ref| plus the summation error, whose 2^-8 share one more
    term of the sum covers.  2^-133 covers the rounding of a value in bf16's
    subnormal range.  The bound is capped at the 2e-2 * s ceiling."""
    ref = np.abs(np.asarray(ref, np.float64))
    scale = np.asarray(scale, np.float64)
    derived = 2.0 ** -8 * ref + (n_terms + 3) * 2.0 ** -22 * scale + 2.0 ** -133
    return np.minimum(derived, RTOL["bf16"] * scale)


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


def assert_scaled_close(got, ref, scale, dtype, what="", n_terms=None):
    """|got - ref| <= bound elementwise (ref, scale in fp64): rtol * scale for
    fp32, bf16_layer_bound for bf16 (which needs the number of products
    summed into every output, n_terms)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = np.asarray(scale, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = np.abs(got - ref)
    if dtype == "bf16":
        if n_terms is None:
            raise ValueError(f"{what}: a bf16 check needs n_terms")
        bound = bf16_layer_bound(ref, scale, n_terms)
        name = f"the derived bf16 bound (n_terms={n_terms})"
    else:
        bound = RTOL[dtype] * scale
        name = f"rtol={RTOL[dtype]} x abs-sum scale"
    bad = err > bound
    if bad.any():
        idx = np.argwhere(bad)[:5]
        worst = np.max(err / np.maximum(bound, 1e-300))
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} outside {name};"
                             f" worst error/bound {worst:.3g}; first at {idx.tolist()}:"
                             f" got {got[tuple(idx[0])]}, ref {ref[tuple(idx[0])]}")


# group normalization: the mean is an fp64 sum; the squared deviations are
# summed in fp32 over a thread's rows (at most 16 positive terms: relative
# error 15 * 2^-24) and in fp64 beyond, so 1/sqrt(var + eps) errs by at most
# about 8 * 2^-24 relative.  Each output is ((x - mu_hi) - mu_lo) * rs in fp32
# with the mean as two fp32 terms: four more roundings of 2^-24 of the output.
# In all about 12 * 2^-24 = 7e-7 relative, under the benchmark spec's 1e-5 for
# fp32; bf16 adds the output's rounding: 2^-8 + 16 * 2^-24.  The absolute
# floor covers outputs near zero, where the rounding of the fp64 mean matters:
# a sum of n values in any order is within (n - 1) 2^-53 sum |x| of exact, so
# mu is within n 2^-53 max |x|, and the output moves by at most that times
# rs <= 1 / sqrt(eps); twice that, n 2^-52 max |x| / sqrt(eps), is taken.
GN_RTOL = {"f32": 1e-5, "bf16": 2.0 ** -8 + 16 * 2.0 ** -24}


def gn_floor(S, row_ptr, G, eps=1e-5):
    """The absolute floor above for the inputs S [n][C] and bodies row_ptr."""
    S = np.asarray(S, np.float64)
    C = S.shape[1]
    rows = int(np.max(np.diff(np.asarray(row_ptr)))) if len(row_ptr) > 1 else 0
    n = max(rows, 1) * (C // G)
    big = float(np.max(np.abs(S))) if S.size else 0.0
    return n * 2.0 ** -52 * big / np.sqrt(eps)


def assert_gn_close(got, ref, dtype, floor, what=""):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = np.abs(got - ref)
    bound = floor + GN_RTOL[dtype] * np.abs(ref)
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
