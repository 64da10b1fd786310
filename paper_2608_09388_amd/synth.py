"""Seeded synthetic inputs for the sparse contact-layer path.

This module draws the data that both the HIP path and the CPU oracle consume:
mesh points, k-nearest-neighbour lists, contact masks, features and weights.
It holds none of the method's arithmetic (no compaction, no layer maths, no
pooling); it only makes inputs.  The paper's workloads are SMPL-X bodies
reduced to 655 vertices with roughly one vertex in ten kept per mask
(Sec. 4.4, Table 4); the body meshes themselves are not available, so the
shapes below stand in for them:

* body surface: seeded uniform points on the unit sphere (655 vertices) or on
  an ellipsoid with axes (0.3, 0.9, 0.2) (10475 vertices, full SMPL-X size);
* neighbourhood: the K = 9 exact Euclidean nearest neighbours of every vertex,
  the vertex itself first, ties broken towards the lower index -- the 9-slot
  mesh analogue of the paper's 3x3 kernel (Sec. 3.2, Eq. 4);
* masks: per-vertex Bernoulli draws (Sec. 3.1, Eq. 1, "binomial" sampling),
  a geometric contact cap, or temporally coherent two-state Markov runs;
* features ~ N(0, 1); weights ~ N(0, std = 1/sqrt(fan_in)).

Every stream is drawn from ``numpy.random.default_rng(seed)`` with
``seed = 1000 * config + stream``; stream 0 = points, 1 = mask, 2 = features,
3 + l = weights of layer l.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import List, Optional, Sequence

import numpy as np

F32 = "f32"
BF16 = "bf16"

# ----------------------------------------------------------------------------
# geometry
# ----------------------------------------------------------------------------


def _rng(config: int, stream: int) -> np.random.Generator:
    return np.random.default_rng(1000 * int(config) + int(stream))


def sphere_points(V: int, rng: np.random.Generator) -> np.ndarray:
    """V points uniform on the unit sphere (normalised Gaussian vectors), fp64."""
    p = rng.standard_normal((V, 3))
    return p / np.linalg.norm(p, axis=1, keepdims=True)


def ellipsoid_points(V: int, rng: np.random.Generator,
                     axes: Sequence[float] = (0.3, 0.9, 0.2)) -> np.ndarray:
    """Unit-sphere points scaled per axis (a body-like elongated surface)."""
    return sphere_points(V, rng) * np.asarray(axes, dtype=np.float64)[None, :]


def knn(points: np.ndarray, K: int, block: int = 1024) -> np.ndarray:
    """Exact K nearest neighbours (Euclidean, fp64), self first, ties -> lower index.

    Returns int32 [V][K].  Squared distances are formed from coordinate
    differences (no |a|^2 + |b|^2 - 2ab cancellation) so the order is exact
    for distinct points.
    """
    P = np.ascontiguousarray(points, dtype=np.float64)
    V = P.shape[0]
    if K > V:
        raise ValueError("K > V")
    out = np.empty((V, K), dtype=np.int32)
    idx_all = np.arange(V)
    for s in range(0, V, block):
        e = min(V, s + block)
        d = np.zeros((e - s, V), dtype=np.float64)
        for ax in range(3):
            diff = P[s:e, ax][:, None] - P[None, :, ax]
            d += diff * diff
        take = min(V, K + 1)
        part = np.argpartition(d, take - 1, axis=1)[:, :take]
        pd = np.take_along_axis(d, part, axis=1)
        # lexicographic (distance, index) order inside the candidates
        rows = []
        for r in range(e - s):
            o = np.lexsort((part[r], pd[r]))
            rows.append(part[r][o][:K])
            if take > K:
                # a tie across the cut would make the candidate set ambiguous
                kth = pd[r][o][K - 1]
                nxt = pd[r][o][K]
                if nxt == kth:
                    full = np.lexsort((idx_all, d[r]))
                    rows[-1] = full[:K]
        out[s:e] = np.stack(rows).astype(np.int32)
    return out


# ----------------------------------------------------------------------------
# masks
# ----------------------------------------------------------------------------


def bernoulli_mask(B: int, V: int, p: float, rng: np.random.Generator) -> np.ndarray:
    """uint8 [B][V], each entry 1 with probability p, i.i.d. (Eq. 1 sampling)."""
    if p >= 1.0:
        return np.ones((B, V), dtype=np.uint8)
    if p <= 0.0:
        return np.zeros((B, V), dtype=np.uint8)
    return (rng.random((B, V)) < p).astype(np.uint8)


def cap_mask(points: np.ndarray, B: int, y_below: float, p_noise: float,
             rng: np.random.Generator) -> np.ndarray:
    """Contact-region mask: vertices with y < y_below, OR-ed with Bernoulli noise."""
    V = points.shape[0]
    cap = (points[:, 1] < y_below).astype(np.uint8)[None, :]
    noise = bernoulli_mask(B, V, p_noise, rng)
    return np.maximum(np.broadcast_to(cap, (B, V)), noise).astype(np.uint8)


def markov_mask(n_seq: int, T: int, V: int, density: float, mean_on: float,
                rng: np.random.Generator) -> np.ndarray:
    """Temporally coherent masks: per (sequence, vertex) two-state Markov chain.

    On-runs are geometric with mean ``mean_on`` frames; the off->on rate is
    chosen so the stationary on-probability is ``density``.  The initial state
    is Bernoulli(density).  Returns uint8 [n_seq * T][V] (row = seq * T + t).
    """
    p_off = 1.0 / mean_on
    p_on = density * p_off / (1.0 - density)
    state = rng.random((n_seq, V)) < density
    out = np.empty((n_seq, T, V), dtype=np.uint8)
    for t in range(T):
        out[:, t, :] = state
        u = rng.random((n_seq, V))
        state = np.where(state, u >= p_off, u < p_on)
    return out.reshape(n_seq * T, V)


# ----------------------------------------------------------------------------
# features, weights, bf16 storage
# ----------------------------------------------------------------------------


def features(rows: int, C: int, rng: np.random.Generator) -> np.ndarray:
    return rng.standard_normal((rows, C), dtype=np.float32)


def conv_weights(K: int, Cin: int, Cout: int, rng: np.random.Generator) -> np.ndarray:
    """W[K][Cin][Cout] fp32, std 1/sqrt(K*Cin) (fan-in init over all slots)."""
    return (rng.standard_normal((K, Cin, Cout)) / np.sqrt(K * Cin)).astype(np.float32)


def linear_weights(Cin: int, Cout: int, rng: np.random.Generator) -> np.ndarray:
    return (rng.standard_normal((Cin, Cout)) / np.sqrt(Cin)).astype(np.float32)


def bias_vector(Cout: int, rng: np.random.Generator, scale: float = 0.5) -> np.ndarray:
    return (scale * rng.standard_normal(Cout)).astype(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Storage conversion of inputs to bfloat16 (round-to-nearest-even), as uint16.

    Uses torch's CPU conversion so that this module carries no rounding code of
    its own; the values returned by :func:`as_dtype` are exactly
    representable in both fp32 and bf16, so both sides see identical inputs.
    """
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns (uint16) to fp32 exactly."""
    return (bits.astype(np.uint32) << 16).view(np.float32)


def as_dtype(x: np.ndarray, dtype: str):
    """Return (storage array, exact fp32 values) for dtype 'f32' or 'bf16'."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if dtype == F32:
        return x, x
    if dtype == BF16:
        b = bf16_bits(x)
        return b, bits_to_f32(b)
    raise ValueError(dtype)


def digest(*arrays: np.ndarray) -> str:
    h = hashlib.sha256()
    for a in arrays:
        a = np.ascontiguousarray(a)
        h.update(str(a.dtype).encode())
        h.update(str(a.shape).encode())
        h.update(a.tobytes())
    return h.hexdigest()


# ----------------------------------------------------------------------------
# workloads
# ----------------------------------------------------------------------------


@dataclasses.dataclass
class Layer:
    kind: str                 # "conv" or "linear"
    Cin: int
    Cout: int
    W: np.ndarray             # fp32 values; conv [K][Cin][Cout], linear [Cin][Cout]
    bias: Optional[np.ndarray]  # fp32 [Cout] or None
    relu: bool = True


@dataclasses.dataclass
class Workload:
    name: str
    B: int
    V: int
    K: int
    dtype: str
    points: np.ndarray        # fp64 [V][3]
    nbr: np.ndarray           # int32 [V][K]
    mask: np.ndarray          # uint8 [B][V]
    x: np.ndarray             # fp32 [B*V][C0] (values exactly representable in dtype)
    layers: List[Layer]
    pool: bool = False
    scatter: bool = False
    note: str = ""

    @property
    def C0(self) -> int:
        return self.x.shape[1]

    @property
    def n_active(self) -> int:
        return int(np.count_nonzero(self.mask))


_MESH_CACHE: dict = {}


def mesh(kind: str, V: int, K: int, config: int):
    key = (kind, V, K, config)
    if key not in _MESH_CACHE:
        rng = _rng(config, 0)
        pts = sphere_points(V, rng) if kind == "sphere" else ellipsoid_points(V, rng)
        _MESH_CACHE[key] = (pts, knn(pts, K))
    return _MESH_CACHE[key]


def _round_to(dtype: str, a: np.ndarray) -> np.ndarray:
    return as_dtype(a, dtype)[1]


def _conv_layers(config: int, K: int, chans: Sequence[int], dtype: str,
                 bias: bool = False) -> List[Layer]:
    layers = []
    for l, (ci, co) in enumerate(zip(chans[:-1], chans[1:])):
        rng = _rng(config, 3 + l)
        W = _round_to(dtype, conv_weights(K, ci, co, rng).reshape(-1)).reshape(K, ci, co)
        b = _round_to(F32, bias_vector(co, rng)) if bias else None
        layers.append(Layer("conv", ci, co, W, b, True))
    return layers


def workload_c1() -> Workload:
    """Tiny sparse spiral-conv layer: B=4, V=655 sphere, K=9, fp32 16->64, p=0.10."""
    B, V, K = 4, 655, 9
    pts, nbr = mesh("sphere", V, K, 1)
    m = bernoulli_mask(B, V, 0.10, _rng(1, 1))
    x = features(B * V, 16, _rng(1, 2))
    return Workload("C1 tiny spiral conv (B=4, V=655, K=9, fp32 16->64, p=0.10)",
                    B, V, K, F32, pts, nbr, m, x, _conv_layers(1, K, [16, 64], F32),
                    scatter=True)


def workload_c2() -> Workload:
    """4-layer bf16 encoder 16->64->64->128->128, B=64, V=655, p=0.10, max-pool."""
    B, V, K = 64, 655, 9
    pts, nbr = mesh("sphere", V, K, 2)
    m = bernoulli_mask(B, V, 0.10, _rng(2, 1))
    x = _round_to(BF16, features(B * V, 16, _rng(2, 2)))
    return Workload("C2 4-layer encoder (B=64, V=655, K=9, bf16 16-64-64-128-128, p=0.10)",
                    B, V, K, BF16, pts, nbr, m, x,
                    _conv_layers(2, K, [16, 64, 64, 128, 128], BF16), pool=True)


def workload_c3(dtype: str = F32, five_percent: bool = False) -> Workload:
    """Full-resolution mesh: B=256, V=10475 ellipsoid, K=9, C 64->64.

    Mask = (y < -0.6) OR Bernoulli(0.02).  ``five_percent`` moves the cap
    threshold to y < -0.845, which leaves about 5% of vertices active.
    """
    B, V, K = 256, 10475, 9
    pts, nbr = mesh("ellipsoid", V, K, 3)
    thr = -0.845 if five_percent else -0.6
    m = cap_mask(pts, B, thr, 0.02, _rng(3, 1))
    x = _round_to(dtype, features(B * V, 64, _rng(3, 2)))
    tag = "5%-cap variant" if five_percent else "cap y<-0.6"
    return Workload(f"C3 full mesh (B=256, V=10475, K=9, {dtype} 64->64, {tag})",
                    B, V, K, dtype, pts, nbr, m, x, _conv_layers(3, K, [64, 64], dtype),
                    scatter=True)


def workload_c4(p: float, dtype: str = BF16, B: int = 128, V: int = 10475) -> Workload:
    """Density sweep point: B=128, V=10475 ellipsoid, K=9, C=128 bf16, Bernoulli(p).

    Layers: sparse linear 128->128 + ReLU, then sparse 9-slot conv 128->128 + ReLU;
    the step ends in a zero-fill scatter and a per-body max-pool.
    """
    K, C = 9, 128
    pts, nbr = mesh("ellipsoid", V, K, 4)
    m = bernoulli_mask(B, V, p, _rng(4, 1))
    x = _round_to(dtype, features(B * V, C, _rng(4, 2)))
    rng_l = _rng(4, 3)
    Wl = _round_to(dtype, linear_weights(C, C, rng_l).reshape(-1)).reshape(C, C)
    layers = [Layer("linear", C, C, Wl, None, True)]
    rng_c = _rng(4, 4)
    Wc = _round_to(dtype, conv_weights(K, C, C, rng_c).reshape(-1)).reshape(K, C, C)
    layers.append(Layer("conv", C, C, Wc, None, True))
    return Workload(f"C4 density sweep p={p:g} (B={B}, V={V}, K=9, {dtype} 128->128)",
                    B, V, K, dtype, pts, nbr, m, x, layers, pool=True, scatter=True)


def workload_c5(n_seq: int = 32, T: int = 64) -> Workload:
    """Sequences: 32 x 64 frames, V=655 sphere, K=9, C=256 bf16, Markov masks,
    3 sparse conv layers + per-frame max-pool."""
    V, K, C = 655, 9, 256
    pts, nbr = mesh("sphere", V, K, 5)
    m = markov_mask(n_seq, T, V, 0.10, 8.0, _rng(5, 1))
    B = n_seq * T
    x = _round_to(BF16, features(B * V, C, _rng(5, 2)))
    return Workload(f"C5 sequences ({n_seq}x{T} frames, V=655, K=9, bf16 C=256, Markov runs)",
                    B, V, K, BF16, pts, nbr, m, x, _conv_layers(5, K, [C, C, C, C], BF16),
                    pool=True)
