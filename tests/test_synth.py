"""Seeded input generators: determinism, k-NN properties, mask statistics."""
import numpy as np
import pytest

from paper_2608_09388_amd import synth


def test_generators_are_deterministic():
    a = synth.workload_c1()
    b = synth.workload_c1()
    assert synth.digest(a.nbr, a.mask, a.x, a.layers[0].W) == \
        synth.digest(b.nbr, b.mask, b.x, b.layers[0].W)
    # different configs draw different streams
    c = synth.workload_c2()
    assert synth.digest(a.mask) != synth.digest(c.mask[:4])


@pytest.mark.parametrize("kind,V", [("sphere", 655), ("ellipsoid", 2000)])
def test_knn_self_first_sorted_exact(kind, V):
    rng = np.random.default_rng(11)
    pts = synth.sphere_points(V, rng) if kind == "sphere" else synth.ellipsoid_points(V, rng)
    nbr = synth.knn(pts, 9, block=333)
    assert nbr.dtype == np.int32 and nbr.shape == (V, 9)
    assert np.array_equal(nbr[:, 0], np.arange(V))
    d = np.linalg.norm(pts[nbr] - pts[:, None, :], axis=2)
    assert np.all(np.diff(d, axis=1) >= 0)
    # brute force on a few rows: the 9 listed are the 9 closest
    for v in np.random.default_rng(1).integers(0, V, 20):
        full = np.linalg.norm(pts - pts[v], axis=1)
        order = np.lexsort((np.arange(V), full))
        assert np.array_equal(order[:9], nbr[v])


def test_knn_ties_go_to_lower_index():
    pts = np.array([[0, 0, 0], [1, 0, 0], [-1, 0, 0], [0, 1, 0], [0, 0, 2]], float)
    nbr = synth.knn(pts, 3)
    assert nbr[0].tolist() == [0, 1, 2]


def test_bernoulli_density_within_4_sigma():
    rng = np.random.default_rng(2)
    for p in (0.01, 0.05, 0.1, 0.5):
        m = synth.bernoulli_mask(64, 10475, p, rng)
        n = m.size
        assert abs(m.mean() - p) < 4 * np.sqrt(p * (1 - p) / n)
    assert synth.bernoulli_mask(3, 5, 1.0, rng).all()
    assert not synth.bernoulli_mask(3, 5, 0.0, rng).any()


def test_markov_mask_density_and_run_length():
    rng = np.random.default_rng(3)
    m = synth.markov_mask(64, 128, 400, 0.10, 8.0, rng)
    assert abs(m.mean() - 0.10) < 0.01
    seq = m.reshape(64, 128, 400).transpose(0, 2, 1).reshape(-1, 128).astype(np.int8)
    # mean length of on-runs that start and end inside the window
    d = np.diff(seq, axis=1)
    starts = np.argwhere(d == 1)
    ends = np.argwhere(d == -1)
    lengths = []
    ends_by_row = {}
    for r, c in ends:
        ends_by_row.setdefault(r, []).append(c)
    for r, c in starts:
        later = [e for e in ends_by_row.get(r, []) if e > c]
        if later:
            lengths.append(later[0] - c)
    assert abs(np.mean(lengths) - 8.0) < 0.5


def test_bf16_inputs_are_exact_in_both_dtypes():
    x = np.random.default_rng(4).standard_normal(1000).astype(np.float32)
    bits, vals = synth.as_dtype(x, synth.BF16)
    assert bits.dtype == np.uint16
    assert np.array_equal(synth.as_dtype(vals, synth.BF16)[0], bits)
    assert np.max(np.abs(vals - x) / np.abs(x)) <= 2.0 ** -8


def test_c3_realised_density_and_five_percent_variant():
    w = synth.workload_c3()
    assert 0.12 < w.mask.mean() < 0.22
    w5 = synth.workload_c3(five_percent=True)
    assert 0.04 < w5.mask.mean() < 0.06
