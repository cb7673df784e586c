"""Pins for the oracle's histogram and exact DP codebook (Alg. 3, App. D).

The histogram is pinned to numpy's own histogram routine (half-open bins, last bin
closed) and to counting invariants. The DP is pinned to brute-force enumeration of
every contiguous partition, to brute force over every (non-contiguous) assignment
of bins to codebook entries, to closed forms, to symmetry, and to Lloyd-Max.
"""
import itertools

import numpy as np
import pytest


# --------------------------------------------------------------------- histogram
def _np_hist_blocks(g, offs, nbins):
    out = np.zeros(nbins, dtype=np.int64)
    for b in range(len(offs) - 1):
        blk = g[offs[b]:offs[b + 1]].astype(np.float64)
        a = np.abs(blk).max() if blk.size else 0.0
        if a == 0:
            continue
        h, _ = np.histogram(blk / a, bins=nbins, range=(-1.0, 1.0))
        out += h
    return out


@pytest.mark.parametrize("nbins", [64, 256, 4096])
def test_histogram_matches_numpy_on_dyadic_values(oracle, nbins):
    # Dyadic values make every normalised x and every bin edge exact, so numpy's
    # binning and the oracle's must agree bin for bin, including values on edges.
    rng = np.random.default_rng(nbins)
    p = 32
    nblk = 40
    g = (rng.integers(-64, 65, size=p * nblk) / 64.0).astype(np.float32)
    g[:p] = 0.0                     # an all-zero block is skipped
    g[p:2 * p] = 0.5                # a constant block: every x = +1
    offs = np.arange(0, p * nblk + 1, p)
    h = oracle.histogram_uniform(g, p, nbins).astype(np.int64)
    np.testing.assert_array_equal(h, _np_hist_blocks(g, offs, nbins))


def test_histogram_matches_numpy_random_blocks(oracle):
    rng = np.random.default_rng(5)
    sizes = rng.integers(1, 90, size=60)
    offs = np.concatenate([[0], np.cumsum(sizes)])
    g = (rng.standard_t(3, size=offs[-1]) * 1e-3).astype(np.float32)
    h = oracle.histogram_blocks(g, offs, 4096).astype(np.int64)
    ref = _np_hist_blocks(g, offs, 4096)
    # numpy computes bin positions with its own arithmetic; allow only edge ties:
    # any difference must be a single count moved to an adjacent bin.
    diff = h - ref
    assert np.abs(diff).sum() <= 2 * max(1, int(0.001 * offs[-1]))
    np.testing.assert_array_equal(h.sum(), ref.sum())


def test_histogram_counting_invariants(oracle):
    rng = np.random.default_rng(9)
    p, nblk, nbins = 50, 30, 4096
    g = rng.standard_normal(p * nblk).astype(np.float32)
    g[3 * p:4 * p] = 0.0
    h = oracle.histogram_uniform(g, p, nbins)
    nonzero_blocks = nblk - 1
    assert int(h.sum()) == p * nonzero_blocks            # total = sizes of nonzero blocks
    assert int(h[0] + h[-1]) >= nonzero_blocks            # each block's absmax hits an end
    # bf16 input
    bits = (g.view(np.uint32) >> 16).astype(np.uint16)
    hb = oracle.histogram_uniform(bits, p, nbins)
    assert int(hb.sum()) == p * nonzero_blocks


# --------------------------------------------------------------------- DP helpers
def _centres(nbins):
    return -1.0 + (np.arange(nbins) + 0.5) * (2.0 / nbins)


def _sse(c, m, centre):
    return float(np.sum(c * (m - centre) ** 2))


def _interval_cost(c, m, j, k):
    """Direct weighted squared error of one interval for codebook entry j (1-based)."""
    if j == 1:
        return _sse(c, m, -1.0), -1.0
    if j == k:
        return _sse(c, m, 1.0), 1.0
    mu = float(np.sum(c * m) / np.sum(c))
    return _sse(c, m, mu), mu


def _brute_contiguous(c, m, k):
    """Minimum over all ways to cut b bins into k non-empty contiguous intervals."""
    b = len(c)
    best = (np.inf, None, None)
    for cuts in itertools.combinations(range(1, b), k - 1):
        edges = (0,) + cuts + (b,)
        tot, cb = 0.0, []
        for j in range(k):
            e, centre = _interval_cost(c[edges[j]:edges[j + 1]], m[edges[j]:edges[j + 1]],
                                       j + 1, k)
            tot += e
            cb.append(centre)
        if tot < best[0]:
            best = (tot, cb, edges)
    return best


def _brute_assignments(c, m, k):
    """Minimum over every surjective assignment of bins to k entries (any order)."""
    b = len(c)
    best, best_assign = np.inf, None
    for assign in itertools.product(range(k), repeat=b):
        a = np.array(assign)
        if len(set(assign)) < k:
            continue
        tot = 0.0
        for j in range(k):
            sel = a == j
            tot += _interval_cost(c[sel], m[sel], j + 1, k)[0]
        if tot < best:
            best, best_assign = tot, a
    return best, best_assign


def _random_hist(rng, nbins, b):
    hist = np.zeros(nbins, dtype=np.uint64)
    idx = np.sort(rng.choice(nbins, size=b, replace=False))
    hist[idx] = rng.integers(1, 50, size=b).astype(np.uint64)
    return hist


# --------------------------------------------------------------------- DP pins
@pytest.mark.parametrize("seed", range(8))
def test_dp_equals_brute_force_contiguous(oracle, seed):
    rng = np.random.default_rng(seed)
    nbins = 64
    b = int(rng.integers(6, 13))
    k = int(rng.integers(2, min(6, b) + 1))
    hist = _random_hist(rng, nbins, b)
    nz = np.nonzero(hist)[0]
    c = hist[nz].astype(np.float64)
    m = _centres(nbins)[nz]
    cb, cost, bounds, st = oracle.dp_codebook(hist, k)
    assert st == 0
    ref_cost, ref_cb, ref_edges = _brute_contiguous(c, m, k)
    assert cost == pytest.approx(ref_cost, rel=1e-12, abs=1e-15)
    np.testing.assert_allclose(cb, ref_cb, rtol=1e-12, atol=1e-15)
    assert (bounds - 1).tolist() == list(ref_edges[:-1])
    assert np.all(np.diff(cb) > 0)


@pytest.mark.parametrize("seed", range(6))
def test_dp_versus_all_assignments(oracle, seed):
    # The recurrence of App. D ranges over contiguous intervals, one non-empty interval
    # per entry. With both end entries forced to -1 and +1, that set does not contain
    # every assignment: a surjective but non-contiguous assignment can be cheaper (the
    # -1 entry may take a low-count bin to the right of a free entry). So the DP is
    # exact over contiguous partitions (pinned above by enumeration), and the
    # all-assignment minimum is a lower bound. When the all-assignment optimum happens
    # to be contiguous, the two must coincide.
    rng = np.random.default_rng(50 + seed)
    nbins = 32
    b = int(rng.integers(4, 8))
    k = int(rng.integers(2, min(4, b) + 1))
    hist = _random_hist(rng, nbins, b)
    nz = np.nonzero(hist)[0]
    c = hist[nz].astype(np.float64)
    m = _centres(nbins)[nz]
    _, cost, _, _ = oracle.dp_codebook(hist, k)
    best, best_assign = _brute_assignments(c, m, k)
    assert best <= cost * (1 + 1e-12)
    if np.all(np.diff(best_assign) >= 0):
        assert cost == pytest.approx(best, rel=1e-12, abs=1e-15)


@pytest.mark.parametrize("k", [2, 3, 5, 16])
def test_dp_exactly_k_bins_closed_form(oracle, k):
    rng = np.random.default_rng(k)
    nbins = 256
    hist = _random_hist(rng, nbins, k)
    nz = np.nonzero(hist)[0]
    m = _centres(nbins)[nz]
    c = hist[nz].astype(np.float64)
    cb, cost, _, st = oracle.dp_codebook(hist, k)
    assert st == 0
    expect = np.concatenate([[-1.0], m[1:-1], [1.0]])
    np.testing.assert_allclose(cb, expect, rtol=0, atol=1e-15)
    assert cost == pytest.approx(c[0] * (m[0] + 1) ** 2 + c[-1] * (1 - m[-1]) ** 2,
                                 rel=1e-12)


def test_dp_two_entries_is_plus_minus_one(oracle):
    rng = np.random.default_rng(1)
    hist = _random_hist(rng, 128, 20)
    cb, _, _, st = oracle.dp_codebook(hist, 2)
    assert st == 0 and cb.tolist() == [-1.0, 1.0]


def test_dp_symmetric_histogram_gives_symmetric_codebook(oracle):
    rng = np.random.default_rng(4)
    nbins, k = 256, 8
    half = np.zeros(nbins // 2, dtype=np.uint64)
    half[rng.choice(nbins // 2, size=30, replace=False)] = rng.integers(
        1, 1000, size=30).astype(np.uint64)
    hist = np.concatenate([half, half[::-1]])
    cb, _, _, st = oracle.dp_codebook(hist, k)
    assert st == 0
    np.testing.assert_allclose(cb, -cb[::-1], rtol=0, atol=1e-14)


def _lloyd_max(c, m, k, init):
    """Weighted Lloyd-Max on bin centres with the two end entries fixed at -1 and +1."""
    cb = init.copy()
    for _ in range(200):
        assign = np.argmin(np.abs(m[:, None] - cb[None, :]), axis=1)
        new = cb.copy()
        for j in range(1, k - 1):
            sel = assign == j
            if sel.any():
                new[j] = np.sum(c[sel] * m[sel]) / np.sum(c[sel])
        new[0], new[-1] = -1.0, 1.0
        new = np.sort(new)
        if np.allclose(new, cb, rtol=0, atol=1e-15):
            break
        cb = new
    assign = np.argmin(np.abs(m[:, None] - cb[None, :]), axis=1)
    return float(np.sum(c * (m - cb[assign]) ** 2))


@pytest.mark.parametrize("seed", range(4))
def test_dp_cost_not_above_lloyd_max(oracle, seed):
    # App. C.1: the exact DP reaches the lowest quantization error; Lloyd-Max with
    # linear or quantile initialisation can only match or exceed it.
    # The histogram is built as Alg. 3 builds it: every block is normalised by its own
    # absmax, so both end bins hold mass and both forced entries own a bin under
    # nearest assignment (otherwise Lloyd-Max may leave -1 or +1 unused, a solution
    # outside the DP's one-interval-per-entry formulation).
    rng = np.random.default_rng(200 + seed)
    nbins, k = 1024, 16
    x = rng.standard_t(3, size=(2000, 100))
    x = (x / np.abs(x).max(axis=1, keepdims=True)).reshape(-1)
    hist = np.histogram(x, bins=nbins, range=(-1, 1))[0].astype(np.uint64)
    assert hist[0] > 0 and hist[-1] > 0
    nz = np.nonzero(hist)[0]
    c = hist[nz].astype(np.float64)
    m = _centres(nbins)[nz]
    _, cost, _, st = oracle.dp_codebook(hist, k)
    assert st == 0
    lin = np.linspace(-1, 1, k)
    q = np.quantile(np.repeat(m, c.astype(np.int64)), np.linspace(0, 1, k))
    q[0], q[-1] = -1.0, 1.0
    for init in (lin, np.sort(q)):
        assert cost <= _lloyd_max(c, m, k, init) * (1 + 1e-12)


def test_dp_degenerate_fewer_bins_than_entries(oracle):
    hist = np.zeros(64, dtype=np.uint64)
    hist[[10, 20, 40]] = [5, 3, 7]
    cb, cost, _, st = oracle.dp_codebook(hist, 8)
    assert st == 1
    # solved with 3 entries (-1, middle mean, +1), padded with +1
    m = _centres(64)
    assert cb[0] == -1.0 and cb[1] == pytest.approx(m[20]) and np.all(cb[2:] == 1.0)
    assert cost == pytest.approx(5 * (m[10] + 1) ** 2 + 7 * (1 - m[40]) ** 2, rel=1e-12)
    empty = np.zeros(64, dtype=np.uint64)
    cb0, cost0, _, st0 = oracle.dp_codebook(empty, 4)
    assert st0 == 1 and cb0.tolist() == [-1.0, 1.0, 1.0, 1.0] and cost0 == 0.0
