"""The row bound of the DP (Alg. 3, App. D), checked on the CPU against the oracle.

The library's DP evaluates, at level j < k, only the rows r <= b - (k - j): a prefix of
more bins leaves fewer bins than entries still to place, so no path to D[k][b] passes
through it. This test restates the recurrence in plain Python (float64, the oracle's
operations in the oracle's order) with that bound and checks codebook, cost and interval
starts bit for bit against the oracle's full scan, on seeded random histograms: sparse
and dense, peaked and flat, and degenerate ones with fewer non-empty bins than entries.
"""
import math

import numpy as np
import pytest

import oracle


def _bounded_dp(hist, k):
    nbins = hist.size
    w = 2.0 / nbins
    cnt, ctr = [], []
    for i in range(nbins):
        if hist[i]:
            cnt.append(float(hist[i]))
            ctr.append(-1.0 + (i + 0.5) * w)
    b = len(cnt)
    z0, z1, z2 = [0.0], [0.0], [0.0]
    for c, m in zip(cnt, ctr):
        z0.append(z0[-1] + c)
        z1.append(z1[-1] + c * m)
        z2.append(z2[-1] + c * m * m)
    keff = k if b >= k else (b if b >= 2 else 0)
    status = 0 if b >= k else 1
    if keff < 2:
        return None, None, None, status

    def cost(l, r, j):
        s0 = z0[r] - z0[l - 1]
        s1 = z1[r] - z1[l - 1]
        s2 = z2[r] - z2[l - 1]
        if j == 1 or j == keff:
            a = -1.0 if j == 1 else 1.0
            return s2 - 2.0 * a * s1 + a * a * s0
        return s2 - s1 * s1 / s0

    inf = math.inf
    D = [[inf] * (b + 1) for _ in range(keff + 1)]
    split = [[0] * (b + 1) for _ in range(keff + 1)]
    D[0][0] = 0.0
    for j in range(1, keff + 1):
        rmax = b if j == keff else b - (keff - j)   # the row bound
        rmin = b if j == keff else j
        for r in range(rmin, rmax + 1):
            best, arg = inf, 0
            for l in range(j, r + 1):
                cand = D[j - 1][l - 1] + cost(l, r, j)
                if cand < best:
                    best, arg = cand, l
            D[j][r] = best
            split[j][r] = arg
    cb = np.ones(k)
    bounds = np.zeros(k, dtype=np.int32)
    r = b
    for j in range(keff, 0, -1):
        l = split[j][r]
        bounds[j - 1] = l
        if j == 1:
            cb[0] = -1.0
        elif j == keff:
            cb[j - 1] = 1.0
        else:
            cb[j - 1] = (z1[r] - z1[l - 1]) / (z0[r] - z0[l - 1])
        r = l - 1
    return cb, D[keff][b], bounds, status


def _hist(seed):
    rng = np.random.default_rng(900 + seed)
    nbins = int(rng.choice([16, 32, 48, 64]))
    kind = seed % 4
    if kind == 0:      # dense, peaked at the centre
        h = rng.poisson(200.0 * np.exp(-np.linspace(-3, 3, nbins) ** 2), nbins)
    elif kind == 1:    # sparse
        h = rng.integers(0, 50, nbins) * (rng.random(nbins) < 0.4)
    elif kind == 2:    # flat
        h = rng.integers(1, 1000, nbins)
    else:              # very few non-empty bins (often degenerate)
        h = np.zeros(nbins, dtype=np.int64)
        h[rng.choice(nbins, int(rng.integers(1, 6)), replace=False)] = rng.integers(1, 9, 1)[0]
    return np.asarray(h, dtype=np.uint64)


@pytest.mark.parametrize("seed", range(24))
def test_row_bound_gives_the_full_scan_result(seed):
    h = _hist(seed)
    for k in (2, 3, 5, 8):
        cb, cost, bounds, status = oracle.dp_codebook(h, k)
        got = _bounded_dp(h, k)
        assert got[3] == status, (seed, k)
        if got[0] is None:   # fewer than two non-empty bins: no DP runs
            continue
        assert np.array_equal(got[0].view(np.uint64), cb.view(np.uint64)), (seed, k, got[0], cb)
        assert np.float64(got[1]).view(np.uint64) == np.float64(cost).view(np.uint64), (seed, k)
        keff = int(np.count_nonzero(h)) if status else k
        assert np.array_equal(got[2][:keff], bounds[:keff]), (seed, k)
