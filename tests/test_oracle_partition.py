"""Pins for the oracle's Automatic Block Partitioning (Sec. 5.1, Alg. 2).

Each test checks the oracle against something the paper or mathematics fixes:
printed divisor-count maxima, brute-force divisor lists and scores, and a closed-form
case whose scores and chosen period follow from the score equation by hand.
"""
import itertools
import os

import numpy as np
import pytest


def _golden_tau_maxima():
    path = os.path.join(os.path.dirname(__file__), "golden", "divisor_count_maxima.txt")
    rows = [ln.split() for ln in open(path) if ln.strip() and not ln.startswith("#")]
    return [(int(a), int(b), int(c)) for a, b, c in rows]


def test_divisor_counts_printed_in_paper(oracle):
    # Sec. 5.1 prints the maximum of tau(n) over [0.9e6, 1.1e6] and [0.9e9, 1.1e9]
    # (tests/golden/divisor_count_maxima.txt). The maximisers are 1,081,080 and
    # 931,170,240; the first interval is swept in full below.
    golden = {(lo, hi): m for lo, hi, m in _golden_tau_maxima()}
    assert oracle.divisors(1081080).size == golden[(900_000, 1_100_000)]
    assert oracle.divisors(931170240).size == golden[(900_000_000, 1_100_000_000)]


def test_divisor_count_maximum_over_interval_by_sieve(oracle):
    # The maximum over [0.9e6, 1.1e6] by an independent numpy divisor-count sieve.
    lo, hi = 900_000, 1_100_000
    tau = np.zeros(hi + 1, dtype=np.int32)
    for d in range(1, hi + 1):
        tau[d::d] += 1
    assert int(tau[lo:hi + 1].max()) == dict(((a, b), c) for a, b, c in _golden_tau_maxima())[
        (lo, hi)]
    # spot-check the oracle's count on a few numbers of the interval
    rng = np.random.default_rng(3)
    for n in rng.integers(lo, hi + 1, size=20):
        assert oracle.divisors(int(n)).size == tau[n]


@pytest.mark.parametrize("n", [1, 2, 3, 12, 36, 97, 360, 1024, 5040, 65536, 99991])
def test_divisors_match_brute_force(oracle, n):
    expect = [d for d in range(1, n + 1) if n % d == 0]
    assert oracle.divisors(n).tolist() == expect


def _brute_scores(g, eps):
    """S(p) for every divisor by direct numpy evaluation of block means."""
    z = np.log(g.astype(np.float64) ** 2 + eps)
    n = z.size
    out = []
    for p in [d for d in range(1, n + 1) if n % d == 0]:
        if n // p < 2:
            out.append(0.0)
            continue
        mu = z.reshape(n // p, p).mean(axis=1)
        out.append(float(np.abs(np.diff(mu)).mean()))
    return np.array(out)


@pytest.mark.parametrize("n,seed", [(24, 0), (60, 1), (96, 2), (210, 3), (256, 4)])
def test_scores_match_brute_force(oracle, n, seed):
    rng = np.random.default_rng(seed)
    g = (rng.standard_normal(n) * np.exp(rng.uniform(-4, 0, size=n))).astype(np.float32)
    divs, scores, _ = oracle.partition(g, 1e-8)
    ref = _brute_scores(g, 1e-8)
    np.testing.assert_allclose(scores, ref, rtol=1e-12, atol=1e-14)


def _brute_period(divs, scores):
    """Strict local maxima of S over the sorted divisor list, then argmax (smallest p)."""
    cands = [(scores[i], -divs[i]) for i in range(1, len(divs) - 1)
             if scores[i] > scores[i - 1] and scores[i] > scores[i + 1]]
    if not cands:
        return 1
    return -max(cands)[1]


@pytest.mark.parametrize("seed", range(6))
def test_selection_rule_brute_force(oracle, seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.choice([48, 72, 120, 144, 180, 240]))
    g = (rng.standard_normal(n) * np.exp(rng.uniform(-5, 0, size=n))).astype(np.float32)
    divs, scores, per = oracle.partition(g, 1e-8)
    assert per == _brute_period(divs.tolist(), scores.tolist())


@pytest.mark.parametrize("n", [1, 2, 7, 97, 7919])
def test_prime_and_unit_sizes_give_period_one(oracle, n):
    # Only 1 and n are divisors, and neither is a candidate (1 < p < n fails).
    g = np.random.default_rng(n).standard_normal(n).astype(np.float32)
    assert oracle.partition(g)[2] == 1


def test_constant_gradient_gives_period_one(oracle):
    # Constant g: every block mean is equal, S(p) = 0 for all p, no strict maximum.
    g = np.full(720, 0.25, dtype=np.float32)
    divs, scores, per = oracle.partition(g)
    assert np.all(scores == 0.0)
    assert per == 1


@pytest.mark.parametrize("q,R", [(8, 6), (12, 10), (16, 4), (30, 6), (64, 12)])
def test_alternating_rows_closed_form(oracle, q, R):
    # R rows of q elements; rows alternate between two gradient magnitudes, so z is a
    # in even rows and b in odd rows. By the score equation:
    #   S(q) = |a-b|, S(2q) = 0, S(q/2) = |a-b|(R-1)/(2R-1), S(jq) = |a-b|/j (odd j | R),
    # and q is the unique strict maximum of S, hence the chosen period.
    ga, gb = np.float32(0.5), np.float32(0.003)
    g = np.empty((R, q), dtype=np.float32)
    g[0::2] = ga
    g[1::2] = gb
    eps = 1e-8
    a = np.log(np.float64(ga) ** 2 + eps)
    b = np.log(np.float64(gb) ** 2 + eps)
    d = abs(a - b)
    divs, scores, per = oracle.partition(g.reshape(-1), eps)
    S = dict(zip(divs.tolist(), scores.tolist()))
    assert S[q] == pytest.approx(d, rel=1e-12)
    assert S[2 * q] == pytest.approx(0.0, abs=1e-12)
    if q % 2 == 0:
        assert S[q // 2] == pytest.approx(d * (R - 1) / (2 * R - 1), rel=1e-12)
    for j in range(3, R + 1, 2):
        if R % j == 0:
            assert S[j * q] == pytest.approx(d / j, rel=1e-12)
    assert per == q


def test_bf16_input_widened_exactly(oracle):
    # bf16 bit patterns must give the same result as the equal fp32 values.
    rng = np.random.default_rng(7)
    f = (rng.standard_normal(192) * np.repeat(np.exp(rng.uniform(-6, 0, 12)), 16))
    f32 = f.astype(np.float32)
    bits = (f32.view(np.uint32) >> 16).astype(np.uint16)
    f32_trunc = (bits.astype(np.uint32) << 16).view(np.float32)
    r1 = oracle.partition(bits)
    r2 = oracle.partition(f32_trunc)
    assert r1[2] == r2[2]
    np.testing.assert_array_equal(r1[1], r2[1])


def test_row_structure_detected_on_small_weight(oracle):
    # Per-row log-uniform gradient scales (rows are contiguous) give the row length.
    rng = np.random.default_rng(11)
    rows, cols = 64, 48
    scale = np.exp(rng.uniform(np.log(1e-3), 0.0, size=rows))[:, None]
    g = (rng.standard_normal((rows, cols)) * scale).astype(np.float32)
    assert oracle.partition(g.reshape(-1))[2] == cols


def test_divisor_list_is_sorted_and_complete_for_composites(oracle):
    for n in itertools.chain(range(1, 200), [720720, 1 << 20]):
        d = oracle.divisors(n)
        assert np.all(np.diff(d) > 0)
        assert d[0] == 1 and d[-1] == n
        assert np.all(n % d == 0)
