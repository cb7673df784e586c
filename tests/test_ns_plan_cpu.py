"""The Gefen-Muon Newton-Schulz plan (paper_2606_13894_amd/csrc/ns_plan.h) on the host,
built with address and undefined-behaviour sanitizers: for the GPT-2 125M, GPT-2 1B and
Llama-3 1.5B shapes (and the odd shapes of the GPU tests) every product of both
ping-pong parities passes the library's own check, every work item decodes to a distinct
in-range tile, and every operand access the kernel's predicates allow stays inside the
lane buffer behind its pointer (tests/ns_plan_check.cpp)."""
import os
import subprocess

import pytest

import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("nsplan") / "ns_plan_check")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
           "-I", os.path.join(ROOT, "paper_2606_13894_amd", "csrc"),
           os.path.join(HERE, "ns_plan_check.cpp"), "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return exe


def _run(exe, tensors):
    text = f"{len(tensors)}\n" + "".join(f"{r} {n}\n" for r, n in tensors)
    out = subprocess.run([exe], input=text, capture_output=True, text=True, timeout=600,
                         env=dict(os.environ, ASAN_OPTIONS="detect_leaks=1"))
    return out.returncode, out.stdout + out.stderr


@pytest.mark.parametrize("name", ["gpt2_125m", "gpt2_1b", "llama3_1p5b"])
def test_workload_plans_stay_in_bounds(checker, name):
    w = W.get(name)
    rc, out = _run(checker, [(t.rows, t.numel) for t in w.tensors])
    assert rc == 0, out
    assert out.strip().splitlines()[-1].startswith("ok:"), out


@pytest.mark.parametrize("name", ["gpt2_125m", "gpt2_1b", "llama3_1p5b"])
def test_lanes_balance_and_order(checker, name):
    """The lanes: groups whose estimated time is the floor of their launches (latency-bound)
    share lane 2 when some group is longer; the others split over lanes 0 and 1 by
    estimated time (each group to the lane with less so far, longest first: the two differ
    by at most their longest group); every lane runs longest first, and every group is on
    one lane."""
    import re
    w = W.get(name)
    rc, out = _run(checker, [(t.rows, t.numel) for t in w.tensors])
    assert rc == 0, out
    lanes = {0: [], 1: [], 2: []}
    seen = set()
    for line in out.splitlines():
        m = re.match(r"lane (\d) group (\d+): .* floor ([0-9.]+), cost ([0-9.]+)$", line)
        if m:
            lanes[int(m.group(1))].append((float(m.group(4)), float(m.group(3))))
            seen.add(int(m.group(2)))
    n_groups = int(re.search(r"ok: (\d+) groups", out).group(1))
    assert len(seen) == n_groups == sum(len(v) for v in lanes.values())
    long_groups = [c for v in lanes.values() for c, f in v if c > f]
    if long_groups:
        assert all(c <= f for c, f in lanes[2]), lanes[2]
        assert all(c > f for c, f in lanes[0] + lanes[1]), lanes
    else:
        assert not lanes[2]
    for l in (0, 1, 2):
        costs = [c for c, _ in lanes[l]]
        assert costs == sorted(costs, reverse=True), (l, costs)
    c01 = [c for c, _ in lanes[0] + lanes[1]]
    if c01:
        assert abs(sum(c for c, _ in lanes[0]) - sum(c for c, _ in lanes[1])) <= max(c01) + 1e-9


@pytest.mark.parametrize("seed", range(10))
def test_random_shapes_stay_in_bounds(checker, seed):
    """Seeded random models: matrices of random sides (1 to 3000, some repeated so that
    they batch, in both orientations), vectors, tiny and very tall or wide ones; every
    product of every group passes the library's check and stays inside its buffers, and
    the lanes cover every group once."""
    import numpy as np
    rng = np.random.default_rng(500 + seed)
    shapes = []
    for _ in range(int(rng.integers(1, 30))):
        kind = int(rng.integers(6))
        if kind == 0:
            r, c = 1, int(rng.integers(1, 5000))
        elif kind == 1:
            r, c = int(rng.integers(1, 5000)), 1
        elif kind == 2:
            r, c = int(rng.integers(2, 40)), int(rng.integers(2, 40))
        elif kind == 3:
            r, c = int(rng.integers(2, 64)), int(rng.integers(2000, 60000))
        else:
            r, c = int(rng.integers(2, 3000)), int(rng.integers(2, 3000))
        shapes += [(r, c)] * int(rng.integers(1, 4))
        if rng.integers(2):
            shapes.append((c, r))   # the other orientation of the same matrix
    rc, out = _run(checker, [(r, r * c) for r, c in shapes])
    assert rc == 0, out
    assert out.strip().splitlines()[-1].startswith("ok:"), out


def test_odd_shapes_stay_in_bounds(checker):
    shapes = [(64, 192), (192, 64), (128, 128), (1, 300), (300, 1), (3, 5), (64, 4096),
              (5000, 48), (1003, 40), (77, 9), (1003, 40), (130, 129), (1008, 40), (40, 1008),
              (1, 50), (50, 1), (48, 5000), (2, 2), (129, 257), (768, 50257), (2048, 50257)]
    rc, out = _run(checker, [(r, r * c) for r, c in shapes])
    assert rc == 0, out
    assert out.strip().splitlines()[-1].startswith("ok:"), out


def test_a_bad_shape_is_refused(checker):
    rc, out = _run(checker, [(7, 50)])
    assert rc == 1 and "does not divide" in out


def test_rows_beyond_the_buffer_offsets_are_refused(checker):
    """A tile's operand rows are read with 32-bit byte offsets: a 2 x 9,000,000 matrix
    (Gram rows of 9 M elements, 128-row tiles) is refused by the library's own check, with the reason."""
    rc, out = _run(checker, [(2, 2 * 9_000_000)])
    assert rc == 1 and "span 2 GiB" in out, out
