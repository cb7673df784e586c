"""The Gefen step's tile planner (paper_2606_13894_amd/csrc/tile_plan.h) on the host, built
with address and undefined-behaviour sanitizers (tests/tile_plan_check.cpp).

For the five workloads -- the model shapes under several period assignments (row
length, head groups, single blocks, tiny blocks), both code widths, and the stress
case's 4e9-element tensor with its 1e6 explicit blocks (both readings of its block
sizes) -- plus edge cases (a tensor past 2^31 elements in uniform blocks and as one
huge block, blocks at every class edge), the planner's output passes the library's own
plan check: every block of every tensor exactly once, every tile inside its tensor,
classes that partition the tiles, and each kernel class's limits. The check itself is
shown to refuse planted mistakes."""
import os
import struct
import subprocess

import numpy as np
import pytest

import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)

DT = {"f32": 0, "bf16": 1}


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("tileplan") / "tile_plan_check")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
           "-I", os.path.join(ROOT, "paper_2606_13894_amd", "csrc"),
           os.path.join(HERE, "tile_plan_check.cpp"), "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return exe


def _write(path, numels, periods, dtypes, code_bits, starts=None):
    with open(path, "wb") as f:
        f.write(struct.pack("<iiii", len(numels), code_bits, 1 if starts is not None else 0, 0))
        for n, p, d in zip(numels, periods, dtypes):
            f.write(struct.pack("<qqii", int(n), int(p), int(d), 0))
        if starts is not None:
            for s in starts:
                s = np.ascontiguousarray(s, dtype="<i8")
                f.write(struct.pack("<q", s.size - 1))
                f.write(s.tobytes())


def _run(exe, path, *extra):
    out = subprocess.run([exe, str(path), *map(str, extra)], capture_output=True, text=True,
                         timeout=900, env=dict(os.environ, ASAN_OPTIONS="detect_leaks=1"))
    return out.returncode, out.stdout + out.stderr


def _periods(w, scheme):
    out = []
    for t in w.tensors:
        n = t.numel
        if len(t.shape) == 1:
            out.append({"rows": n, "heads": 1, "whole": n, "fine": 1}[scheme])
            continue
        row = t.shape[1]
        if scheme == "rows":
            out.append(row)
        elif scheme == "heads":
            out.append(t.head_rows * row if t.head_rows else row)
        elif scheme == "whole":
            out.append(n)
        else:   # "fine": 4-element blocks
            out.append(4)
    return out


def _assert_ok(rc, out):
    assert rc == 0, out
    assert out.strip().splitlines()[-1].startswith("ok:"), out


@pytest.mark.parametrize("code_bits", [8, 4])
@pytest.mark.parametrize("name,scheme", [
    ("tiny", "rows"), ("tiny", "heads"), ("tiny", "whole"), ("tiny", "fine"),
    ("gpt2_125m", "rows"), ("gpt2_125m", "heads"), ("gpt2_125m", "whole"),
    ("gpt2_125m", "fine"),
    ("gpt2_1b", "rows"), ("gpt2_1b", "heads"), ("gpt2_1b", "whole"),
    ("llama3_1p5b", "rows"), ("llama3_1p5b", "heads"), ("llama3_1p5b", "whole")])
def test_model_plans(checker, tmp_path, name, scheme, code_bits):
    w = W.get(name)
    path = tmp_path / "plan.bin"
    _write(path, [t.numel for t in w.tensors], _periods(w, scheme),
           [DT[w.grad_dtype]] * len(w.tensors), code_bits)
    _assert_ok(*_run(checker, path))


@pytest.mark.parametrize("code_bits", [8, 4])
@pytest.mark.parametrize("variant", ["rescaled", "sequential"])
def test_stress_plan(checker, tmp_path, variant, code_bits):
    """The 4e9-element tensor (int64 element indices throughout) in its explicit blocks."""
    w = W.get("stress_4b")
    if variant == "rescaled":
        offs = W.stress_block_offsets(w.numel, w.n_blocks)
    else:
        offs = W.stress_block_offsets(w.numel, variant="sequential")
    assert offs[-1] == w.numel > 2 ** 31
    path = tmp_path / "plan.bin"
    _write(path, [w.numel], [0], [DT[w.grad_dtype]], code_bits, starts=[offs])
    rc, out = _run(checker, path)
    _assert_ok(rc, out)
    if code_bits == 8:
        assert "class G" in out


def test_edges_and_huge_tensors(checker, tmp_path):
    """Blocks at every class edge (32/33 one lane or a workgroup, 2042/2043 register run
    or not, 65536/65537 one workgroup or split), a one-element block, and two tensors
    past 2^31 elements: one in 64-element uniform blocks (register class), one a single
    split block."""
    sizes = np.array([1, 3, 32, 33, 2042, 2043, 65536, 65537, 31, 5, 4096, 70000] * 3,
                     dtype=np.int64)
    big = 2 ** 31 + 2 ** 20
    path = tmp_path / "a.bin"
    _write(path, [int(sizes.sum())], [0], [1], 8,
           starts=[np.concatenate([[0], np.cumsum(sizes)])])
    _assert_ok(*_run(checker, path))
    path = tmp_path / "b.bin"
    _write(path, [big, big + 8, 1, 7, 8196 * 3], [64, big + 8, 1, 7, 8196], [1, 1, 0, 0, 1], 8)
    rc, out = _run(checker, path)
    _assert_ok(rc, out)
    assert "class H" in out and "class U" in out


@pytest.mark.parametrize("seed", range(40))
def test_random_tables(checker, tmp_path, seed):
    """Seeded random workloads: several tensors of either gradient type, each with explicit
    blocks drawn from every class's range (1-32, 33-2042, 2043-65536, beyond 65536) or a
    uniform period (divisors of a random size: small, register-held, streamed or split),
    at both code widths; every plan passes the library's check."""
    rng = np.random.default_rng(1000 + seed)
    code_bits = int(rng.choice([8, 4]))
    explicit = bool(rng.integers(2))
    n_t = int(rng.integers(1, 6))
    numels, periods, dts, starts = [], [], [], []
    for _ in range(n_t):
        if explicit:
            ranges = [(1, 33), (33, 2043), (2043, 65537), (65537, 300000)]
            sizes = []
            for _ in range(int(rng.integers(1, 400))):
                lo, hi = ranges[int(rng.choice(4, p=[0.3, 0.4, 0.25, 0.05]))]
                sizes.append(int(rng.integers(lo, hi)))
            offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
            numels.append(int(offs[-1]))
            periods.append(0)
            starts.append(offs)
        else:
            p = int(rng.choice([1, 3, 4, 20, 31, 32, 64, 768, 999, 2048, 8192, 8196, 70000]))
            nb = int(rng.integers(1, 5000 if p < 8192 else 40))
            numels.append(p * nb)
            periods.append(p)
        dts.append(int(rng.integers(2)))
    path = tmp_path / "r.bin"
    _write(path, numels, periods, dts, code_bits, starts=starts if explicit else None)
    _assert_ok(*_run(checker, path))


@pytest.mark.parametrize("corruption", [1, 2, 3, 4, 5])
def test_check_refuses_planted_mistakes(checker, tmp_path, corruption):
    """The plan check is not vacuous: a repeated, shifted or dropped tile, a wrong chunk
    index of a split block and an oversized register run are each refused."""
    sizes = np.array([40, 500, 33, 70000, 100, 1, 2, 3000, 200000, 64] * 4, dtype=np.int64)
    path = tmp_path / "c.bin"
    _write(path, [int(sizes.sum())], [0], [1], 8,
           starts=[np.concatenate([[0], np.cumsum(sizes)])])
    rc, out = _run(checker, path, corruption)
    assert rc == 0 and out.startswith("caught:"), out
