"""C ABI checks that need no GPU: the library loads, exports every function that
include/gefen.h declares, and rejects bad arguments before touching the device."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gefen.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gefen_[a-z_0-9]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    import paper_2606_13894_amd as gf
    if not os.path.exists(gf.LIB_PATH):
        pytest.skip("libgefen.so is not built (run __graft_entry__.build())")
    return gf.load_library()


def test_header_declares_the_abi():
    names = _declared()
    for must in ("gefen_init", "gefen_step", "gefen_fit_codebook", "gefen_partition_scores",
                 "gefen_histogram", "gefen_dp_codebook", "gefen_destroy", "gefen_last_error"):
        assert must in names


def test_library_exports_every_declared_symbol(lib):
    for name in _declared():
        assert hasattr(lib, name), name


def test_binding_lists_every_declared_symbol():
    import paper_2606_13894_amd as gf
    assert sorted(gf.SYMBOLS) == _declared()


def _tensor(ptr=0x1000, numel=16, dtype=0):
    import paper_2606_13894_amd as gf
    t = (gf.gefen_tensor * 1)()
    t[0].ptr = ptr
    t[0].numel = numel
    t[0].dtype = dtype
    return t


def test_init_argument_errors(lib):
    out = ctypes.c_void_p()
    assert lib.gefen_init(_tensor(), 1, None, None, 0, 8, 1e-8, None, None) == -1
    assert b"out" in lib.gefen_last_error()
    assert lib.gefen_init(_tensor(), 0, None, None, 0, 8, 1e-8, None, ctypes.byref(out)) == -1
    assert lib.gefen_init(None, 1, None, None, 0, 8, 1e-8, None, ctypes.byref(out)) == -1
    assert lib.gefen_init(_tensor(ptr=0), 1, None, None, 0, 8, 1e-8, None,
                          ctypes.byref(out)) == -1
    assert lib.gefen_init(_tensor(numel=0), 1, None, None, 0, 8, 1e-8, None,
                          ctypes.byref(out)) == -1
    assert lib.gefen_init(_tensor(dtype=7), 1, None, None, 0, 8, 1e-8, None,
                          ctypes.byref(out)) == -2
    assert b"dtype" in lib.gefen_last_error()
    assert lib.gefen_init(_tensor(), 1, None, None, 0, 5, 1e-8, None, ctypes.byref(out)) == -1
    assert b"code_bits" in lib.gefen_last_error()
    assert lib.gefen_init(_tensor(), 1, None, None, 0, 8, -1.0, None, ctypes.byref(out)) == -1
    assert out.value is None


def test_step_and_queries_reject_null_state(lib):
    t = _tensor()
    assert lib.gefen_step(None, t, t, 1, 1e-3, 0.9, 0.999, 1e-8, 0.0, 1, None) == -1
    assert b"state" in lib.gefen_last_error()
    assert lib.gefen_step_fit(None, t, t, 1, 1e-3, 0.9, 0.999, 1e-8, 0.0, 1, None) == -1
    assert b"state" in lib.gefen_last_error()
    assert lib.gefen_fit_codebook(None, t, 1, None) == -1
    assert lib.gefen_get_periods(None, None) == -1
    n = ctypes.c_int64()
    assert lib.gefen_checkpoint_bytes(None, ctypes.byref(n)) == -1
    lib.gefen_destroy(None)


def test_dp_argument_errors(lib):
    cb = ctypes.c_void_p(0x1000)
    assert lib.gefen_dp_codebook(cb, 4096, 1, cb, cb, cb, None) == -1      # k < 2
    assert lib.gefen_dp_codebook(cb, 4096, 512, cb, cb, cb, None) == -1    # k > 256
    assert lib.gefen_dp_codebook(cb, 0, 16, cb, cb, cb, None) == -1        # no bins
    assert lib.gefen_dp_codebook(None, 256, 16, cb, cb, cb, None) == -1


def test_binding_refuses_missing_library(monkeypatch, tmp_path):
    import paper_2606_13894_amd as gf
    monkeypatch.setattr(gf, "_lib", None)
    with pytest.raises(ImportError):
        gf.load_library(str(tmp_path / "nope.so"))


def test_workload_shapes_and_counts():
    import workloads as W
    counts = {"tiny": (4, 262_912), "gpt2_125m": (148, 124_439_808),
              "gpt2_1b": (292, 1_313_626_112), "llama3_1p5b": (147, 1_498_482_688),
              "stress_4b": (1, 4_000_000_000)}
    for name, (nt, n) in counts.items():
        w = W.get(name)
        assert (len(w.tensors), w.numel) == (nt, n), name
    # AdamW keeps 8 bytes per parameter: 11.16 GiB for the Llama-3 1.5B shape
    assert abs(8 * W.get("llama3_1p5b").numel / 2**30 - 11.16) < 0.01


def test_stress_block_recipe():
    import workloads as W
    offs = W.stress_block_offsets()
    sizes = np.diff(offs)
    assert offs[0] == 0 and offs[-1] == 4_000_000_000 and sizes.size == 1_000_000
    assert sizes.min() == 64 and sizes.max() <= 65536
    assert abs(sizes.mean() - 4000) < 1e-9
    seq = W.stress_block_offsets(n=10_000_000, variant="sequential")
    s2 = np.diff(seq)
    assert seq[-1] == 10_000_000 and s2[:-1].min() >= 64 and s2.max() <= 65536


def test_stream_mix_argument_errors(lib):
    """The measurement pass checks its arguments before any device call."""
    a16, a8 = 0x10000, 0x10008
    assert lib.gefen_stream_mix(a16, a16, 0, a16, -1, None) == -1
    assert lib.gefen_stream_mix(a16, a16, 9, a16, 16, None) == -2
    assert lib.gefen_stream_mix(None, a16, 0, a16, 16, None) == -1
    assert lib.gefen_stream_mix(a16 + 4, a16, 0, a16, 16, None) == -1      # theta 16 B
    assert lib.gefen_stream_mix(a16, a8, 0, a16, 16, None) == -1           # fp32 grad 16 B
    assert lib.gefen_stream_mix(a16, a16 + 2, 1, a16, 16, None) == -1      # bf16 grad 8 B
    assert lib.gefen_stream_mix(a16, a16, 0, a16 + 1, 16, None) == -1      # codes 4 B
    assert b"aligned" in lib.gefen_last_error()
    assert lib.gefen_stream_mix(None, None, 0, None, 0, None) == 0         # n = 0: no-op


def test_header_is_c99_and_links(lib, tmp_path):
    """include/gefen.h compiles as strict C99 (no C++ in the ABI), every declared function
    resolves when a C program links libgefen.so, and a call that fails its argument
    checks returns GEFEN_EINVAL with a message, without touching the device."""
    import shutil
    import subprocess
    import paper_2606_13894_amd as gf
    cc = shutil.which("gcc")
    if cc is None:
        pytest.skip("no C compiler")
    names = _declared()
    src = tmp_path / "abi.c"
    src.write_text(
        '#include "gefen.h"\n#include <stdio.h>\n'
        "typedef void (*fn)(void);\n"
        "static const fn table[] = {\n"
        + "".join(f"    (fn){n},\n" for n in names)
        + "};\n"
        "int main(void)\n{\n"
        "    gefen_state* st = 0;\n"
        "    int rc = gefen_init(NULL, 1, NULL, NULL, 0, 8, 1e-8, NULL, &st);\n"
        "    const char* msg = gefen_last_error();\n"
        '    printf("%d %d %s\\n", rc, (int)(sizeof table / sizeof table[0]), msg);\n'
        "    return rc == GEFEN_EINVAL && msg && msg[0] && st == 0 ? 0 : 1;\n}\n")
    exe = tmp_path / "abi"
    libdir = os.path.dirname(gf.LIB_PATH)
    subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror",
                    "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe),
                    "-L", libdir, "-lgefen", f"-Wl,-rpath,{libdir}"],
                   check=True, capture_output=True, text=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert out.returncode == 0, out.stdout + out.stderr
    rc, count, _ = out.stdout.split(" ", 2)
    assert int(rc) == -1 and int(count) == len(names)
