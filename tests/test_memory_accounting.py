"""Optimizer-state memory against the values the paper prints
(tests/golden/optimizer_state_memory.txt, each with its citation).

The library's persistent state is one code per parameter (8-bit: 1 byte; tensors padded
to 32 codes), 8 bytes per block (scale and shared second moment, fp32) and two codebook
slots; AdamW keeps 8 bytes per parameter. This test models that layout on the
workload shapes with one block per row (the period block inference finds on these
shapes for the 2-D weights) and compares it, at the paper's printed precision, with the
paper's figures. The GPU test of the same accounting checks the library's own count
with the periods it infers.
"""
import os

import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "optimizer_state_memory.txt")


def _golden():
    out = {}
    for ln in open(GOLDEN):
        if ln.strip() and not ln.startswith("#"):
            key, val, unit = ln.split()
            out[key] = (float(val), unit)
    return out


def codebook_bytes(k=256):
    guide = (16 * k + 1 + 15) // 16 * 16
    return 2 * (4 * k + 8 * k + 4 * k + guide)


def gefen_persistent_bytes(w, code_bits=8):
    """Codes + per-block fp32 scale and second moment + codebooks, one block per row
    (a 1-D tensor is one row)."""
    codes = sum((t.numel + 31) // 32 * 32 for t in w.tensors) * code_bits // 8
    blocks = sum(t.rows for t in w.tensors)
    return codes + 8 * blocks + codebook_bytes(1 << code_bits)


def test_reduction_per_billion_parameters():
    g = _golden()["reduction_per_billion_params"]
    assert g[1] == "GiB"
    # AdamW 8 bytes, Gefen 1 byte per parameter (+ 8 bytes per block of >= 768 elements)
    lo = (8 - 1 - 8 / 768) * 1e9 / 2**30
    hi = (8 - 1) * 1e9 / 2**30
    assert round(lo, 1) == g[0] and round(hi, 1) == g[0]


def test_adamw_state_of_a_13b_model():
    g = _golden()["adamw_13b_params"]
    assert g[1] == "GiB" and round(13e9 * 8 / 2**30) == g[0]


def test_llama3_state_sizes():
    g = _golden()
    w = W.get("llama3_1p5b")
    adamw = 8 * w.numel
    assert g["llama3_1p5b_adamw"][1] == "GiB"
    assert round(adamw / 2**30, 1) == g["llama3_1p5b_adamw"][0]
    gefen = gefen_persistent_bytes(w)
    printed, unit = g["llama3_1p5b_gefen"]
    assert unit == "GiB"
    # Recorded discrepancy: the paper prints 1.5 GiB, the layout holds 1.40 GiB. The
    # printed figure is the byte count in decimal gigabytes (1.50 GB); no reading of the
    # state (one byte per parameter, 8 bytes per block) reaches 1.5 GiB.
    assert round(gefen / 2**30, 2) == 1.40
    assert round(gefen / 1e9, 1) == printed
    assert round(gefen / 2**30, 1) != printed
    assert 7.9 < adamw / gefen < 8.0


def test_gpt2_125m_footprint_ratios():
    g = _golden()
    w = W.get("gpt2_125m")
    params = 4 * w.numel
    # AdamW: exactly x2.00; the paper prints x2.01 (framework overhead), one unit off
    assert abs(8 * w.numel / params - g["gpt2_125m_adamw_persistent"][0]) <= 0.01 + 1e-12
    assert round(gefen_persistent_bytes(w) / params, 2) == g["gpt2_125m_gefen_persistent"][0]
