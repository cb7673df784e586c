"""Gefen oracle: float64 CPU definition of the method, for checking the HIP library.

TEST INFRASTRUCTURE ONLY. Only tests, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py`` may import this package. The product library never loads it.

Thin ctypes wrappers over ``gefen_oracle.c`` (plain C, float64, built with gcc).
Each wrapper cites the paper passage that the C routine follows:

* :func:`divisors`, :func:`partition` -- Sec. 5.1, Alg. 2 (Automatic Block
  Partitioning) and the partition-score equation.
* :func:`histogram_uniform`, :func:`histogram_blocks` -- Alg. 3, histogram of the
  block-absmax-normalised gradients over [-1, 1].
* :func:`dp_codebook` -- Alg. 3 and App. D (exact interval DP with forced +-1 ends).
* :func:`step_uniform`, :func:`step_blocks` -- Alg. 1, one optimizer step.
* :func:`muon_codec_blocks`, :func:`newton_schulz`, :func:`muon_step` -- appendix
  "Gefen-Muon": Muon's momentum held in Gefen's quantized form, then Muon's
  Newton-Schulz orthogonalisation and update. The paper runs the orthogonalisation of
  the official PyTorch Muon, in bfloat16; :func:`newton_schulz` takes the same steps
  with every tensor-valued result rounded to bfloat16 (``bf16=True``), or in float64.

Gradients are numpy ``float32`` arrays, or ``uint16`` arrays holding bf16 bit patterns.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gefen_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

F32 = 0
BF16 = 1


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain C, float64, no contraction, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
               "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build(force=True)
    lib = ctypes.CDLL(_LIB_PATH)
    i64, i32, f64, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_double, ctypes.c_void_p
    lib.oracle_divisors.restype = i64
    lib.oracle_divisors.argtypes = [i64, vp, i64]
    lib.oracle_partition.restype = ctypes.c_int
    lib.oracle_partition.argtypes = [vp, i32, i64, f64, vp, vp, i64, vp, vp]
    lib.oracle_histogram_blocks.restype = None
    lib.oracle_histogram_blocks.argtypes = [vp, i32, vp, i64, i32, vp]
    lib.oracle_histogram_uniform.restype = None
    lib.oracle_histogram_uniform.argtypes = [vp, i32, i64, i64, i32, vp]
    lib.oracle_dp_codebook.restype = ctypes.c_int
    lib.oracle_dp_codebook.argtypes = [vp, i32, i32, vp, vp, vp]
    step_args = [vp, vp, i32, vp, vp, vp]
    lib.oracle_step_blocks.restype = None
    lib.oracle_step_blocks.argtypes = step_args + [vp, i64, vp, vp, i32, f64, f64, f64, f64,
                                                   f64, i64, i32, vp, vp]
    lib.oracle_muon_codec_blocks.restype = None
    lib.oracle_muon_codec_blocks.argtypes = [vp, i32, vp, vp, vp, i64, vp, vp, i32, f64, i32,
                                             vp]
    lib.oracle_step_uniform.restype = None
    lib.oracle_step_uniform.argtypes = step_args + [i64, i64, vp, vp, i32, f64, f64, f64,
                                                    f64, f64, i64, i32, vp, vp]
    _lib = lib
    return lib


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data_as(ctypes.c_void_p)


def _grad(g: np.ndarray):
    if g.dtype == np.float32:
        return np.ascontiguousarray(g), F32
    if g.dtype == np.uint16:
        return np.ascontiguousarray(g), BF16
    raise TypeError("gradients must be float32 or uint16 (bf16 bits)")


def divisors(n: int) -> np.ndarray:
    """Sorted divisors of n (the candidate periods of Alg. 2)."""
    lib = _load()
    cnt = lib.oracle_divisors(int(n), None, 0)
    out = np.zeros(max(cnt, 1), dtype=np.int64)
    lib.oracle_divisors(int(n), _ptr(out), cnt)
    return out[:cnt]


def partition(g: np.ndarray, eps: float = 1e-8):
    """Alg. 2 on one flattened tensor. Returns (divisors, scores S(p), chosen period)."""
    lib = _load()
    g, dt = _grad(g.reshape(-1))
    n = g.size
    cnt = lib.oracle_divisors(n, None, 0)
    divs = np.zeros(cnt, dtype=np.int64)
    scores = np.zeros(cnt, dtype=np.float64)
    nd = ctypes.c_int64(0)
    per = ctypes.c_int64(0)
    rc = lib.oracle_partition(_ptr(g), dt, n, float(eps), _ptr(divs), _ptr(scores), cnt,
                              ctypes.byref(nd), ctypes.byref(per))
    if rc != 0:
        raise RuntimeError("oracle_partition failed")
    return divs, scores, int(per.value)


def histogram_uniform(g: np.ndarray, p: int, nbins: int, hist: np.ndarray | None = None):
    """Alg. 3 histogram of one tensor split into uniform blocks of p elements."""
    lib = _load()
    g, dt = _grad(g.reshape(-1))
    if hist is None:
        hist = np.zeros(nbins, dtype=np.uint64)
    assert hist.dtype == np.uint64 and hist.size == nbins
    assert g.size % p == 0
    lib.oracle_histogram_uniform(_ptr(g), dt, g.size, int(p), int(nbins), _ptr(hist))
    return hist


def histogram_blocks(g: np.ndarray, offsets: np.ndarray, nbins: int,
                     hist: np.ndarray | None = None):
    """Alg. 3 histogram with explicit blocks [offsets[b], offsets[b+1])."""
    lib = _load()
    g, dt = _grad(g.reshape(-1))
    offs = np.ascontiguousarray(offsets, dtype=np.int64)
    if hist is None:
        hist = np.zeros(nbins, dtype=np.uint64)
    lib.oracle_histogram_blocks(_ptr(g), dt, _ptr(offs), offs.size - 1, int(nbins),
                                _ptr(hist))
    return hist


def dp_codebook(hist: np.ndarray, k: int):
    """Alg. 3 / App. D. Returns (codebook float64[k], cost, bounds int32[k], status)."""
    lib = _load()
    hist = np.ascontiguousarray(hist, dtype=np.uint64)
    cb = np.zeros(k, dtype=np.float64)
    bounds = np.zeros(k, dtype=np.int32)
    cost = ctypes.c_double(0.0)
    st = lib.oracle_dp_codebook(_ptr(hist), hist.size, int(k), _ptr(cb), ctypes.byref(cost),
                                _ptr(bounds))
    if st < 0:
        raise ValueError("invalid DP arguments")
    return cb, float(cost.value), bounds, int(st)


def _step_common(theta, codes, s, v, cb_dec, cb_enc, m_full):
    for name, a, dt in (("theta", theta, np.float64), ("s", s, np.float64),
                        ("v", v, np.float64), ("cb_dec", cb_dec, np.float64),
                        ("cb_enc", cb_enc, np.float64)):
        if a.dtype != dt or not a.flags["C_CONTIGUOUS"]:
            raise TypeError(f"{name} must be C-contiguous {dt}")
    if codes is not None and (codes.dtype != np.uint8 or not codes.flags["C_CONTIGUOUS"]):
        raise TypeError("codes must be C-contiguous uint8")
    if m_full is not None and m_full.dtype != np.float64:
        raise TypeError("m_full must be float64")


def step_uniform(theta, g, codes, s, v, p, cb_dec, cb_enc, lr, beta1, beta2, eps, wd, t,
                 quantize=True, m_full=None, m_out=None):
    """Alg. 1 step, uniform blocks of p elements; arrays are updated in place.

    ``m_out`` (float64 array, optional) receives the step's unquantized momentum."""
    lib = _load()
    _step_common(theta, codes, s, v, cb_dec, cb_enc, m_full)
    g, dt = _grad(g.reshape(-1))
    n = theta.size
    assert g.size == n and n % p == 0 and s.size == n // p and v.size == n // p
    if codes is None:
        codes = np.zeros(n, dtype=np.uint8)
    lib.oracle_step_uniform(_ptr(theta), _ptr(g), dt, _ptr(codes), _ptr(s), _ptr(v), n,
                            int(p), _ptr(cb_dec), _ptr(cb_enc), cb_enc.size, float(lr),
                            float(beta1), float(beta2), float(eps), float(wd), int(t),
                            1 if quantize else 0, _ptr(m_full), _ptr(m_out))


def step_blocks(theta, g, codes, s, v, offsets, cb_dec, cb_enc, lr, beta1, beta2, eps, wd,
                t, quantize=True, m_full=None, m_out=None):
    """Alg. 1 step over explicit blocks [offsets[b], offsets[b+1]); in place."""
    lib = _load()
    _step_common(theta, codes, s, v, cb_dec, cb_enc, m_full)
    g, dt = _grad(g.reshape(-1))
    offs = np.ascontiguousarray(offsets, dtype=np.int64)
    nb = offs.size - 1
    assert s.size == nb and v.size == nb and g.size == theta.size
    if codes is None:
        codes = np.zeros(theta.size, dtype=np.uint8)
    lib.oracle_step_blocks(_ptr(theta), _ptr(g), dt, _ptr(codes), _ptr(s), _ptr(v),
                           _ptr(offs), nb, _ptr(cb_dec), _ptr(cb_enc), cb_enc.size,
                           float(lr), float(beta1), float(beta2), float(eps), float(wd),
                           int(t), 1 if quantize else 0, _ptr(m_full), _ptr(m_out))


# ---------------------------------------------------------------------------- Gefen-Muon
MUON_NS_COEFFS = (3.4445, -4.7750, 2.0315)   # Muon's quintic Newton-Schulz coefficients
MUON_NS_STEPS = 5
MUON_EPS = 1e-7


def muon_codec_blocks(g, codes, s, offsets, cb_dec, cb_enc, mu, nesterov=True):
    """Gefen-Muon momentum codec over explicit blocks (the C routine's comment gives
    the equations). Updates codes and s in place; returns u (float64), the matrix that
    Muon orthogonalises."""
    lib = _load()
    g, dt = _grad(np.asarray(g).reshape(-1))
    offs = np.ascontiguousarray(offsets, dtype=np.int64)
    cb_dec = np.ascontiguousarray(cb_dec, dtype=np.float64)
    cb_enc = np.ascontiguousarray(cb_enc, dtype=np.float64)
    assert codes.dtype == np.uint8 and codes.flags.c_contiguous and codes.size == g.size
    assert s.dtype == np.float64 and s.flags.c_contiguous and s.size == offs.size - 1
    u = np.zeros(g.size, dtype=np.float64)
    lib.oracle_muon_codec_blocks(_ptr(g), dt, _ptr(codes), _ptr(s), _ptr(offs), offs.size - 1,
                                 _ptr(cb_dec), _ptr(cb_enc), cb_enc.size, float(mu),
                                 int(bool(nesterov)), _ptr(u))
    return u


def to_bf16(x):
    """Round to bfloat16 as a float32 accumulator is rounded to a bfloat16 result:
    float64 -> float32 -> bfloat16, both round-to-nearest-even. Returns float64."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float64).astype(np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


def ns_normalise(u, rows, cols, eps=MUON_EPS, bf16=True):
    """First stage of Muon's orthogonalisation: the wide orientation of the rows x cols
    matrix (transposed when rows > cols), divided by its Frobenius norm (at least eps).
    With bf16 the input, the norm, eps and the quotient are bfloat16 values."""
    r = to_bf16 if bf16 else (lambda z: np.asarray(z, dtype=np.float64))
    x = r(np.asarray(u, dtype=np.float64).reshape(rows, cols))
    if rows > cols:
        x = x.T
    norm = float(r(np.array([np.sqrt(np.sum(x * x))]))[0])
    return r(x / max(norm, float(r(np.array([eps]))[0])))


def ns_gram(x, bf16=True):
    """A = X X^T, one rounding of the exact product (a float32 accumulator rounded to
    bfloat16 with bf16)."""
    r = to_bf16 if bf16 else (lambda z: np.asarray(z, dtype=np.float64))
    return r(x @ x.T)


def ns_poly(gram, b, c, bf16=True):
    """B = b A + c A A, one rounding of the whole expression (a matrix product whose
    epilogue adds the scaled input before the result is rounded)."""
    r = to_bf16 if bf16 else (lambda z: np.asarray(z, dtype=np.float64))
    return r(b * gram + c * (gram @ gram))


def ns_combine(x, poly, a, bf16=True):
    """X' = a X + B X, one rounding of the whole expression."""
    r = to_bf16 if bf16 else (lambda z: np.asarray(z, dtype=np.float64))
    return r(a * x + poly @ x)


def newton_schulz(u, rows, cols, steps=MUON_NS_STEPS, coeffs=MUON_NS_COEFFS, eps=MUON_EPS,
                  bf16=True):
    """Muon's orthogonalisation of a rows x cols matrix: work on the wide orientation
    (transpose when rows > cols), divide by the Frobenius norm (at least eps), then
    `steps` times X <- a X + (b A + c A^2) X with A = X X^T; transpose back.
    With bf16, the input, the norm and every matrix result are rounded to bfloat16,
    as the implementation the paper uses does (three rounded products per iteration:
    A, then b A + c A A, then a X + B X). Returns a float64 rows x cols array."""
    a, b, c = coeffs
    x = ns_normalise(u, rows, cols, eps, bf16)
    for _ in range(steps):
        x = ns_combine(x, ns_poly(ns_gram(x, bf16), b, c, bf16), a, bf16)
    return np.ascontiguousarray(x.T if rows > cols else x)


def muon_lr_scale(rows, cols):
    """Muon's shape-dependent learning-rate factor, sqrt(max(1, rows / cols))."""
    return float(np.sqrt(max(1.0, rows / cols)))


def muon_step(theta, g, codes, s, offsets, rows, cols, cb_dec, cb_enc, lr, mu, wd,
              nesterov=True, steps=MUON_NS_STEPS, coeffs=MUON_NS_COEFFS, eps=MUON_EPS,
              bf16=True):
    """One Gefen-Muon step of a rows x cols parameter (float64 theta, updated in place):
    codec, orthogonalisation, then theta <- theta (1 - lr wd) - lr sqrt(max(1, rows/cols)) O.
    Returns (u, O)."""
    u = muon_codec_blocks(g, codes, s, offsets, cb_dec, cb_enc, mu, nesterov)
    o = newton_schulz(u, rows, cols, steps, coeffs, eps, bf16).reshape(-1)
    theta *= 1.0 - lr * wd
    theta -= lr * muon_lr_scale(rows, cols) * o
    return u, o
