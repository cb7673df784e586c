"""Python binding of libgefen (Gefen optimizer for MI355X / gfx950).

Argument marshalling only: every step of the method runs in the HIP kernels of
``libgefen.so``. PyTorch provides device memory and the current stream. There is no
CPU fallback: importing works without a GPU, but every call needs the HIP library and
a device, and raises otherwise.

Entry points mirror ``include/gefen.h``:

* :class:`GefenState` -- ``gefen_init`` / ``gefen_step`` / ``gefen_fit_codebook`` and
  the state queries, checkpoint export and import.
* :func:`partition_scores` -- ``gefen_partition_scores`` (Alg. 2 on one tensor).
* :func:`dp_codebook` -- ``gefen_dp_codebook`` (Alg. 3 / App. D DP on a histogram).
* :class:`Gefen` -- a ``torch.optim.Optimizer`` front end (AdamW-compatible arguments)
  that initialises the state from the first gradients.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgefen.so")

GEFEN_OK = 0
ERRORS = {-1: "EINVAL", -2: "EDTYPE", -3: "EHIP", -4: "ENOMEM", -5: "EDEGENERATE"}
F32, BF16 = 0, 1

# symbols declared in include/gefen.h
SYMBOLS = [
    "gefen_init", "gefen_step", "gefen_step_fit", "gefen_fit_codebook", "gefen_partition_scores",
    "gefen_histogram", "gefen_dp_codebook", "gefen_get_periods", "gefen_get_layout",
    "gefen_read_state", "gefen_write_state", "gefen_get_fit_info", "gefen_state_bytes",
    "gefen_checkpoint_bytes", "gefen_export", "gefen_import", "gefen_profile_begin",
    "gefen_profile_end", "gefen_destroy", "gefen_last_error", "gefen_muon_init",
    "gefen_muon_step", "gefen_muon_profile_end", "gefen_stream_mix", "gefen_newton_schulz",
    "gefen_dp_codebook_static",
]


class GefenError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


class gefen_tensor(ctypes.Structure):
    _fields_ = [("ptr", ctypes.c_void_p), ("numel", ctypes.c_int64),
                ("dtype", ctypes.c_int32), ("reserved", ctypes.c_int32)]


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libgefen.so (built by ``paper_2606_13894_amd.build``); raise if missing."""
    global _lib
    if _lib is not None:
        return _lib
    # Load PyTorch's HIP runtime first, so that the library binds to the same runtime
    # instance torch uses (a second copy would see no device from torch's context).
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    if not os.path.exists(path):
        raise ImportError(f"libgefen.so not found at {path}; build it with "
                          "`python -m paper_2606_13894_amd.build`")
    lib = ctypes.CDLL(path)
    vp, i32, i64, f32, f64 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                              ctypes.c_float, ctypes.c_double)
    P = ctypes.POINTER
    lib.gefen_init.argtypes = [P(gefen_tensor), i32, vp, vp, i64, i32, f64, vp, P(vp)]
    lib.gefen_step.argtypes = [vp, P(gefen_tensor), P(gefen_tensor), i32, f64, f64, f64, f64,
                               f64, i64, vp]
    lib.gefen_step_fit.argtypes = [vp, P(gefen_tensor), P(gefen_tensor), i32, f64, f64, f64,
                                   f64, f64, i64, vp]
    lib.gefen_fit_codebook.argtypes = [vp, P(gefen_tensor), i32, vp]
    lib.gefen_partition_scores.argtypes = [P(gefen_tensor), f64, vp, vp, i32, P(i32), P(i64), vp]
    lib.gefen_histogram.argtypes = [vp, P(gefen_tensor), i32, vp, vp]
    lib.gefen_dp_codebook.argtypes = [vp, i32, i32, vp, vp, vp, vp]
    lib.gefen_dp_codebook_static.argtypes = [vp, i32, i32, vp, vp, vp, vp]
    lib.gefen_get_periods.argtypes = [vp, vp]
    lib.gefen_get_layout.argtypes = [vp, vp, vp, P(i64), P(i64), P(i32)]
    lib.gefen_read_state.argtypes = [vp, i32, vp, i64, vp]
    lib.gefen_write_state.argtypes = [vp, i32, vp, i64, vp]
    lib.gefen_get_fit_info.argtypes = [vp, P(f64), P(i32), vp]
    lib.gefen_state_bytes.argtypes = [vp, P(i64), P(i64)]
    lib.gefen_checkpoint_bytes.argtypes = [vp, P(i64)]
    lib.gefen_export.argtypes = [vp, vp, i64, vp]
    lib.gefen_import.argtypes = [vp, vp, i64, vp]
    lib.gefen_profile_begin.argtypes = [vp, i32]
    lib.gefen_profile_end.argtypes = [vp, i32, P(i32), vp, vp, vp, vp, vp, vp, vp, vp]
    lib.gefen_muon_init.argtypes = [vp, vp, i32, vp]
    lib.gefen_muon_step.argtypes = [vp, P(gefen_tensor), P(gefen_tensor), i32, f64, f64, f64,
                                    i32, i32, f64, f64, f64, f64, vp]
    lib.gefen_muon_profile_end.argtypes = [vp, P(i32), P(f64), P(f64)]
    lib.gefen_stream_mix.argtypes = [vp, vp, i32, vp, i64, vp]
    lib.gefen_newton_schulz.argtypes = [vp, vp, i32, i64, i64, i32, f64, f64, f64, vp]
    lib.gefen_destroy.argtypes = [vp]
    lib.gefen_destroy.restype = None
    lib.gefen_last_error.argtypes = []
    lib.gefen_last_error.restype = ctypes.c_char_p
    for name in SYMBOLS:
        if name not in ("gefen_destroy", "gefen_last_error"):
            getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _check(rc: int):
    if rc != GEFEN_OK:
        raise GefenError(rc, _lib.gefen_last_error().decode())


def _torch():
    import torch
    return torch


def _stream(stream=None):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _tensors(ts: Sequence, what: str):
    arr = (gefen_tensor * len(ts))()
    for i, t in enumerate(ts):
        if not t.is_cuda:
            raise ValueError(f"{what}[{i}] must be a device tensor")
        if not t.is_contiguous():
            raise ValueError(f"{what}[{i}] must be contiguous")
        arr[i].ptr = t.data_ptr()
        arr[i].numel = t.numel()
        arr[i].dtype = _dtype_code(t)
        arr[i].reserved = 0
    return arr


def _i64_array(vals):
    a = (ctypes.c_int64 * len(vals))()
    for i, v in enumerate(vals):
        a[i] = int(v)
    return a


STATE_CODES, STATE_SCALE, STATE_V, STATE_CB_DEC, STATE_CB_ENC, STATE_CB_DEC64 = range(6)
STATE_MUON_U = 6          # Gefen-Muon bfloat16 momentum matrix (after muon_init)
STATE_HIST = 7            # histogram of the last codebook fit (uint64[16 k])
MUON_NS_COEFFS = (3.4445, -4.7750, 2.0315)


class GefenState:
    """Library-owned Gefen state for a fixed list of tensors (``gefen_init``)."""

    def __init__(self, grads0: Sequence, period_override: Optional[Sequence[int]] = None,
                 block_offsets=None, code_bits: int = 8, eps_part: float = 1e-8,
                 stream=None):
        lib = load_library()
        self._n = len(grads0)
        self._numels = [int(g.numel()) for g in grads0]
        self._dtypes = [g.dtype for g in grads0]
        gt = _tensors(grads0, "grads0")
        po = _i64_array(period_override) if period_override is not None else None
        if block_offsets is not None:
            import numpy as np
            bo_np = np.ascontiguousarray(np.asarray(block_offsets, dtype=np.int64))
            bo = bo_np.ctypes.data_as(ctypes.c_void_p)
            nb = bo_np.size - 1
        else:
            bo, nb, bo_np = None, 0, None
        out = ctypes.c_void_p()
        _check(lib.gefen_init(gt, self._n, po, bo, nb, int(code_bits), float(eps_part),
                              _stream(stream), ctypes.byref(out)))
        self._h = out
        del bo_np

    # --------------------------------------------------------------- lifecycle
    def close(self):
        if getattr(self, "_h", None):
            _lib.gefen_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # --------------------------------------------------------------- the path
    def step(self, params: Sequence, grads: Sequence, lr: float, betas=(0.9, 0.999),
             eps: float = 1e-8, weight_decay: float = 0.0, t: int = 1, stream=None,
             fit: bool = False):
        """One step; with fit=True also the codebook refit on these gradients
        (gefen_step_fit: the same as step followed by fit_codebook(grads))."""
        pt = _tensors(params, "params")
        gt = _tensors(grads, "grads")
        fn = _lib.gefen_step_fit if fit else _lib.gefen_step
        _check(fn(self._h, pt, gt, self._n, float(lr), float(betas[0]), float(betas[1]),
                  float(eps), float(weight_decay), int(t), _stream(stream)))

    def muon_init(self, rows: Sequence[int], stream=None):
        """Prepare Gefen-Muon steps; tensor i is rows[i] x (numel / rows[i])."""
        a = (ctypes.c_int64 * self._n)(*[int(r) for r in rows])
        _check(_lib.gefen_muon_init(self._h, a, self._n, _stream(stream)))

    def muon_step(self, params: Sequence, grads: Sequence, lr: float, momentum: float = 0.95,
                  weight_decay: float = 0.0, nesterov: bool = True, ns_steps: int = 5,
                  ns_coefficients=MUON_NS_COEFFS, ns_eps: float = 1e-7, stream=None):
        pt = _tensors(params, "params")
        gt = _tensors(grads, "grads")
        a, b, c = ns_coefficients
        _check(_lib.gefen_muon_step(self._h, pt, gt, self._n, float(lr), float(momentum),
                                    float(weight_decay), int(bool(nesterov)), int(ns_steps),
                                    float(a), float(b), float(c), float(ns_eps),
                                    _stream(stream)))

    def muon_profile_end(self):
        """Profiled Gefen-Muon steps: {steps, codec_ms, ortho_ms} (sums; ortho_ms is the
        wall time of normalise + Newton-Schulz + update over all lanes)."""
        n = ctypes.c_int32()
        a, b = ctypes.c_double(), ctypes.c_double()
        _check(_lib.gefen_muon_profile_end(self._h, ctypes.byref(n), ctypes.byref(a),
                                           ctypes.byref(b)))
        return {"steps": n.value, "codec_ms": a.value, "ortho_ms": b.value}

    def fit_codebook(self, grads: Sequence, stream=None):
        _check(_lib.gefen_fit_codebook(self._h, _tensors(grads, "grads"), self._n,
                                       _stream(stream)))

    def histogram(self, grads: Sequence, stream=None):
        torch = _torch()
        h = torch.empty(16 * self.k, dtype=torch.int64, device=grads[0].device)
        _check(_lib.gefen_histogram(self._h, _tensors(grads, "grads"), self._n,
                                    ctypes.c_void_p(h.data_ptr()), _stream(stream)))
        return h

    # --------------------------------------------------------------- queries
    @property
    def periods(self):
        a = (ctypes.c_int64 * self._n)()
        _check(_lib.gefen_get_periods(self._h, a))
        return list(a)

    def layout(self):
        co = (ctypes.c_int64 * (self._n + 1))()
        bi = (ctypes.c_int64 * (self._n + 1))()
        cb, nb, k = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int32()
        _check(_lib.gefen_get_layout(self._h, co, bi, ctypes.byref(cb), ctypes.byref(nb),
                                     ctypes.byref(k)))
        return {"code_offsets": list(co), "block_index": list(bi),
                "code_bytes": cb.value, "total_blocks": nb.value, "k": k.value}

    @property
    def k(self) -> int:
        return self.layout()["k"]

    def read(self, which: int, device=None, stream=None):
        """Copy a state array into a new tensor (device tensor by default)."""
        torch = _torch()
        lay = self.layout()
        spec = {STATE_CODES: (torch.uint8, lay["code_bytes"]),
                STATE_SCALE: (torch.float32, lay["total_blocks"]),
                STATE_V: (torch.float32, lay["total_blocks"]),
                STATE_CB_DEC: (torch.float32, lay["k"]),
                STATE_CB_ENC: (torch.float32, lay["k"]),
                STATE_CB_DEC64: (torch.float64, lay["k"]),
                STATE_MUON_U: (torch.int16, lay["code_offsets"][-1]),
                STATE_HIST: (torch.int64, 16 * lay["k"])}[which]
        dev = device if device is not None else torch.device("cuda", torch.cuda.current_device())
        out = torch.empty(spec[1], dtype=spec[0], device=dev)
        nbytes = out.numel() * out.element_size()
        _check(_lib.gefen_read_state(self._h, int(which), ctypes.c_void_p(out.data_ptr()),
                                     nbytes, _stream(stream)))
        return out

    def write(self, which: int, src, stream=None):
        src = src.contiguous()
        nbytes = src.numel() * src.element_size()
        _check(_lib.gefen_write_state(self._h, int(which), ctypes.c_void_p(src.data_ptr()),
                                      nbytes, _stream(stream)))

    def fit_info(self, stream=None):
        c, s = ctypes.c_double(), ctypes.c_int32()
        _check(_lib.gefen_get_fit_info(self._h, ctypes.byref(c), ctypes.byref(s),
                                       _stream(stream)))
        return c.value, s.value

    def state_bytes(self):
        p, w = ctypes.c_int64(), ctypes.c_int64()
        _check(_lib.gefen_state_bytes(self._h, ctypes.byref(p), ctypes.byref(w)))
        return p.value, w.value

    def export(self, device=None, stream=None):
        torch = _torch()
        n = ctypes.c_int64()
        _check(_lib.gefen_checkpoint_bytes(self._h, ctypes.byref(n)))
        dev = device if device is not None else torch.device("cuda", torch.cuda.current_device())
        buf = torch.empty(n.value, dtype=torch.uint8, device=dev)
        _check(_lib.gefen_export(self._h, ctypes.c_void_p(buf.data_ptr()), n.value,
                                 _stream(stream)))
        return buf

    def import_(self, buf, stream=None):
        buf = buf.contiguous()
        _check(_lib.gefen_import(self._h, ctypes.c_void_p(buf.data_ptr()), buf.numel(),
                                 _stream(stream)))


    # --------------------------------------------------------------- measurement
    def profile_begin(self, max_steps: int):
        _check(_lib.gefen_profile_begin(self._h, int(max_steps)))

    def profile_end(self):
        """Per kernel class: kind, vpl, gradient dtype, launches, total ms, elements
        and algorithmic bytes per launch (HIP events on the step's stream)."""
        cap = 64
        n = ctypes.c_int32()
        arrs = [(ctypes.c_int32 * cap)() for _ in range(4)]
        launches = (ctypes.c_int64 * cap)()
        ms = (ctypes.c_double * cap)()
        elems = (ctypes.c_int64 * cap)()
        nbytes = (ctypes.c_int64 * cap)()
        _check(_lib.gefen_profile_end(self._h, cap, ctypes.byref(n), arrs[0], arrs[1], arrs[2],
                                      arrs[3], launches, ms, elems, nbytes))
        names = {0: "uniform_registers", 1: "streamed_block", 2: "lane_per_block",
                 3: "split_block", 4: "small_any"}
        return [{"kind": names[arrs[0][i]], "vpl": arrs[1][i], "threads": arrs[2][i],
                 "grad_dtype": "f32" if arrs[3][i] == F32 else "bf16",
                 "launches": launches[i], "total_ms": ms[i], "elems_per_launch": elems[i],
                 "bytes_per_launch": nbytes[i]} for i in range(n.value)]


def partition_scores(grad, eps_part: float = 1e-8, stream=None):
    """Alg. 2 on one tensor: (divisors, scores, period), computed on the device."""
    lib = load_library()
    import numpy as np
    gt = _tensors([grad], "grad")
    cap = 4096
    divs = np.zeros(cap, dtype=np.int64)
    scores = np.zeros(cap, dtype=np.float64)
    nd, per = ctypes.c_int32(), ctypes.c_int64()
    _check(lib.gefen_partition_scores(gt, float(eps_part), divs.ctypes.data_as(ctypes.c_void_p),
                                      scores.ctypes.data_as(ctypes.c_void_p), cap,
                                      ctypes.byref(nd), ctypes.byref(per), _stream(stream)))
    return divs[:nd.value], scores[:nd.value], per.value


def dp_codebook(hist, k: int, stream=None):
    """Alg. 3 DP on a device histogram (int64/uint64 tensor of NB counts).

    Returns (codebook float64 device tensor [k], cost float, status int)."""
    lib = load_library()
    torch = _torch()
    hist = hist.contiguous()
    cb = torch.empty(k, dtype=torch.float64, device=hist.device)
    cost = torch.empty(1, dtype=torch.float64, device=hist.device)
    st = torch.empty(1, dtype=torch.int32, device=hist.device)
    _check(lib.gefen_dp_codebook(ctypes.c_void_p(hist.data_ptr()), hist.numel(), int(k),
                                 ctypes.c_void_p(cb.data_ptr()), ctypes.c_void_p(cost.data_ptr()),
                                 ctypes.c_void_p(st.data_ptr()), _stream(stream)))
    return cb, float(cost.item()), int(st.item())


def newton_schulz(x, steps: int = 5, coeffs=(3.4445, -4.7750, 2.0315), out=None, stream=None):
    """Muon's Newton-Schulz iterations on the library's matrix-core products: x is a
    bfloat16 device tensor of shape [batch, m, n] (or [m, n]) with m <= n, already
    normalised; returns the result (a new tensor, or `out`)."""
    lib = load_library()
    torch = _torch()
    if x.dtype != torch.bfloat16:
        raise TypeError("x must be bfloat16")
    x = x.contiguous()
    shape = x.shape
    x3 = x.reshape(-1, shape[-2], shape[-1])
    if out is None:
        out = torch.empty_like(x)
    _check(lib.gefen_newton_schulz(ctypes.c_void_p(x3.data_ptr()), ctypes.c_void_p(out.data_ptr()),
                                   x3.shape[0], x3.shape[1], x3.shape[2], int(steps),
                                   float(coeffs[0]), float(coeffs[1]), float(coeffs[2]),
                                   _stream(stream)))
    return out


def dp_codebook_static(hist, k: int, out=None, stream=None):
    """gefen_dp_codebook_static: the DP with the library's fixed workspace (no allocation
    in the library). `out` = (codebook float64 [k], cost float64 [1], status int32 [1])
    device tensors to write, else new ones. Returns the three tensors."""
    lib = load_library()
    torch = _torch()
    hist = hist.contiguous()
    if out is None:
        out = (torch.empty(k, dtype=torch.float64, device=hist.device),
               torch.empty(1, dtype=torch.float64, device=hist.device),
               torch.empty(1, dtype=torch.int32, device=hist.device))
    cb, cost, st = out
    _check(lib.gefen_dp_codebook_static(ctypes.c_void_p(hist.data_ptr()), hist.numel(), int(k),
                                        ctypes.c_void_p(cb.data_ptr()),
                                        ctypes.c_void_p(cost.data_ptr()),
                                        ctypes.c_void_p(st.data_ptr()), _stream(stream)))
    return cb, cost, st


def stream_mix(theta, grad, codes, stream=None):
    """One pass of the step's byte mix (theta fp32 read + write, grad read, one code byte
    read + write per element) with no optimizer arithmetic: the streaming ceiling."""
    lib = load_library()
    torch = _torch()
    n = theta.numel()
    if grad.numel() != n or codes.numel() != n or codes.dtype != torch.uint8:
        raise ValueError("theta, grad and codes must have the same numel; codes uint8")
    gdt = F32 if grad.dtype == torch.float32 else BF16
    _check(lib.gefen_stream_mix(ctypes.c_void_p(theta.data_ptr()),
                                ctypes.c_void_p(grad.data_ptr()), gdt,
                                ctypes.c_void_p(codes.data_ptr()), n, _stream(stream)))


class Gefen:
    """AdamW-compatible front end: ``Gefen(params, lr, betas, eps, weight_decay)``.

    The first ``step()`` initialises the library state from the current gradients
    (block partitioning and codebook fit, Alg. 1) and then applies step t = 1 with the
    same gradients. Parameters must be fp32 device tensors; gradients fp32 or bf16.
    """

    def __init__(self, params, lr: float = 1e-3, betas=(0.9, 0.999), eps: float = 1e-8,
                 weight_decay: float = 1e-2, code_bits: int = 8, eps_part: Optional[float] = None):
        self.params = [p for p in params]
        self.lr, self.betas, self.eps, self.weight_decay = lr, tuple(betas), eps, weight_decay
        self.code_bits = code_bits
        self.eps_part = eps if eps_part is None else eps_part
        self.state: Optional[GefenState] = None
        self.t = 0

    def zero_grad(self, set_to_none: bool = True):
        for p in self.params:
            if p.grad is not None:
                if set_to_none:
                    p.grad = None
                else:
                    p.grad.zero_()

    def step(self):
        grads = [p.grad.contiguous() for p in self.params]
        if self.state is None:
            self.state = GefenState(grads, code_bits=self.code_bits, eps_part=self.eps_part)
        self.t += 1
        self.state.step(self.params, grads, self.lr, self.betas, self.eps, self.weight_decay,
                        self.t)


class GefenMuon:
    """``torch.optim.Muon``-style front end for Gefen-Muon (appendix "Gefen-Muon"):
    ``GefenMuon(params, lr, weight_decay, momentum, nesterov, ns_coefficients, eps,
    ns_steps)`` with Muon's defaults. Parameter i is the matrix shape[0] x (numel /
    shape[0]) (a 1-D parameter is 1 x numel). The first ``step()`` infers the blocks and
    fits the codebook from the current gradients (Alg. 1), then steps with them.
    Parameters must be fp32 device tensors; gradients fp32 or bf16.
    """

    def __init__(self, params, lr: float = 1e-3, weight_decay: float = 0.1,
                 momentum: float = 0.95, nesterov: bool = True,
                 ns_coefficients=MUON_NS_COEFFS, eps: float = 1e-7, ns_steps: int = 5,
                 code_bits: int = 8, eps_part: float = 1e-8):
        self.params = [p for p in params]
        self.lr, self.weight_decay, self.momentum = lr, weight_decay, momentum
        self.nesterov, self.ns_coefficients = nesterov, tuple(ns_coefficients)
        self.eps, self.ns_steps = eps, ns_steps
        self.code_bits, self.eps_part = code_bits, eps_part
        self.state: Optional[GefenState] = None

    def zero_grad(self, set_to_none: bool = True):
        for p in self.params:
            if p.grad is not None:
                if set_to_none:
                    p.grad = None
                else:
                    p.grad.zero_()

    def step(self):
        grads = [p.grad.contiguous() for p in self.params]
        if self.state is None:
            self.state = GefenState(grads, code_bits=self.code_bits, eps_part=self.eps_part)
            self.state.muon_init([p.shape[0] if p.dim() >= 2 else 1 for p in self.params])
        self.state.muon_step(self.params, grads, self.lr, self.momentum, self.weight_decay,
                             self.nesterov, self.ns_steps, self.ns_coefficients, self.eps)
