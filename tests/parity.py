"""Teacher-forced parity between the HIP library and the float64 oracle.

Test infrastructure. Before every step the oracle is loaded with the library's state
after the previous step (parameters, codes, scales, second moments, both codebooks,
widened exactly to float64), gets the same gradient bits, and every output of the
step is compared element by element with the gates of tests/gates.py (codes equal up
to ties decided by rounding, scales and second moments to 1e-6 and 4e-6 relative,
parameters to 1e-5 relative with floors for values near zero and cancelled momenta).

Teacher forcing is needed because a legitimate tie flip changes the next momentum by a
codebook gap times the scale, which a free-running comparison would accumulate.
"""
from __future__ import annotations

import numpy as np
import torch

import gates
import oracle
import paper_2606_13894_amd as gf


def grad_bits(g: torch.Tensor) -> np.ndarray:
    """Gradient as the oracle takes it: float32 values or bf16 bit patterns (uint16)."""
    if g.dtype == torch.float32:
        return g.detach().reshape(-1).cpu().numpy()
    if g.dtype == torch.bfloat16:
        return g.detach().reshape(-1).view(torch.int16).cpu().numpy().view(np.uint16)
    raise TypeError(g.dtype)


def unpack_codes(raw: np.ndarray, k: int) -> np.ndarray:
    """Codes by code index from the library's code buffer: one per byte for k = 256,
    two per byte (low nibble = even index) for k = 16."""
    raw = np.asarray(raw, dtype=np.uint8)
    if k == 256:
        return raw
    out = np.empty(2 * raw.size, dtype=np.uint8)
    out[0::2] = raw & 0xF
    out[1::2] = raw >> 4
    return out


def grad_f64(g: torch.Tensor) -> np.ndarray:
    return g.detach().reshape(-1).float().cpu().numpy().astype(np.float64)


class Run:
    """A library state plus the per-tensor block structure, for parity checks."""

    def __init__(self, params, grads0, block_offsets=None, **init_kwargs):
        self.params = list(params)
        self.state = gf.GefenState(grads0, block_offsets=block_offsets, **init_kwargs)
        self.numels = [p.numel() for p in self.params]
        lay = self.state.layout()
        self.code_off = lay["code_offsets"]
        self.blk_idx = lay["block_index"]
        self.k = lay["k"]
        periods = self.state.periods
        self.offsets = []
        if block_offsets is not None:
            bo = np.asarray(block_offsets, dtype=np.int64)
            base = 0
            for n in self.numels:
                sel = bo[(bo >= base) & (bo <= base + n)] - base
                self.offsets.append(np.ascontiguousarray(sel))
                base += n
        else:
            for n, p in zip(self.numels, periods):
                self.offsets.append(np.arange(0, n + 1, p, dtype=np.int64))
        self.periods = periods

    def snapshot(self):
        torch.cuda.synchronize()
        codes = unpack_codes(self.state.read(gf.STATE_CODES).cpu().numpy(), self.k)
        scale = self.state.read(gf.STATE_SCALE).cpu().numpy().astype(np.float64)
        v = self.state.read(gf.STATE_V).cpu().numpy().astype(np.float64)
        snap = {"theta": [], "codes": [], "s": [], "v": [],
                "cb_dec": self.state.read(gf.STATE_CB_DEC).cpu().numpy().astype(np.float64),
                "cb_enc": self.state.read(gf.STATE_CB_ENC).cpu().numpy().astype(np.float64)}
        for i, p in enumerate(self.params):
            n = self.numels[i]
            snap["theta"].append(p.detach().reshape(-1).cpu().numpy().astype(np.float64))
            snap["codes"].append(codes[self.code_off[i]:self.code_off[i] + n].copy())
            snap["s"].append(scale[self.blk_idx[i]:self.blk_idx[i + 1]].copy())
            snap["v"].append(v[self.blk_idx[i]:self.blk_idx[i + 1]].copy())
        return snap

    def step(self, grads, lr, betas, eps, wd, t):
        self.state.step(self.params, grads, lr, betas, eps, wd, t)

    def oracle_step(self, pre, grads, lr, betas, eps, wd, t):
        ref = {"theta": [], "codes": [], "s": [], "v": [], "m": []}
        for i in range(len(self.params)):
            th = pre["theta"][i].copy()
            cq = pre["codes"][i].copy()
            s = pre["s"][i].copy()
            v = pre["v"][i].copy()
            m = np.zeros_like(th)
            oracle.step_blocks(th, grad_bits(grads[i]), cq, s, v, self.offsets[i], pre["cb_dec"],
                               pre["cb_enc"], lr, betas[0], betas[1], eps, wd, t, m_out=m)
            for key, val in (("theta", th), ("codes", cq), ("s", s), ("v", v), ("m", m)):
                ref[key].append(val)
        return ref

    def check(self, pre, post, ref, grads, lr, betas, eps, wd, t, where=""):
        """Apply the gates (tests/gates.py) to every tensor; returns a small report,
        raises AssertionError on a breach."""
        rep = gates.empty_report()
        for i in range(len(self.params)):
            gates.merge(rep, gates.check_tensor(
                pre["theta"][i], pre["codes"][i], pre["s"][i],
                post["theta"][i], post["codes"][i], post["s"][i], post["v"][i],
                ref["theta"][i], ref["codes"][i], ref["s"][i], ref["v"][i], ref["m"][i],
                grad_f64(grads[i]), self.offsets[i], pre["cb_dec"], pre["cb_enc"],
                lr, betas, eps, wd, t, f"{where} tensor {i}"))
        return rep

    def teacher_forced_step(self, grads, lr, betas, eps, wd, t, where=""):
        pre = self.snapshot()
        self.step(grads, lr, betas, eps, wd, t)
        post = self.snapshot()
        ref = self.oracle_step(pre, grads, lr, betas, eps, wd, t)
        return self.check(pre, post, ref, grads, lr, betas, eps, wd, t, where)
