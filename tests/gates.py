"""Parity gates of one step, per tensor (or any run of whole blocks of a tensor).

Test infrastructure, numpy only (no torch, no HIP library), so that worker processes
checking a full-size step in parallel can use it. The gates:

* codes: equal, or the oracle's x = m / s' lies within
  delta = 1e-6 * max(1, (beta1*s + (1-beta1)*max|g|) / s') of the decision interval of
  the library's code (for adjacent codes: of their midpoint; a tie decided by fp32
  rounding). The second term widens the window where the block's momentum cancelled to
  well below its inputs; where it cancelled exactly (a zero float64 scale from nonzero
  inputs) every code is a tie;
* scale s': |diff| <= 1e-6 * s' + 1e-6 * (beta1*s + (1-beta1)*max|g|);
* second moment v': relative error <= 4e-6 (fp32 tree sum of up to 2^16 terms);
* parameters: |diff| <= 1e-5 * |theta_ref| + 1e-5 * lr * u_scale, where u_scale is the
  magnitude of the update's operands, (beta1*|c[q]*s| + (1-beta1)*|g|) / (1 - beta1^t)
  / (sqrt(v_hat) + eps) + wd*|theta| >= |u_ref|: relative 1e-5 in fp32, with a floor
  for parameters near zero and for momenta that cancel (the fp32 error of
  m = beta1*c[q]*s + (1-beta1)*g is relative to its summands, not to m).
"""
from __future__ import annotations

import numpy as np


def empty_report():
    return {"code_ties": 0, "codes": 0, "max_rel_theta": 0.0, "max_theta_gate": 0.0,
            "max_rel_v": 0.0}


def merge(rep, part):
    rep["code_ties"] += part["code_ties"]
    rep["codes"] += part["codes"]
    for k in ("max_rel_theta", "max_theta_gate", "max_rel_v"):
        rep[k] = max(rep[k], part[k])
    return rep


def check_tensor(pre_theta, pre_codes, pre_s, post_theta, post_codes, post_s, post_v,
                 ref_theta, ref_codes, ref_s, ref_v, ref_m, g, offs, cb_dec, cb_enc,
                 lr, betas, eps, wd, t, where=""):
    """All arrays float64 except codes (integers); g is the gradient as float64; offs
    are the block offsets of these elements (relative, starting at 0). Returns the
    report; raises AssertionError on a breach."""
    b1 = betas[0]
    rep = empty_report()
    sizes = np.diff(offs)
    g = np.abs(g)
    gmax = np.maximum.reduceat(g, offs[:-1]) if g.size else g
    s_prev = pre_s
    floor = b1 * s_prev + (1 - b1) * gmax
    bad = np.abs(post_s - ref_s) > 1e-6 * ref_s + 1e-6 * floor
    assert not bad.any(), f"{where}: scale mismatch at blocks {np.nonzero(bad)[0][:5]}"
    relv = np.abs(post_v - ref_v) / np.maximum(np.abs(ref_v), 1e-300)
    relv[(ref_v == 0) & (post_v == 0)] = 0.0
    rep["max_rel_v"] = float(relv.max(initial=0.0))
    assert (relv <= 4e-6).all(), f"{where}: v mismatch {relv.max()}"
    # codes
    c_ref, c_gpu = ref_codes.astype(np.int64), post_codes.astype(np.int64)
    diff = c_ref != c_gpu
    rep["codes"] = int(c_ref.size)
    if diff.any():
        idx = np.nonzero(diff)[0]
        blk = np.searchsorted(offs, idx, side="right") - 1
        sr, fl = ref_s[blk], floor[blk]
        # A block whose new scale is 0 in float64 with nonzero inputs has a momentum that
        # cancelled exactly in real arithmetic (e.g. bf16 gradients with g_t = -0.9 g_t-1
        # in a block of one element): both sides then hold rounding noise of either sign,
        # and any code is a tie. A block whose inputs are all zero must match.
        zero = sr == 0
        assert (fl[zero] > 0).all(), f"{where}: code differs in a block of zero inputs"
        nz = ~zero
        j, bj = idx[nz], blk[nz]
        x = ref_m[j] / sr[nz]
        cg = c_gpu[j]
        k = cb_enc.size
        lo = np.where(cg > 0, 0.5 * (cb_enc[np.maximum(cg - 1, 0)] + cb_enc[cg]), -np.inf)
        hi = np.where(cg < k - 1, 0.5 * (cb_enc[cg] + cb_enc[np.minimum(cg + 1, k - 1)]),
                      np.inf)
        # distance from the oracle's x to the decision interval of the library's code
        dist = np.maximum(np.maximum(lo - x, x - hi), 0.0)
        delta = 1e-6 * np.maximum(1.0, fl[nz] / sr[nz])
        ok = dist <= delta
        if not ok.all():
            jj = j[~ok][:4]
            bb = bj[~ok][:4]
            raise AssertionError(
                f"{where}: {int((~ok).sum())} code mismatches of {idx.size} outside the tie "
                f"window; first at elements {jj.tolist()} (blocks {bb.tolist()}, sizes "
                f"{sizes[bb].tolist()}): code pre {pre_codes[jj].tolist()} ref "
                f"{c_ref[jj].tolist()} gpu {c_gpu[jj].tolist()}; x_ref "
                f"{(ref_m[jj] / ref_s[bb]).tolist()}; s pre {pre_s[bb].tolist()} ref "
                f"{ref_s[bb].tolist()} gpu {post_s[bb].tolist()}; |g| {g[jj].tolist()}")
        rep["code_ties"] = int(idx.size)
    # parameters
    elem_blk = np.repeat(np.arange(sizes.size), sizes)
    dq = cb_dec[pre_codes.astype(np.int64)] * s_prev[elem_blk]
    terms = b1 * np.abs(dq) + (1 - b1) * g
    bc1 = 1.0 - b1 ** t
    vhat = ref_v[elem_blk] / (1.0 - betas[1] ** t)
    u_scale = terms / bc1 / (np.sqrt(vhat) + eps) + abs(wd) * np.abs(pre_theta)
    gate = 1e-5 * np.abs(ref_theta) + 1e-5 * abs(lr) * u_scale + 1e-30
    err = np.abs(post_theta - ref_theta)
    ratio = err / gate
    rep["max_theta_gate"] = float(ratio.max(initial=0))
    rel = err / np.maximum(np.abs(ref_theta), 1e-30)
    rep["max_rel_theta"] = float(rel.max(initial=0))
    if not (err <= gate).all():
        j = int(ratio.argmax())
        raise AssertionError(
            f"{where}: theta gate exceeded ({ratio[j]:.3g}x) at element {j}: "
            f"theta_pre={pre_theta[j]:.9g} ref={ref_theta[j]:.9g} gpu={post_theta[j]:.9g} "
            f"m_ref={ref_m[j]:.6g} terms={terms[j]:.6g} u_scale={u_scale[j]:.6g}")
    return rep
