"""Seeded synthetic workloads shaped like the paper's models (inputs only).

This module holds no arithmetic of the optimizer: it only draws parameters and
gradients, so that the HIP library and the float64 oracle receive the same bits.

Gradient structure follows the paper's observation that squared-gradient periodicity
follows the hidden dimension and attention heads (Sec. 5.1, App. E): every weight row
(the contiguous ``in_features`` axis of a ``[out, in]`` PyTorch weight) gets its own
scale drawn log-uniform in [1e-3, 1]; rows or column groups that belong to one
attention head share an extra head scale drawn log-uniform in [1e-2, 1]. A 1-D tensor
is one row. Per step t the gradient is ``g_t = sigma * z_t``, with ``sigma`` fixed for
the run (numpy ``default_rng(seed)``) and ``z_t`` fresh each step from a torch
generator seeded ``1000 * config + t``; ``z`` is standard normal, or Student-t with
3 degrees of freedom for the Llama-3 shape. bf16 gradients are the round-to-nearest-
even bf16 of the fp32 values. Parameters start as N(0, 0.02^2) for 2-D weights, 1 for
norm weights and 0 for biases.

The five configurations (model shapes from the paper's experiments: nanoGPT GPT-2 small,
GPT2-1B, Llama-3 1.5B of TorchTitan; the datasets themselves are not needed, only
tensor shapes and gradient structure):

* ``tiny``    -- [256,512], [512], [512,256], [256]; fp32 grads; 10 steps.
* ``gpt2_125m`` -- GPT-2 small (d 768, 12 layers, 12 heads, MLP 3072, vocab 50257,
  biases, tied head); fp32 grads; 100 steps.
* ``gpt2_1b`` -- same layout with d 2048, 24 layers, 16 heads, MLP 8192; bf16 grads.
* ``llama3_1p5b`` -- Llama-3 (d 2048, 16 layers, 32 q / 8 kv heads of 64, SwiGLU 8192,
  vocab 128256, untied output); bf16 grads, Student-t(3).
* ``stress_4b`` -- one flat tensor of 4e9 elements split into 1e6 explicit blocks
  (log-uniform sizes, rescaled to sum to 4e9); bf16 grads; refit every 10 steps.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Tuple

import numpy as np


@dataclasses.dataclass
class TensorSpec:
    name: str
    shape: Tuple[int, ...]
    kind: str                     # "weight", "norm", "bias", "flat"
    head_rows: int = 0            # rows per head along dim 0 (0: none)
    head_cols: int = 0            # columns per head along dim 1 (0: none)

    @property
    def numel(self) -> int:
        return int(np.prod(self.shape))

    @property
    def rows(self) -> int:
        return self.shape[0] if len(self.shape) == 2 else 1


@dataclasses.dataclass
class Workload:
    name: str
    index: int                    # 1-based configuration number (seeds use it)
    tensors: List[TensorSpec]
    grad_dtype: str               # "f32" or "bf16"
    steps: int
    lr: float
    betas: Tuple[float, float]
    eps: float
    wd: float
    dist: str = "normal"          # "normal" or "student_t3"
    seed: int = 0
    n_blocks: int = 0             # explicit blocks (flat tensor only)
    refit_every: int = 0

    @property
    def numel(self) -> int:
        return sum(t.numel for t in self.tensors)


def _gpt2(d, layers, heads, mlp, vocab=50257, ctx=1024):
    hd = d // heads
    ts = [TensorSpec("wte", (vocab, d), "weight"), TensorSpec("wpe", (ctx, d), "weight")]
    for i in range(layers):
        p = f"h{i}."
        ts += [
            TensorSpec(p + "ln_1.weight", (d,), "norm"),
            TensorSpec(p + "ln_1.bias", (d,), "bias"),
            TensorSpec(p + "attn.c_attn.weight", (3 * d, d), "weight", head_rows=hd),
            TensorSpec(p + "attn.c_attn.bias", (3 * d,), "bias"),
            TensorSpec(p + "attn.c_proj.weight", (d, d), "weight", head_cols=hd),
            TensorSpec(p + "attn.c_proj.bias", (d,), "bias"),
            TensorSpec(p + "ln_2.weight", (d,), "norm"),
            TensorSpec(p + "ln_2.bias", (d,), "bias"),
            TensorSpec(p + "mlp.c_fc.weight", (mlp, d), "weight"),
            TensorSpec(p + "mlp.c_fc.bias", (mlp,), "bias"),
            TensorSpec(p + "mlp.c_proj.weight", (d, mlp), "weight"),
            TensorSpec(p + "mlp.c_proj.bias", (d,), "bias"),
        ]
    ts += [TensorSpec("ln_f.weight", (d,), "norm"), TensorSpec("ln_f.bias", (d,), "bias")]
    return ts


def _llama3(d=2048, layers=16, n_q=32, n_kv=8, hd=64, ffn=8192, vocab=128256):
    ts = [TensorSpec("tok_embeddings", (vocab, d), "weight")]
    for i in range(layers):
        p = f"layers.{i}."
        ts += [
            TensorSpec(p + "attention.wq", (n_q * hd, d), "weight", head_rows=hd),
            TensorSpec(p + "attention.wk", (n_kv * hd, d), "weight", head_rows=hd),
            TensorSpec(p + "attention.wv", (n_kv * hd, d), "weight", head_rows=hd),
            TensorSpec(p + "attention.wo", (d, n_q * hd), "weight", head_cols=hd),
            TensorSpec(p + "feed_forward.w1", (ffn, d), "weight"),
            TensorSpec(p + "feed_forward.w3", (ffn, d), "weight"),
            TensorSpec(p + "feed_forward.w2", (d, ffn), "weight"),
            TensorSpec(p + "attention_norm", (d,), "norm"),
            TensorSpec(p + "ffn_norm", (d,), "norm"),
        ]
    ts += [TensorSpec("norm", (d,), "norm"), TensorSpec("output", (vocab, d), "weight")]
    return ts


def get(name: str) -> Workload:
    if name == "tiny":
        ts = [TensorSpec("fc1.weight", (256, 512), "weight"),
              TensorSpec("fc1.bias", (512,), "bias"),
              TensorSpec("fc2.weight", (512, 256), "weight"),
              TensorSpec("fc2.bias", (256,), "bias")]
        return Workload(name, 1, ts, "f32", 10, 1e-3, (0.9, 0.999), 1e-8, 0.1)
    if name == "gpt2_125m":
        return Workload(name, 2, _gpt2(768, 12, 12, 3072), "f32", 100, 6e-4, (0.9, 0.95),
                        1e-8, 0.1)
    if name == "gpt2_1b":
        return Workload(name, 3, _gpt2(2048, 24, 16, 8192), "bf16", 50, 6e-4, (0.9, 0.95),
                        1e-8, 0.1)
    if name == "llama3_1p5b":
        return Workload(name, 4, _llama3(), "bf16", 50, 1e-4, (0.9, 0.999), 1e-8, 0.0,
                        dist="student_t3")
    if name == "stress_4b":
        return Workload(name, 5, [TensorSpec("flat", (4_000_000_000,), "flat")], "bf16", 30,
                        1e-3, (0.9, 0.999), 1e-8, 0.1, n_blocks=1_000_000, refit_every=10)
    raise KeyError(name)


NAMES = ["tiny", "gpt2_125m", "gpt2_1b", "llama3_1p5b", "stress_4b"]


def _logu(rng, lo, hi, size):
    return np.exp(rng.uniform(math.log(lo), math.log(hi), size=size))


def scale_fields(w: Workload):
    """Per tensor: (row_scale [rows], col_scale [cols] or None), float32.

    sigma[r, c] = row_scale[r] * (col_scale[c] if col_scale is not None else 1).
    Row scales include the head scale of rows that belong to one head.
    """
    rng = np.random.default_rng(w.seed)
    out = []
    for t in w.tensors:
        if t.kind == "flat":
            out.append((None, None))
            continue
        rows = t.rows
        row = _logu(rng, 1e-3, 1.0, rows)
        col = None
        if t.head_rows:
            nh = rows // t.head_rows
            row = row * np.repeat(_logu(rng, 1e-2, 1.0, nh), t.head_rows)
        if t.head_cols:
            nh = t.shape[1] // t.head_cols
            col = np.repeat(_logu(rng, 1e-2, 1.0, nh), t.head_cols).astype(np.float32)
        out.append((row.astype(np.float32), col))
    return out


def stress_block_offsets(n: int = 4_000_000_000, n_blocks: int = 1_000_000,
                         lo: int = 64, hi: int = 65536, seed: int = 0,
                         variant: str = "rescaled") -> np.ndarray:
    """Block offsets (int64, n_blocks+1) of the flat stress tensor.

    ``rescaled``: draw sizes lo * (hi/lo)^u, scale them to sum to n, clamp to >= lo,
    rescale the unclamped rest until no new clamp appears, then round with largest
    remainders so the sizes sum to n exactly. ``sequential``: draw log-uniform sizes
    until n is covered; the last block is cut short.
    """
    rng = np.random.default_rng(seed)
    if variant == "sequential":
        sizes = []
        tot = 0
        while tot < n:
            s = int(lo * (hi / lo) ** rng.uniform())
            s = min(s, n - tot)
            sizes.append(s)
            tot += s
        return np.concatenate([[0], np.cumsum(np.array(sizes, dtype=np.int64))])
    raw = lo * (hi / lo) ** rng.uniform(size=n_blocks)
    x = raw * (n / raw.sum())
    clamped = np.zeros(n_blocks, dtype=bool)
    for _ in range(100):
        new = (x < lo) & ~clamped
        if not new.any():
            break
        clamped |= new
        x[clamped] = lo
        free = ~clamped
        x[free] *= (n - lo * clamped.sum()) / x[free].sum()
    base = np.floor(x).astype(np.int64)
    rem = n - int(base.sum())
    order = np.argsort(-(x - base), kind="stable")
    base[order[:rem]] += 1
    assert int(base.sum()) == n and base.min() >= 1
    return np.concatenate([[0], np.cumsum(base)]).astype(np.int64)


# ----------------------------------------------------------------- torch generation
def _torch():
    import torch
    return torch


def init_params(w: Workload, device, flat: bool = False):
    """Parameters as fp32 tensors on ``device``; with ``flat`` they are views of one
    contiguous buffer (like a flattened-parameter layout), else separate tensors."""
    torch = _torch()
    gen = torch.Generator(device=device)
    gen.manual_seed(7 + 1000 * w.index)
    total = w.numel
    if flat:
        buf = torch.empty(total, dtype=torch.float32, device=device)
    out = []
    off = 0
    for t in w.tensors:
        n = t.numel
        p = buf[off:off + n].view(t.shape) if flat else torch.empty(
            t.shape, dtype=torch.float32, device=device)
        if t.kind in ("weight", "flat"):
            p.normal_(0.0, 0.02, generator=gen)
        elif t.kind == "norm":
            p.fill_(1.0)
        else:
            p.zero_()
        out.append(p)
        off += n
    return out


def _noise(torch, shape, dist, gen, device):
    if dist == "normal":
        return torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
    # Student-t(3) = N / sqrt(chi2_3 / 3), chi2_3 = sum of three squared normals
    z = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
    c = torch.zeros(shape, device=device, dtype=torch.float32)
    for _ in range(3):
        e = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
        c.addcmul_(e, e)
    return z / torch.sqrt(c / 3.0)


def make_grads(w: Workload, fields, t: int, device, out: Optional[list] = None,
               block_scales: Optional[np.ndarray] = None, offsets=None):
    """Gradient tensors for step t (same shapes as the parameters).

    For the flat stress tensor, ``block_scales`` (one per explicit block) and
    ``offsets`` give a per-block scale field.
    """
    torch = _torch()
    gen = torch.Generator(device=device)
    gen.manual_seed(1000 * w.index + t)
    dt = torch.float32 if w.grad_dtype == "f32" else torch.bfloat16
    res = []
    for i, (spec, (row, col)) in enumerate(zip(w.tensors, fields)):
        if spec.kind == "flat":
            g = _flat_grad(torch, w, spec, gen, device, dt, block_scales, offsets)
        else:
            z = _noise(torch, spec.shape, w.dist, gen, device)
            r = torch.from_numpy(row).to(device)
            if z.dim() == 2:
                z.mul_(r[:, None])
                if col is not None:
                    z.mul_(torch.from_numpy(col).to(device)[None, :])
            else:
                z.mul_(r[0])
            g = z.to(dt)
        if out is not None:
            out[i].copy_(g)
            res.append(out[i])
        else:
            res.append(g)
    return res


def _flat_grad(torch, w, spec, gen, device, dt, block_scales, offsets):
    n = spec.numel
    g = torch.empty(n, dtype=dt, device=device)
    chunk = 1 << 28
    # per-element scale from the per-block scale, built chunk by chunk
    scales_t = torch.from_numpy(block_scales.astype(np.float32)).to(device)
    ends_t = torch.from_numpy(np.ascontiguousarray(offsets[1:])).to(device)
    start = 0
    while start < n:
        stop = min(n, start + chunk)
        idx = torch.arange(start, stop, device=device, dtype=torch.int64)
        block_of = torch.searchsorted(ends_t, idx, right=True)
        z = _noise(torch, (stop - start,), w.dist, gen, device)
        z.mul_(scales_t[block_of])
        g[start:stop] = z.to(dt)
        del idx, block_of, z
        start = stop
    return g


def stress_block_scales(n_blocks: int, seed: int = 0) -> np.ndarray:
    rng = np.random.default_rng(seed + 1)
    return _logu(rng, 1e-3, 1.0, n_blocks).astype(np.float32)
