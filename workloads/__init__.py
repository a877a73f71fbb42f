"""Seeded synthetic inputs for the MeqMuon hidden-weight update.

This module holds no arithmetic of the method: it only draws weights and
gradients.  Both the fp64 oracle (in its tests) and the HIP path (in tests,
``smoke()`` and the benchmark) take their inputs from here, so the two sides
see the same numbers without sharing any code of the update itself.

The paper trains Llama/SmolLM2/Qwen2 models on C4 (Section "Experiments"),
whose data and checkpoints are not available.  The generators below stand in
for them with the same matrix shapes (Table "Model architectures") and with
the row- and column-magnitude imbalance the paper documents for momentum and
gradients (Section "Imbalance patterns", Tables "row-column-imbalance" and
"remaining-momentum-imbalance"):

    G = s_mat * Z * (r c^T)

with Z ~ N(0, 1) fresh every step, r_i, c_j ~ LogNormal(0, sigma) drawn once
per matrix and kept across steps, and a per-matrix magnitude s_mat.  Initial
weights are W0 ~ N(0, 0.02) (0.02 is a standard deviation).  Values destined
for bf16 storage are rounded to nearest-even once, by torch's float32 ->
bfloat16 cast, so every returned float32 array is exactly representable in
the storage dtype.
"""
from __future__ import annotations

import dataclasses
from typing import List, Sequence, Tuple

import numpy as np

__all__ = [
    "MatrixSpec",
    "Workload",
    "workload",
    "WORKLOAD_NAMES",
    "weight_init",
    "grad_at_step",
    "to_storage",
    "device_inputs",
]

# Stream tags for numpy SeedSequence: each (seed, tag, matrix[, step]) names one
# independent stream, so any single matrix can be regenerated on its own.
_TAG_W0 = 0x57
_TAG_STRUCT = 0x5C
_TAG_Z = 0x2A


@dataclasses.dataclass(frozen=True)
class MatrixSpec:
    name: str
    rows: int
    cols: int


@dataclasses.dataclass(frozen=True)
class Workload:
    """A set of hidden-layer weight matrices and how their gradients look."""

    name: str
    seed: int
    matrices: Tuple[MatrixSpec, ...]
    param_dtype: str          # "f32" or "bf16"; gradients use the same dtype
    grad_scale: str           # "fixed" (s_mat = 1e-3) or "lognormal" (LogNormal(-7, 1))
    sigma: float              # row/column log-normal spread
    hot_row_frac: float = 0.0  # fraction of rows multiplied by hot_row_gain
    hot_row_gain: float = 1.0
    steps: int = 1

    @property
    def count(self) -> int:
        return len(self.matrices)

    @property
    def elements(self) -> int:
        return sum(m.rows * m.cols for m in self.matrices)


def _llama_layers(layers: int, d: int, ffn: int, kv: int | None = None) -> Tuple[MatrixSpec, ...]:
    """Hidden 2D weights of a Llama-style block stack, in (q, k, v, o, gate, up, down) order.

    Shapes follow PyTorch's Linear layout: rows = output features.
    """
    kv = d if kv is None else kv
    out: List[MatrixSpec] = []
    for i in range(layers):
        out += [
            MatrixSpec(f"L{i}.q", d, d),
            MatrixSpec(f"L{i}.k", kv, d),
            MatrixSpec(f"L{i}.v", kv, d),
            MatrixSpec(f"L{i}.o", d, d),
            MatrixSpec(f"L{i}.gate", ffn, d),
            MatrixSpec(f"L{i}.up", ffn, d),
            MatrixSpec(f"L{i}.down", d, ffn),
        ]
    return tuple(out)


_WORKLOADS = {
    # One 256x512 fp32 matrix, one step, fixed gradient magnitude 1e-3.
    "single-256x512": Workload("single-256x512", 0, (MatrixSpec("W", 256, 512),), "f32", "fixed", 1.0),
    # Llama-style 130M hidden weights: 12 layers, d=768, ffn=2048 (84 matrices), 10 steps.
    "llama-130m": Workload("llama-130m", 1, _llama_layers(12, 768, 2048), "bf16", "lognormal", 1.0, steps=10),
    # Llama-style 350M hidden weights: 24 layers, d=1024, ffn=2816 (168 matrices).
    "llama-350m": Workload("llama-350m", 2, _llama_layers(24, 1024, 2816), "bf16", "lognormal", 1.0),
    # 1B-shape hidden weights: 16 layers, d=2048, ffn=8192, GQA 32 q heads / 8 kv heads of dim 64.
    "llama-1b": Workload("llama-1b", 3, _llama_layers(16, 2048, 8192, kv=512), "bf16", "lognormal", 1.0),
    # One 7B-shape block (d=4096, ffn=11008) repeated 4 times, extreme imbalance.
    "llama-7b-block-x4": Workload("llama-7b-block-x4", 4, _llama_layers(4, 4096, 11008), "bf16",
                                  "lognormal", 2.0, hot_row_frac=0.01, hot_row_gain=100.0),
    # The paper's own Llama-350M FFN width (2736, not a multiple of 64): correctness variant.
    "llama-350m-ffn2736": Workload("llama-350m-ffn2736", 2, _llama_layers(24, 1024, 2736), "bf16",
                                   "lognormal", 1.0),
}

WORKLOAD_NAMES = tuple(_WORKLOADS)


def workload(name: str) -> Workload:
    return _WORKLOADS[name]


def custom(shapes: Sequence[Tuple[int, int]], param_dtype: str = "bf16", seed: int = 7,
           grad_scale: str = "lognormal", sigma: float = 1.0, hot_row_frac: float = 0.0,
           hot_row_gain: float = 1.0, name: str = "custom") -> Workload:
    """An ad-hoc workload with the same generator (used for odd shapes and edge cases)."""
    mats = tuple(MatrixSpec(f"M{i}", int(r), int(c)) for i, (r, c) in enumerate(shapes))
    return Workload(name, seed, mats, param_dtype, grad_scale, sigma, hot_row_frac, hot_row_gain)


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(k) for k in key])))


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round a float array to the storage dtype; returns float32 values exact in that dtype."""
    x32 = np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "f32":
        return x32
    if dtype != "bf16":
        raise ValueError(dtype)
    import torch

    return torch.from_numpy(x32).to(torch.bfloat16).to(torch.float32).numpy()


def _structure(wl: Workload, idx: int):
    spec = wl.matrices[idx]
    g = _rng(wl.seed, _TAG_STRUCT, idx)
    s_mat = 1e-3 if wl.grad_scale == "fixed" else float(g.lognormal(-7.0, 1.0))
    r = g.lognormal(0.0, wl.sigma, size=spec.rows)
    c = g.lognormal(0.0, wl.sigma, size=spec.cols)
    if wl.hot_row_frac > 0:
        k = int(np.ceil(wl.hot_row_frac * spec.rows))
        hot = g.choice(spec.rows, size=k, replace=False)
        r[hot] *= wl.hot_row_gain
    return s_mat, r, c


def weight_init(wl: Workload, idx: int) -> np.ndarray:
    """W0 ~ N(0, 0.02) rounded to the parameter dtype (float32 array)."""
    spec = wl.matrices[idx]
    w = _rng(wl.seed, _TAG_W0, idx).normal(0.0, 0.02, size=(spec.rows, spec.cols))
    return to_storage(w, wl.param_dtype)


def grad_at_step(wl: Workload, idx: int, step: int) -> np.ndarray:
    """G_t = s_mat * Z_t * (r c^T), rounded to the gradient dtype (float32 array)."""
    spec = wl.matrices[idx]
    s_mat, r, c = _structure(wl, idx)
    z = _rng(wl.seed, _TAG_Z, idx, step).standard_normal(size=(spec.rows, spec.cols))
    g = (s_mat * z) * r[:, None] * c[None, :]
    return to_storage(g, wl.param_dtype)


def device_inputs(wl: Workload, device, seed: int | None = None, which: Sequence[int] | None = None,
                  momenta: bool = False):
    """Same distributions, drawn on the device with torch (for full-size timing runs).

    Returns (params, grads, momenta) lists of torch tensors; momenta are zero
    tensors when ``momenta`` is true, else an empty list.  The
    values differ from the numpy streams (different generator) but follow the same
    recipe; use :func:`weight_init` / :func:`grad_at_step` where exact values matter.
    """
    import torch

    gen = torch.Generator(device=device)
    gen.manual_seed(wl.seed * 1000003 + 12345 if seed is None else seed)
    pdt = torch.float32 if wl.param_dtype == "f32" else torch.bfloat16
    params, grads, moms = [], [], []
    idxs = range(wl.count) if which is None else which
    for idx in idxs:
        spec = wl.matrices[idx]
        w = torch.empty(spec.rows, spec.cols, device=device, dtype=torch.float32)
        w.normal_(0.0, 0.02, generator=gen)
        s_mat = 1e-3 if wl.grad_scale == "fixed" else float(
            torch.empty(1, device=device).log_normal_(-7.0, 1.0, generator=gen).item())
        r = torch.empty(spec.rows, 1, device=device).log_normal_(0.0, wl.sigma, generator=gen)
        c = torch.empty(1, spec.cols, device=device).log_normal_(0.0, wl.sigma, generator=gen)
        if wl.hot_row_frac > 0:
            k = int(np.ceil(wl.hot_row_frac * spec.rows))
            hot = torch.randperm(spec.rows, device=device, generator=gen)[:k]
            r[hot] *= wl.hot_row_gain
        g = torch.empty(spec.rows, spec.cols, device=device, dtype=torch.float32)
        g.normal_(0.0, 1.0, generator=gen)
        g.mul_(r).mul_(c).mul_(s_mat)
        params.append(w.to(pdt).contiguous())
        grads.append(g.to(pdt).contiguous())
        if momenta:
            moms.append(torch.zeros(spec.rows, spec.cols, device=device, dtype=torch.float32))
        del w, g
    return params, grads, moms
