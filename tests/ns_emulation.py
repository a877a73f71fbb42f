"""A CPU model of the GPU kernels' Newton-Schulz arithmetic (test infrastructure, not the oracle).

It stores every matrix in the format the kernels use and accumulates every product in float32,
so the tests can pin tolerances to the arithmetic itself rather than to one GPU run:

- X_0 = bf16(V) unscaled; the first X X^T is scaled by 1/||V||^2 and the first X product by
  1/||V|| in their fp32 epilogues (the prescale of eq. "ns" folded in);
- A = X X^T is stored in fp16 times 2^13; a step's P = a I + b A + c A A in bf16 when it feeds the
  X product (a one-step segment) and in fp16 inside a longer Gram-space segment, whose other
  matrices (T = P A, A <- P T, Q <- P Q) are fp16 and whose final Q is bf16;
- X <- P X (or Q X) is stored in bf16;
- products of two different factors keep their upper triangle and mirror it, as the kernels'
  symmetric tiles do.

Float32 products here run in numpy's own summation order, not the matrix cores', so results agree
with the GPU statistically (error sizes), not bit for bit.  Written from the kernels' documented
formats; it imports neither the oracle nor the HIP library.
"""
from __future__ import annotations

import numpy as np
import torch

GRAM_SCALE = 8192.0  # A and T are stored times 2^13


def bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest even), returned as float32."""
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16).to(torch.float32).numpy()


def f16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to fp16 (nearest even), returned as float32."""
    return np.ascontiguousarray(x, np.float32).astype(np.float16).astype(np.float32)


def mm(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Product of two float32 matrices with float32 accumulation."""
    return np.matmul(a.astype(np.float32), b.astype(np.float32), dtype=np.float32)


def sym_upper(c: np.ndarray) -> np.ndarray:
    """The upper triangle (with the diagonal) of c, mirrored onto the lower one."""
    u = np.triu(c)
    return u + np.triu(c, 1).T


def schedule(s: int, l: int, steps: int, gram_steps: int = 3) -> list:
    """Segments of the K steps for an s x l (wide) matrix: padded sides S, L (multiples of 256); segments
    of `gram_steps` steps when L >= 2 S, else single printed steps."""
    S, L = -(-s // 256) * 256, -(-l // 256) * 256
    n = gram_steps if (gram_steps >= 2 and L >= 2 * S) else 1
    out, left = [], steps
    while left > 0:
        out.append(min(n, left))
        left -= n
    return out


def newton_schulz(v: np.ndarray, a: float, b: float, c: float, segs: list) -> np.ndarray:
    """U for a wide fp32 V (s x l, s <= l) under the schedule `segs` (all ones: the printed step)."""
    v = np.asarray(v, np.float32)
    s = v.shape[0]
    normsq = float(np.sum(v.astype(np.float64) ** 2))
    inv_norm = np.float32(1.0 / np.sqrt(normsq))
    inv_normsq = np.float32(1.0 / normsq)
    x = bf16(v)
    eye = np.eye(s, dtype=np.float32)
    sc = np.float32(GRAM_SCALE)
    ca, cb, cc = np.float32(a), np.float32(b / GRAM_SCALE), np.float32(c / GRAM_SCALE ** 2)
    for si, n in enumerate(segs):
        first = si == 0
        scale = np.float32(sc * inv_normsq) if first else sc
        A = f16(scale * sym_upper(mm(x, x.T)))
        q = None
        for j in range(n):
            out = f16 if n >= 2 else bf16  # P feeds fp16 products inside a longer segment
            P = out(cc * sym_upper(mm(A, A)) + cb * A + ca * eye)
            if j == 0:
                q = P
            else:
                q = (f16 if j + 1 < n else bf16)(sym_upper(mm(P, q)))
            if j + 1 < n:
                T = f16(sym_upper(mm(P, A)))
                A = f16(sym_upper(mm(P, T)))
        xs = mm(q, x)
        x = bf16(xs * inv_norm if first else xs)
    return x


def write_back(w: np.ndarray, u: np.ndarray, scale: np.ndarray, lr: float, rho: float, wd: float,
               rows: bool) -> np.ndarray:
    """The write-back kernel's float32 arithmetic: W <- fma(1 - lr wd, W, -(rho lr) (u s)), with the
    scale vector s per row (rows=True) or per column; returns the float32 result before the final
    rounding to the parameter dtype."""
    decay = np.float32(1.0 - np.float64(np.float32(lr)) * np.float32(wd))
    step = np.float32(np.float64(np.float32(rho)) * np.float32(lr))
    s = scale[:, None] if rows else scale[None, :]
    us = (np.asarray(u, np.float32) * np.asarray(s, np.float32)).astype(np.float32)
    prod = (step * us).astype(np.float32)
    exact = decay.astype(np.float64) * np.asarray(w, np.float64) - prod.astype(np.float64)
    return exact.astype(np.float32)  # one rounding: the fused multiply-add


def momentum(b: np.ndarray, g: np.ndarray, mu: float, nesterov: bool):
    """The momentum kernel's float32 arithmetic: B <- fma(mu, B, G), and the orthogonalized input
    V = fma(mu, B, G) with Nesterov (else V = B). A product of two float32 values is exact in
    float64, so one rounding of the float64 sum models the fused multiply-add (up to the rare
    double rounding). Returns (B, V) in float32."""
    mu32 = np.float64(np.float32(mu))
    b32 = (mu32 * np.asarray(b, np.float32).astype(np.float64) + np.asarray(g, np.float32)).astype(np.float32)
    if not nesterov:
        return b32, b32
    v32 = (mu32 * b32.astype(np.float64) + np.asarray(g, np.float32)).astype(np.float32)
    return b32, v32
