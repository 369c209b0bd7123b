"""Oracle: fp32 gradient accumulation, the AdamW shard step and the bf16 cast.

Piper keeps one flat gradient buffer per model-state bucket and accumulates
microbatch gradients into it between optimizer steps (Section 4.3.2,
"Memory management"; Section 6.2 contrasts this with a per-backward
reduction). Under ZeRO-1 each data-parallel rank runs the optimizer over its
own shard of the flat buffers (Section 6.2). The paper names no optimizer;
the reading used here is AdamW with decoupled weight decay and bias
correction (Loshchilov & Hutter), over fp32 master parameters, followed by a
round-to-nearest-even cast of the updated parameters to bf16.

These functions are defined in float32: each step below is one separately
rounded IEEE float32 operation (numpy ufuncs on float32 arrays round every
operation and never fuse a multiply into an add).
"""
from __future__ import annotations

import numpy as np

F32 = np.float32


def accumulate(G: np.ndarray, g: np.ndarray) -> np.ndarray:
    """G + g elementwise in float32 (g may hold bf16 values); returns a new array."""
    return (np.asarray(G, F32) + np.asarray(g, F32)).astype(F32)


def adam_scalars(lr, beta1, beta2, eps, weight_decay, step: int):
    """Host-side scalars, computed in float64 from the float32 hyper-parameters
    and rounded once to float32:

      c_wd = 1 - lr*wd, 1-beta1, 1-beta2,
      step_size = lr / (1 - beta1^t), bc2s = sqrt(1 - beta2^t).
    """
    lr, b1, b2, wd = (float(F32(x)) for x in (lr, beta1, beta2, weight_decay))
    t = int(step)
    return dict(
        c_wd=F32(1.0 - lr * wd),
        b1=F32(b1), b2=F32(b2),
        omb1=F32(1.0 - b1), omb2=F32(1.0 - b2),
        step_size=F32(lr / (1.0 - b1 ** t)),
        bc2s=F32(np.sqrt(1.0 - b2 ** t)),
        eps=F32(eps),
    )


def adamw(p, m, v, g, lr, beta1, beta2, eps, weight_decay, step: int):
    """One AdamW step in float32. Returns (p, m, v) as new arrays.

      p   <- p * c_wd
      m   <- b1*m + (1-b1)*g
      v   <- b2*v + (1-b2)*(g*g)
      den <- sqrt(v) / bc2s + eps          (= sqrt(v_hat) + eps)
      p   <- p - step_size * (m / den)     (= p - lr * m_hat / den)
    """
    s = adam_scalars(lr, beta1, beta2, eps, weight_decay, step)
    p = np.asarray(p, F32)
    m = np.asarray(m, F32)
    v = np.asarray(v, F32)
    g = np.asarray(g, F32)
    p = p * s["c_wd"]
    m = s["b1"] * m + s["omb1"] * g
    gg = g * g
    v = s["b2"] * v + s["omb2"] * gg
    den = np.sqrt(v) / s["bc2s"] + s["eps"]
    p = p - s["step_size"] * (m / den)
    return p.astype(F32), m.astype(F32), v.astype(F32)


def bf16_rne_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest, ties to even.

    Adds 0x7FFF plus the lowest kept bit to the 32-bit pattern and keeps the
    upper half; a NaN keeps its sign and upper payload and is made quiet.
    """
    u = np.ascontiguousarray(x, F32).view(np.uint32).astype(np.uint64)
    is_nan = (u & 0x7FFFFFFF) > 0x7F800000
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    quiet = (u >> 16) | 0x0040
    return np.where(is_nan, quiet, rounded).astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float32 values (exact)."""
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(F32)
