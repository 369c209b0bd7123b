"""Helpers shared by the GPU tests: device transfers and error metrics."""
import sys

import numpy as np
import torch

from oracle import optim as OP

DEV = "cuda"


def banner(msg):
    """Names the case before a GPU step, so an abort still identifies it."""
    print(f"[gpu case] {msg}", flush=True)
    sys.stdout.flush()


def f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(DEV)


def bf16(a):
    """float32 array of bf16-representable values -> bf16 device tensor (exact)."""
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16).to(DEV)


def dev(a, is_bf16):
    return bf16(a) if is_bf16 else f32(a)


def host(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def bits32(t):
    return t.detach().cpu().view(torch.int32).numpy().view(np.uint32)


def bits16(t):
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


def rel_err(got, ref):
    """max |got - ref| / max |ref| (normwise infinity error)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.max(np.abs(ref))
    return float(np.max(np.abs(got - ref)) / (den if den > 0 else 1.0))


def ints(rng, shape, lo=-8, hi=8):
    return rng.integers(lo, hi + 1, size=shape).astype(np.float32)


def bf16_round(a):
    return OP.bf16_to_f32(OP.bf16_rne_bits(np.asarray(a, np.float32)))
