"""Pins for the optimizer oracle (oracle/optim.py):

* AdamW closed forms (first step, zero gradient with decay, beta = 0)
* several steps against a float64 textbook AdamW written in the m_hat/v_hat
  form (not the oracle's op sequence)
* the bf16 cast against torch's float->bfloat16 conversion (a library
  routine) on every bf16 value times a set of rounding-sensitive low halves
* accumulation: integer-valued sums are exact and follow the given order
"""
import numpy as np
import pytest
import torch

from oracle import optim as OP

F32 = np.float32


def ulp(x):
    return np.spacing(np.abs(np.asarray(x, F32))).astype(np.float64)


def test_first_step_closed_form():
    rng = np.random.default_rng(0)
    n = 100_000
    p = rng.standard_normal(n).astype(F32) * F32(0.02)
    g = rng.standard_normal(n).astype(F32) * F32(1e-3)
    z = np.zeros(n, F32)
    lr, eps = 1e-3, 1e-8
    p1, m1, v1 = OP.adamw(p, z, z, g, lr, 0.9, 0.999, eps, 0.0, 1)
    exact = p.astype(np.float64) - float(F32(lr)) * g / (np.abs(g.astype(np.float64)) + float(F32(eps)))
    assert np.all(np.abs(p1 - exact) <= 4 * ulp(exact) + 4 * ulp(F32(lr)))
    # beta1 = beta2 = 0 reduces to the same closed form at any step
    p2, _, _ = OP.adamw(p, z, z, g, lr, 0.0, 0.0, eps, 0.0, 5)
    assert np.all(np.abs(p2 - exact) <= 4 * ulp(exact) + 4 * ulp(F32(lr)))


def test_zero_gradient_is_pure_decay_with_one_rounding():
    rng = np.random.default_rng(1)
    p = rng.standard_normal(10_000).astype(F32)
    z = np.zeros_like(p)
    lr, wd = 3e-4, 0.1
    p1, m1, v1 = OP.adamw(p, z, z, z, lr, 0.9, 0.95, 1e-8, wd, 1)
    factor = F32(1.0 - float(F32(lr)) * float(F32(wd)))
    # the float64 product of two float32 values is exact; one rounding to float32
    expect = (p.astype(np.float64) * np.float64(factor)).astype(F32)
    assert np.array_equal(p1, expect)
    assert np.all(m1 == 0) and np.all(v1 == 0)


def textbook_adamw(p, m, v, g, lr, b1, b2, eps, wd, t):
    p, m, v, g = (np.asarray(a, np.float64) for a in (p, m, v, g))
    m = b1 * m + (1 - b1) * g
    v = b2 * v + (1 - b2) * g * g
    mhat = m / (1 - b1 ** t)
    vhat = v / (1 - b2 ** t)
    p = p - lr * wd * p - lr * mhat / (np.sqrt(vhat) + eps)
    return p, m, v


@pytest.mark.parametrize("wd", [0.0, 0.1])
def test_many_steps_track_float64_textbook(wd):
    rng = np.random.default_rng(2)
    n = 20_000
    p = rng.standard_normal(n).astype(F32) * F32(0.02)
    m = np.zeros(n, F32)
    v = np.zeros(n, F32)
    pr, mr, vr = p.astype(np.float64), m.astype(np.float64), v.astype(np.float64)
    hp = dict(lr=float(F32(3e-4)), b1=float(F32(0.9)), b2=float(F32(0.95)),
              eps=float(F32(1e-8)), wd=float(F32(wd)))
    for t in range(1, 11):
        g = (rng.standard_normal(n) * 1e-3).astype(F32)
        p, m, v = OP.adamw(p, m, v, g, 3e-4, 0.9, 0.95, 1e-8, wd, t)
        pr, mr, vr = textbook_adamw(pr, mr, vr, g, hp["lr"], hp["b1"], hp["b2"],
                                    hp["eps"], hp["wd"], t)
    # float32 rounding of p itself dominates (about one ulp of |p| per step);
    # a dropped bias correction or decay term is off by ~lr = 3e-4
    assert np.max(np.abs(p - pr)) <= 1e-6 * np.max(np.abs(pr))
    assert np.max(np.abs(m - mr)) <= 1e-5 * np.max(np.abs(mr))
    assert np.max(np.abs(v - vr)) <= 1e-5 * np.max(np.abs(vr))


def test_bf16_cast_matches_torch_on_every_bf16_value():
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0x0000, 0x0001, 0x3FFF, 0x7FFF, 0x8000, 0x8001, 0xC000, 0xFFFF],
                    dtype=np.uint32)
    bits = (hi[:, None] | lows[None, :]).reshape(-1)
    x = bits.view(F32)
    ours = OP.bf16_rne_bits(x)
    ref = torch.from_numpy(x.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    nan = np.isnan(x)
    assert np.array_equal(ours[~nan], ref[~nan])
    # NaN stays NaN, keeps its sign, and is quiet
    assert np.all((ours[nan] & 0x7F80) == 0x7F80) and np.all((ours[nan] & 0x007F) != 0)
    assert np.all((ours[nan] & 0x0040) != 0)
    assert np.array_equal(ours[nan] >> 15, (bits[nan] >> 31).astype(np.uint16))


def test_bf16_cast_random_patterns():
    rng = np.random.default_rng(3)
    bits = rng.integers(0, 1 << 32, size=4_000_000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(F32)
    ours = OP.bf16_rne_bits(x)
    ref = torch.from_numpy(x.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    nan = np.isnan(x)
    assert np.array_equal(ours[~nan], ref[~nan])


def test_accumulate_exact_integers_in_order():
    rng = np.random.default_rng(4)
    G = np.zeros(1000, F32)
    parts = [rng.integers(-1000, 1000, size=1000).astype(F32) for _ in range(16)]
    for g in parts:
        G = OP.accumulate(G, g)
    assert np.array_equal(G, np.sum(np.stack(parts).astype(np.int64), axis=0).astype(F32))
    # +0 plus -0 stays +0: the accumulator is added to, never assigned
    Z = OP.accumulate(np.zeros(4, F32), np.array([-0.0] * 4, F32))
    assert np.all(np.signbit(Z) == False)
