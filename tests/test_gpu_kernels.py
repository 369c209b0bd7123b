"""Parity of the individual HIP kernels (through the C-ABI) with the oracle.

Bit-exact: gradient accumulation, AdamW + bf16 cast, the cast itself, and
GEMMs on integer-valued operands (every partial sum is an exact integer in
fp32). Within tolerance: GEMM on random operands, the fused epilogues,
RMSNorm and attention (fp32 path 1e-4, bf16 path 2e-2, max-normwise).
"""
import numpy as np
import pytest
import torch

import synth
from oracle import optim as OP
from oracle import stage as OS
from paper_2606_11169_amd import libchunk as lc
from paper_2606_11169_amd.runner import require_gpu
from tests.gpu_util import (DEV, banner, bf16, bf16_round, bits16, bits32, dev, f32, host, ints,
                            rel_err)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


# ---------------------------------------------------------------- accumulation

@pytest.mark.parametrize("gdt", ["f32", "bf16"])
@pytest.mark.parametrize("n", [1, 3, 255, 4097, (1 << 20) + 5])
def test_accumulate_bit_exact_and_covering(n, gdt):
    banner(f"accumulate n={n} g={gdt}")
    rng = np.random.default_rng(n)
    G0 = rng.standard_normal(n).astype(np.float32)
    g = rng.standard_normal(n).astype(np.float32)
    if gdt == "bf16":
        g = bf16_round(g)
    pad = 64
    Gd = f32(np.concatenate([G0, np.full(pad, 7.0, np.float32)]))
    gd = dev(np.concatenate([g, np.full(pad, 3.0, np.float32)]), gdt == "bf16")
    lc.chunk_accumulate_grad(Gd, gd, lc.LC_BF16 if gdt == "bf16" else lc.LC_FP32, n)
    torch.cuda.synchronize()
    got = bits32(Gd)
    want = OP.accumulate(G0, g).view(np.uint32)
    assert np.array_equal(got[:n], want)
    assert np.all(host(Gd)[n:] == 7.0)  # canary words untouched
    # sentinel: G = 0, g[i] = i  -> each element updated exactly once
    idx = (np.arange(n) % 256).astype(np.float32)
    Z = f32(np.zeros(n, np.float32))
    lc.chunk_accumulate_grad(Z, dev(idx, gdt == "bf16"), lc.LC_BF16 if gdt == "bf16" else lc.LC_FP32, n)
    torch.cuda.synchronize()
    assert np.array_equal(host(Z), idx)


def test_accumulate_disjoint_shards_leave_each_other_intact():
    banner("accumulate shards")
    n = 10_000
    G = f32(np.zeros(2 * n, np.float32))
    g = f32(np.ones(2 * n, np.float32))
    lc.chunk_accumulate_grad(G, g, lc.LC_FP32, n)
    lc.chunk_accumulate_grad(G.data_ptr() + 4 * n, g.data_ptr() + 4 * n, lc.LC_FP32, n)
    lc.chunk_accumulate_grad(G, g, lc.LC_FP32, n)
    torch.cuda.synchronize()
    h = host(G)
    assert np.all(h[:n] == 2.0) and np.all(h[n:] == 1.0)


# ---------------------------------------------------------------- AdamW

ADAM_CASES = [
    # (lr, b1, b2, eps, wd)
    (1e-3, 0.9, 0.999, 1e-8, 0.0),
    (3e-4, 0.9, 0.95, 1e-8, 0.1),
]


@pytest.mark.parametrize("hp", ADAM_CASES)
@pytest.mark.parametrize("state,step", [("zero", 1), ("warm", 10)])
@pytest.mark.parametrize("gdt", ["bf16", "f32"])
@pytest.mark.parametrize("n", [1, 7, 4099, (1 << 20) + 3])
def test_adam_bit_exact(n, gdt, state, step, hp):
    banner(f"adam n={n} g={gdt} {state} t={step} hp={hp}")
    p, m, v, g = synth.adam_inputs(n, seed=1, state=state)
    if gdt == "f32":
        g = synth.normal(1, 777, n, 1e-3)
    lr, b1, b2, eps, wd = hp
    p1, m1, v1 = OP.adamw(p, m, v, g, lr, b1, b2, eps, wd, step)
    out_ref = OP.bf16_rne_bits(p1)
    P, Mo, V = f32(p), f32(m), f32(v)
    Gd = dev(g, gdt == "bf16")
    out = torch.zeros(n + 8, dtype=torch.int16, device=DEV)
    lc.shard_adam_step(P, Mo, V, Gd, lc.LC_BF16 if gdt == "bf16" else lc.LC_FP32, out, n, lr, b1,
                       b2, eps, wd, step)
    torch.cuda.synchronize()
    assert np.array_equal(bits32(P), p1.view(np.uint32))
    assert np.array_equal(bits32(Mo), m1.view(np.uint32))
    assert np.array_equal(bits32(V), v1.view(np.uint32))
    ob = bits16(out)
    assert np.array_equal(ob[:n], out_ref)
    assert np.all(ob[n:] == 0)


def test_adam_without_cast_and_nonfinite_propagation():
    banner("adam no-cast + nan")
    n = 1000
    p, m, v, g = synth.adam_inputs(n, seed=2, state="warm")
    g = g.copy()
    g[5] = np.nan
    g[6] = np.inf
    p1, m1, v1 = OP.adamw(p, m, v, g, 3e-4, 0.9, 0.95, 1e-8, 0.1, 3)
    P, Mo, V = f32(p), f32(m), f32(v)
    lc.shard_adam_step(P, Mo, V, f32(g), lc.LC_FP32, None, n, 3e-4, 0.9, 0.95, 1e-8, 0.1, 3)
    torch.cuda.synchronize()
    # IEEE 754 leaves the sign and payload of a NaN produced by an operation
    # unspecified: compare NaN-ness there and every bit elsewhere
    got, want = bits32(P), p1.view(np.uint32)
    nan = np.isnan(p1)
    assert np.array_equal(np.isnan(host(P)), nan) and nan[5] and nan[6]
    assert np.array_equal(got[~nan], want[~nan])


# ---------------------------------------------------------------- cast

def test_cast_bf16_every_bf16_value_and_random_patterns():
    banner("cast bf16")
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0x0000, 0x0001, 0x3FFF, 0x7FFF, 0x8000, 0x8001, 0xC000, 0xFFFF], np.uint32)
    rng = np.random.default_rng(0)
    bits = np.concatenate([(hi[:, None] | lows[None, :]).reshape(-1),
                           rng.integers(0, 1 << 32, size=3_000_001, dtype=np.uint64).astype(np.uint32)])
    x = bits.view(np.float32)
    xin = torch.from_numpy(bits.view(np.int32).copy()).to(DEV).view(torch.float32)
    out = torch.empty(x.size, dtype=torch.int16, device=DEV)
    lc.lc_cast_bf16(xin, out, x.size)
    torch.cuda.synchronize()
    assert np.array_equal(bits16(out), OP.bf16_rne_bits(x))


# ---------------------------------------------------------------- GEMM

LAYOUTS = [(True, True), (True, False), (False, False)]


def operands(rng, M, N, K, a_k, b_k, integer, brows=None):
    brows = brows or N
    if integer:
        A, B = ints(rng, (M, K)), ints(rng, (brows, K))
    else:
        A = bf16_round(rng.standard_normal((M, K)).astype(np.float32))
        B = bf16_round(rng.standard_normal((brows, K)).astype(np.float32))
    Am = A if a_k else np.ascontiguousarray(A.T)
    Bm = B if b_k else np.ascontiguousarray(B.T)
    return A, B, bf16(Am), bf16(Bm), (K if a_k else M), (K if b_k else brows)


@pytest.mark.parametrize("layout", LAYOUTS, ids=["NT", "NN", "TN"])
@pytest.mark.parametrize("shape", [(256, 256, 64), (304, 264, 200), (512, 768, 1024), (8, 8, 8),
                                   (1024, 256, 4096)])
def test_gemm_integer_operands_bit_exact(shape, layout):
    M, N, K = shape
    a_k, b_k = layout
    banner(f"gemm int {shape} layout={layout}")
    rng = np.random.default_rng(M + N + K)
    A, B, Ad, Bd, lda, ldb = operands(rng, M, N, K, a_k, b_k, True)
    exact = (A.astype(np.int64) @ B.astype(np.int64).T).astype(np.float32)
    C = torch.full((M, N), -1.0, dtype=torch.float32, device=DEV)
    lc.lc_gemm(lc.LC_BF16, lc.LC_EPI_STORE_F32, M, N, K, Ad, lda, a_k, Bd, ldb, b_k, C, N)
    torch.cuda.synchronize()
    assert np.array_equal(host(C), exact)
    if not (a_k and not b_k):
        C0 = ints(rng, (M, N), -1000, 1000)
        Cacc = f32(C0)
        lc.lc_gemm(lc.LC_BF16, lc.LC_EPI_ACCUM_F32, M, N, K, Ad, lda, a_k, Bd, ldb, b_k, Cacc, N)
        torch.cuda.synchronize()
        assert np.array_equal(host(Cacc), C0 + exact)
    Cb = torch.empty((M, N), dtype=torch.bfloat16, device=DEV)
    lc.lc_gemm(lc.LC_BF16, lc.LC_EPI_STORE, M, N, K, Ad, lda, a_k, Bd, ldb, b_k, Cb, N)
    torch.cuda.synchronize()
    assert np.array_equal(bits16(Cb).reshape(M, N), OP.bf16_rne_bits(exact))


@pytest.mark.parametrize("layout", LAYOUTS, ids=["NT", "NN", "TN"])
def test_gemm_random_operands(layout):
    a_k, b_k = layout
    M, N, K = 520, 384, 1032
    banner(f"gemm random layout={layout}")
    rng = np.random.default_rng(5)
    A, B, Ad, Bd, lda, ldb = operands(rng, M, N, K, a_k, b_k, False)
    ref = A.astype(np.float64) @ B.astype(np.float64).T
    C = torch.empty((M, N), dtype=torch.float32, device=DEV)
    lc.lc_gemm(lc.LC_BF16, lc.LC_EPI_STORE_F32, M, N, K, Ad, lda, a_k, Bd, ldb, b_k, C, N)
    torch.cuda.synchronize()
    assert rel_err(host(C), ref) <= 1e-5


TORCH_DT = {lc.LC_BF16: torch.bfloat16, lc.LC_FP16: torch.float16, lc.LC_FP32: torch.float32}
# normwise bound for one rounding of the output to its type
ROUND_TOL = {lc.LC_BF16: 8e-3, lc.LC_FP16: 1e-3, lc.LC_FP32: 1e-5}


@pytest.mark.parametrize("r_dt,c_dt", [(lc.LC_BF16, lc.LC_BF16), (lc.LC_BF16, lc.LC_FP32),
                                       (lc.LC_FP32, lc.LC_FP32), (lc.LC_FP32, lc.LC_BF16)])
def test_gemm_residual_epilogue(r_dt, c_dt):
    banner(f"gemm residual r={r_dt} c={c_dt}")
    rng = np.random.default_rng(6)
    M, N, K = 384, 512, 256
    A, B, Ad, Bd, lda, ldb = operands(rng, M, N, K, True, True, False)
    R = rng.standard_normal((M, N)).astype(np.float32)
    if r_dt == lc.LC_BF16:
        R = bf16_round(R)
    C = torch.empty((M, N), dtype=TORCH_DT[c_dt], device=DEV)
    lc.lc_gemm(lc.LC_BF16, lc.LC_EPI_RESIDUAL, M, N, K, Ad, lda, 1, Bd, ldb, 1, C, N,
               R=dev(R, r_dt == lc.LC_BF16), ldr=N, r_dtype=r_dt, c_dtype=c_dt)
    torch.cuda.synchronize()
    ref = R + A.astype(np.float64) @ B.astype(np.float64).T
    assert rel_err(host(C), ref) <= ROUND_TOL[c_dt]


@pytest.mark.parametrize("c_dt", [lc.LC_BF16, lc.LC_FP16])
def test_gemm_rope_epilogue(c_dt):
    banner(f"gemm rope c={c_dt}")
    rng = np.random.default_rng(7)
    H, hd, S, b = 2, 128, 256, 2
    d = H * hd
    T, N, K = b * S, 3 * d, d
    A, B, Ad, Bd, lda, ldb = operands(rng, T, N, K, True, True, False)
    cos, sin = OS.rope_tables(S, hd, 10000.0)
    C = torch.empty((T, N), dtype=TORCH_DT[c_dt], device=DEV)
    lc.lc_gemm(lc.LC_BF16, lc.LC_EPI_ROPE, T, N, K, Ad, lda, 1, Bd, ldb, 1, C, N,
               rope_cos=f32(cos), rope_sin=f32(sin), rope_seq=S, rope_cols=2 * d, head_dim=hd,
               c_dtype=c_dt)
    torch.cuda.synchronize()
    prod = (A.astype(np.float64) @ B.astype(np.float64).T).reshape(b, S, 3, H, hd)
    q = OS.rope_apply(prod[:, :, 0], cos, sin)
    k = OS.rope_apply(prod[:, :, 1], cos, sin)
    ref = np.stack([q, k, prod[:, :, 2]], axis=2).reshape(T, N)
    assert rel_err(host(C), ref) <= ROUND_TOL[c_dt]


@pytest.mark.parametrize("aux_dt", [lc.LC_BF16, lc.LC_FP32])
def test_gemm_swiglu_epilogues(aux_dt):
    banner(f"gemm swiglu fwd/bwd aux={aux_dt}")
    rng = np.random.default_rng(8)
    T, F, D = 384, 320, 256
    A, B13, Ad, Bd, lda, ldb = operands(rng, T, F, D, True, True, False, brows=2 * F)
    act = torch.empty((T, F), dtype=torch.bfloat16, device=DEV)
    gate = torch.empty((T, F), dtype=TORCH_DT[aux_dt], device=DEV)
    up = torch.empty_like(gate)
    lc.lc_gemm(lc.LC_BF16, lc.LC_EPI_SWIGLU, T, F, D, Ad, lda, 1, Bd, ldb, 1, act, F,
               aux0=gate, aux1=up, ld_aux=F, aux_dtype=aux_dt)
    torch.cuda.synchronize()
    prod = A.astype(np.float64) @ B13.astype(np.float64).T
    g_ref, u_ref = prod[:, :F], prod[:, F:]
    assert rel_err(host(gate), g_ref) <= ROUND_TOL[aux_dt]
    assert rel_err(host(up), u_ref) <= ROUND_TOL[aux_dt]
    assert rel_err(host(act), OS.silu(g_ref) * u_ref) <= 1e-2
    # backward: da = dy W2 (W2 [D, F] read with k = D not contiguous)
    dy = bf16_round(rng.standard_normal((T, D)).astype(np.float32))
    W2 = bf16_round(rng.standard_normal((D, F)).astype(np.float32) * 0.05)
    gv, uv = host(gate), host(up)
    dgu = torch.empty((T, 2 * F), dtype=torch.bfloat16, device=DEV)
    lc.lc_gemm(lc.LC_BF16, lc.LC_EPI_SWIGLU_BWD, T, F, D, bf16(dy), D, 1, bf16(W2), F, 0, dgu,
               2 * F, aux0=gate, aux1=up, ld_aux=F, aux_dtype=aux_dt)
    torch.cuda.synchronize()
    da = dy.astype(np.float64) @ W2.astype(np.float64)
    s = OS.sigmoid(gv)
    ref = np.concatenate([da * uv * s * (1 + gv * (1 - s)), da * OS.silu(gv)], axis=1)
    assert rel_err(host(dgu), ref) <= 1e-2


@pytest.mark.parametrize("layout", LAYOUTS, ids=["NT", "NN", "TN"])
def test_gemm_fp32_path(layout):
    a_k, b_k = layout
    banner(f"gemm fp32 layout={layout}")
    rng = np.random.default_rng(9)
    M, N, K = 130, 90, 70
    A = rng.standard_normal((M, K)).astype(np.float32)
    B = rng.standard_normal((N, K)).astype(np.float32)
    Am = A if a_k else np.ascontiguousarray(A.T)
    Bm = B if b_k else np.ascontiguousarray(B.T)
    C = torch.empty((M, N), dtype=torch.float32, device=DEV)
    lc.lc_gemm(lc.LC_FP32, lc.LC_EPI_STORE, M, N, K, f32(Am), K if a_k else M, a_k, f32(Bm),
               K if b_k else N, b_k, C, N)
    torch.cuda.synchronize()
    assert rel_err(host(C), A.astype(np.float64) @ B.astype(np.float64).T) <= 1e-5


# ---------------------------------------------------------------- RMSNorm

def typed(rng_arr, dt):
    """host values representable in dt, and the device tensor"""
    a = rng_arr.astype(np.float32)
    if dt == lc.LC_BF16:
        a = bf16_round(a)
    elif dt == lc.LC_FP16:
        a = a.astype(np.float16).astype(np.float32)
    return a, torch.from_numpy(a).to(TORCH_DT[dt]).to(DEV)


# (x, weights/out, dn, dres, dx) element types: the fp32 path, the bf16 stage's
# first-layer norm (bf16 input) and its inner norms (fp32 residual stream)
NORM_TYPES = [
    (lc.LC_FP32, lc.LC_FP32, lc.LC_FP32, lc.LC_FP32, lc.LC_FP32),
    (lc.LC_BF16, lc.LC_BF16, lc.LC_FP32, lc.LC_BF16, lc.LC_BF16),
    (lc.LC_FP32, lc.LC_BF16, lc.LC_FP32, lc.LC_FP32, lc.LC_FP32),
]


@pytest.mark.parametrize("types", NORM_TYPES, ids=["fp32", "bf16_in", "fp32_res"])
def test_rmsnorm_forward_backward(types):
    x_dt, w_dt, dn_dt, dres_dt, dx_dt = types
    banner(f"rmsnorm types={types}")
    rng = np.random.default_rng(10)
    T, d, eps = 300, 512, 1e-5
    x, xd = typed(rng.standard_normal((T, d)), x_dt)
    g, gd = typed(1 + 0.1 * rng.standard_normal(d), w_dt)
    dn, dnd = typed(rng.standard_normal((T, d)), dn_dt)
    dres, dresd = typed(rng.standard_normal((T, d)), dres_dt)
    n = torch.empty((T, d), dtype=TORCH_DT[w_dt], device=DEV)
    rstd = torch.empty(T, dtype=torch.float32, device=DEV)
    lc.lc_rmsnorm_forward(T, d, xd, gd, eps, n, rstd, x_dt, w_dt, w_dt)
    n_ref, r_ref = OS.rmsnorm_forward(x.astype(np.float64), g.astype(np.float64), eps)
    torch.cuda.synchronize()
    assert rel_err(host(n), n_ref) <= ROUND_TOL[w_dt]
    assert rel_err(host(rstd), r_ref[:, 0]) <= 1e-5
    dx = torch.empty((T, d), dtype=TORCH_DT[dx_dt], device=DEV)
    dx_copy = torch.empty((T, d), dtype=torch.bfloat16, device=DEV)
    dg0 = rng.standard_normal(d).astype(np.float32)
    dg = f32(dg0)
    sb = lc.lc_rmsnorm_scratch_bytes(T, d)
    scratch = torch.empty(sb, dtype=torch.uint8, device=DEV)
    lc.lc_rmsnorm_backward(T, d, dnd, xd, rstd, gd, dresd, dx, dg, scratch, sb, dn_dt, x_dt, w_dt,
                           dres_dt, dx_dt, dx_copy=dx_copy)
    torch.cuda.synchronize()
    dx_ref, dg_ref = OS.rmsnorm_backward(dn.astype(np.float64), x.astype(np.float64),
                                         host(rstd)[:, None], g.astype(np.float64))
    assert rel_err(host(dx), dres + dx_ref) <= ROUND_TOL[dx_dt] + 1e-5
    assert rel_err(host(dx_copy), dres + dx_ref) <= ROUND_TOL[lc.LC_BF16]
    assert rel_err(host(dg), dg0 + dg_ref) <= 1e-5


# ---------------------------------------------------------------- attention

def packed_qkv(rng, B, S, H, hd, dt, identical_keys=False):
    d = H * hd
    qkv = rng.standard_normal((B, S, 3, H, hd)).astype(np.float32)
    if identical_keys:
        qkv[:, :, 1] = qkv[:, :1, 1]
    qkv, qkvd = typed(qkv.reshape(B * S, 3 * d), dt)
    return qkv.reshape(B, S, 3, H, hd), qkvd


def attn_case(B, S, H, hd, dt, seed, rope):
    banner(f"attention B={B} S={S} H={H} hd={hd} dtype={dt} rope={rope}")
    rng = np.random.default_rng(seed)
    d = H * hd
    mc = dt != lc.LC_FP32
    o_dt = lc.LC_BF16 if mc else lc.LC_FP32
    qkv, qkvd = packed_qkv(rng, B, S, H, hd, dt)
    esz = 2 if mc else 4
    base = qkvd.data_ptr()
    o = torch.empty((B * S, d), dtype=TORCH_DT[o_dt], device=DEV)
    lse = torch.empty(B * H * S, dtype=torch.float32, device=DEV)
    lc.lc_attention_forward(dt, o_dt, B, S, H, hd, base, base + d * esz, base + 2 * d * esz, 3 * d,
                            o, d, lse)
    q, k, v = (qkv[:, :, i].astype(np.float64) for i in range(3))
    o_ref = OS.attention_forward(q, k, v)
    s = np.einsum("bihe,bjhe->bhij", q, k) / np.sqrt(hd)
    s = np.where(np.triu(np.ones((S, S), bool), 1)[None, None], -np.inf, s)
    mx = s.max(-1, keepdims=True)
    lse_ref = (mx + np.log(np.exp(s - mx).sum(-1, keepdims=True)))[..., 0]
    torch.cuda.synchronize()
    tol = 2e-2 if mc else 1e-4
    assert rel_err(host(o).reshape(B, S, H, hd), o_ref) <= tol / 2
    assert np.max(np.abs(host(lse).reshape(B, H, S) - lse_ref)) <= (1e-2 if mc else 1e-5)
    do, dod = typed(rng.standard_normal((B * S, d)), o_dt)
    do = do.reshape(B, S, H, hd)
    dqkv = torch.zeros((B * S, 3 * d), dtype=TORCH_DT[o_dt], device=DEV)
    cos = sin = None
    if rope:
        cos, sin = OS.rope_tables(S, hd, 10000.0)
    sb = lc.lc_attention_scratch_bytes(B, S, H)
    scratch = torch.empty(sb, dtype=torch.uint8, device=DEV)
    g0 = dqkv.data_ptr()
    lc.lc_attention_backward(dt, o_dt, B, S, H, hd, base, base + d * esz, base + 2 * d * esz, 3 * d,
                             o, dod, d, lse, g0, g0 + d * esz, g0 + 2 * d * esz, 3 * d,
                             None if cos is None else f32(cos), None if sin is None else f32(sin),
                             scratch, sb)
    # reference uses the kernel's own (rounded) O only through D = rowsum(dO*O): use exact O
    dq, dk, dv = OS.attention_backward(do.astype(np.float64), q, k, v)
    if rope:
        dq = OS.rope_apply(dq, cos, sin, inverse=True)
        dk = OS.rope_apply(dk, cos, sin, inverse=True)
    torch.cuda.synchronize()
    got = host(dqkv).reshape(B, S, 3, H, hd)
    errs = [rel_err(got[:, :, i], ref) for i, ref in enumerate((dq, dk, dv))]
    print(f"attention errors: o {rel_err(host(o).reshape(B, S, H, hd), o_ref):.2e} "
          f"dq {errs[0]:.2e} dk {errs[1]:.2e} dv {errs[2]:.2e}", flush=True)
    for i, e in enumerate(errs):
        assert e <= tol, ("dq", "dk", "dv")[i]


@pytest.mark.parametrize("dt", [lc.LC_FP16, lc.LC_BF16], ids=["fp16", "bf16"])
@pytest.mark.parametrize("rope", [False, True])
def test_attention_matrix_cores(rope, dt):
    attn_case(2, 256, 2, 128, dt, 11, rope)


def test_attention_longer_sequence():
    attn_case(1, 512, 1, 128, lc.LC_FP16, 12, True)


@pytest.mark.parametrize("dt", [lc.LC_FP16, lc.LC_BF16], ids=["fp16", "bf16"])
@pytest.mark.parametrize("rope", [False, True])
def test_attention_half_full_last_block(rope, dt):
    """S = 384: workgroups own 256 queries or keys, so the last block is half
    full after a full one (partial-block masking in the forward, dK/dV and
    dQ, and the heavy-first block order over unequal blocks)."""
    attn_case(2, 384, 2, 128, dt, 15, rope)


@pytest.mark.parametrize("dt", [lc.LC_FP16, lc.LC_BF16], ids=["fp16", "bf16"])
@pytest.mark.parametrize("S", [2048, 4096])
def test_attention_full_length(S, dt):
    """The benchmark stages' sequence lengths, every position compared: the
    long off-diagonal key loops of the forward and both backward kernels."""
    attn_case(1, S, 2, 128, dt, 16 + S, True)


def test_attention_backward_with_caller_bf16_copies():
    """fp16 q/k/v with the bf16 copies supplied by the caller (qkv_bf16): the
    backward reads them instead of writing its own, bit for bit the same."""
    banner("attention backward with caller bf16 copies")
    rng = np.random.default_rng(31)
    B, S, H, hd = 1, 384, 2, 128
    d = H * hd
    qkv, qkvd = packed_qkv(rng, B, S, H, hd, lc.LC_FP16)
    base = qkvd.data_ptr()
    o = torch.empty((B * S, d), dtype=torch.bfloat16, device=DEV)
    lse = torch.empty(B * H * S, dtype=torch.float32, device=DEV)
    lc.lc_attention_forward(lc.LC_FP16, lc.LC_BF16, B, S, H, hd, base, base + 2 * d, base + 4 * d,
                            3 * d, o, d, lse)
    _, dod = typed(rng.standard_normal((B * S, d)), lc.LC_BF16)
    cos, sin = OS.rope_tables(S, hd, 10000.0)
    copies = torch.zeros((B * S, 3 * d + 64), dtype=torch.bfloat16, device=DEV)  # padded rows
    copies[:, :3 * d] = qkvd.to(torch.bfloat16)
    outs = []
    for caller in (False, True):
        sb = lc.lc_attention_scratch_bytes(B, S, H)
        scratch = torch.empty(sb, dtype=torch.uint8, device=DEV)
        dqkv = torch.zeros((B * S, 3 * d), dtype=torch.bfloat16, device=DEV)
        g0 = dqkv.data_ptr()
        lc.lc_attention_backward(lc.LC_FP16, lc.LC_BF16, B, S, H, hd, base, base + 2 * d,
                                 base + 4 * d, 3 * d, o, dod, d, lse, g0, g0 + 2 * d, g0 + 4 * d,
                                 3 * d, f32(cos), f32(sin), scratch, sb,
                                 qkv_bf16=copies if caller else None,
                                 ld_qkv_bf16=3 * d + 64 if caller else 0)
        torch.cuda.synchronize()
        outs.append(bits16(dqkv))
    assert np.array_equal(outs[0], outs[1])


def test_gqa_attention_backward_with_caller_bf16_copies():
    """Grouped-query attention (4 query heads over 2 key/value heads), fp16 q/k/v:
    caller-supplied bf16 copies (k at column H*hd, v at (H + Hkv)*hd of the copy
    rows) give the gradients of the backward's own copy pass, bit for bit."""
    banner("gqa attention backward with caller bf16 copies")
    rng = np.random.default_rng(33)
    B, S, H, Hkv, hd = 1, 256, 4, 2, 128
    d, dkv = H * hd, Hkv * hd
    ld = d + 2 * dkv
    _, qkvd = typed(rng.standard_normal((B * S, ld)), lc.LC_FP16)
    base = qkvd.data_ptr()
    o = torch.empty((B * S, d), dtype=torch.bfloat16, device=DEV)
    lse = torch.empty(B * H * S, dtype=torch.float32, device=DEV)
    lc.lc_attention_forward(lc.LC_FP16, lc.LC_BF16, B, S, H, hd, base, base + 2 * d,
                            base + 2 * (d + dkv), ld, o, d, lse, Hkv=Hkv)
    _, dod = typed(rng.standard_normal((B * S, d)), lc.LC_BF16)
    cos, sin = OS.rope_tables(S, hd, 10000.0)
    copies = torch.zeros((B * S, ld + 32), dtype=torch.bfloat16, device=DEV)  # padded rows
    copies[:, :ld] = qkvd.to(torch.bfloat16)
    outs = []
    for caller in (False, True):
        sb = lc.lc_attention_scratch_bytes(B, S, H, Hkv)
        scratch = torch.empty(sb, dtype=torch.uint8, device=DEV)
        dqkv = torch.zeros((B * S, ld), dtype=torch.bfloat16, device=DEV)
        g0 = dqkv.data_ptr()
        lc.lc_attention_backward(lc.LC_FP16, lc.LC_BF16, B, S, H, hd, base, base + 2 * d,
                                 base + 2 * (d + dkv), ld, o, dod, d, lse, g0, g0 + 2 * d,
                                 g0 + 2 * (d + dkv), ld, f32(cos), f32(sin), scratch, sb, Hkv=Hkv,
                                 qkv_bf16=copies if caller else None,
                                 ld_qkv_bf16=ld + 32 if caller else 0)
        torch.cuda.synchronize()
        outs.append(bits16(dqkv))
    assert np.array_equal(outs[0], outs[1])


def test_gemm_rope_epilogue_second_copy():
    """LC_EPI_ROPE with aux0: the rotated q|k|v in fp16 (C) and in bf16 (aux0)."""
    banner("gemm rope second copy")
    rng = np.random.default_rng(32)
    H, hd, S = 2, 128, 256
    d = H * hd
    T, N, K = S, 3 * d, d
    A, B, Ad, Bd, lda, ldb = operands(rng, T, N, K, True, True, False)
    cos, sin = OS.rope_tables(S, hd, 10000.0)
    C = torch.empty((T, N), dtype=torch.float16, device=DEV)
    Cb = torch.empty((T, N + 8), dtype=torch.bfloat16, device=DEV)
    lc.lc_gemm(lc.LC_BF16, lc.LC_EPI_ROPE, T, N, K, Ad, lda, 1, Bd, ldb, 1, C, N,
               rope_cos=f32(cos), rope_sin=f32(sin), rope_seq=S, rope_cols=2 * d, head_dim=hd,
               c_dtype=lc.LC_FP16, aux0=Cb, ld_aux=N + 8, aux_dtype=lc.LC_BF16)
    torch.cuda.synchronize()
    prod = (A.astype(np.float64) @ B.astype(np.float64).T).reshape(1, S, 3, H, hd)
    q = OS.rope_apply(prod[:, :, 0], cos, sin)
    k = OS.rope_apply(prod[:, :, 1], cos, sin)
    ref = np.stack([q, k, prod[:, :, 2]], axis=2).reshape(T, N)
    assert rel_err(host(C), ref) <= ROUND_TOL[lc.LC_FP16]
    assert rel_err(host(Cb)[:, :N], ref) <= ROUND_TOL[lc.LC_BF16]


@pytest.mark.parametrize("hd", [32, 8])
def test_attention_fp32(hd):
    attn_case(2, 64, 4, hd, lc.LC_FP32, 13, True)


@pytest.mark.parametrize("dt", [lc.LC_FP16, lc.LC_BF16], ids=["fp16", "bf16"])
def test_attention_identical_keys_prefix_mean(dt):
    banner("attention identical keys")
    rng = np.random.default_rng(14)
    B, S, H, hd = 1, 256, 2, 128
    d = H * hd
    qkv, qkvd = packed_qkv(rng, B, S, H, hd, dt, identical_keys=True)
    base = qkvd.data_ptr()
    o = torch.empty((B * S, d), dtype=torch.bfloat16, device=DEV)
    lse = torch.empty(B * H * S, dtype=torch.float32, device=DEV)
    lc.lc_attention_forward(dt, lc.LC_BF16, B, S, H, hd, base, base + 2 * d, base + 4 * d, 3 * d,
                            o, d, lse)
    torch.cuda.synchronize()
    v = qkv[:, :, 2].astype(np.float64)
    prefix_mean = np.cumsum(v, axis=1) / np.arange(1, S + 1)[None, :, None, None]
    assert rel_err(host(o).reshape(B, S, H, hd), prefix_mean) <= 1e-2


# ---------------------------------------------------------------- grouped-query attention

def gqa_case(B, S, H, Hkv, hd, dt, seed, rope):
    """Packed rows [q (H heads) | k (Hkv) | v (Hkv)] against the oracle's
    attention over key/value heads repeated per group (query head h reads
    key/value head h // (H / Hkv)); dk, dv sum over each group."""
    banner(f"gqa attention B={B} S={S} H={H} Hkv={Hkv} hd={hd} dtype={dt} rope={rope}")
    rng = np.random.default_rng(seed)
    d, dkv = H * hd, Hkv * hd
    G = H // Hkv
    ld = d + 2 * dkv
    mc = dt != lc.LC_FP32
    o_dt = lc.LC_BF16 if mc else lc.LC_FP32
    esz = 2 if mc else 4
    qkv, qkvd = typed(rng.standard_normal((B * S, ld)), dt)
    q = qkv[:, :d].reshape(B, S, H, hd).astype(np.float64)
    k = qkv[:, d:d + dkv].reshape(B, S, Hkv, hd).astype(np.float64)
    v = qkv[:, d + dkv:].reshape(B, S, Hkv, hd).astype(np.float64)
    base = qkvd.data_ptr()
    o = torch.empty((B * S, d), dtype=TORCH_DT[o_dt], device=DEV)
    lse = torch.empty(B * H * S, dtype=torch.float32, device=DEV)
    lc.lc_attention_forward(dt, o_dt, B, S, H, hd, base, base + d * esz, base + (d + dkv) * esz,
                            ld, o, d, lse, Hkv=Hkv)
    o_ref = OS.attention_forward(q, OS.repeat_kv(k, G), OS.repeat_kv(v, G))
    tol = 2e-2 if mc else 1e-4
    torch.cuda.synchronize()
    assert rel_err(host(o).reshape(B, S, H, hd), o_ref) <= tol / 2
    do, dod = typed(rng.standard_normal((B * S, d)), o_dt)
    dqkv = torch.full((B * S, ld), float("nan"), dtype=TORCH_DT[o_dt], device=DEV)
    cos = sin = None
    if rope:
        cos, sin = OS.rope_tables(S, hd, 10000.0)
    sb = lc.lc_attention_scratch_bytes(B, S, H, Hkv)
    scratch = torch.empty(sb, dtype=torch.uint8, device=DEV)
    g0 = dqkv.data_ptr()
    lc.lc_attention_backward(dt, o_dt, B, S, H, hd, base, base + d * esz, base + (d + dkv) * esz,
                             ld, o, dod, d, lse, g0, g0 + d * esz, g0 + (d + dkv) * esz, ld,
                             None if cos is None else f32(cos), None if sin is None else f32(sin),
                             scratch, sb, Hkv=Hkv)
    dq, dke, dve = OS.attention_backward(do.reshape(B, S, H, hd).astype(np.float64), q,
                                         OS.repeat_kv(k, G), OS.repeat_kv(v, G))
    dk, dv = OS.sum_groups(dke, G), OS.sum_groups(dve, G)
    if rope:
        dq = OS.rope_apply(dq, cos, sin, inverse=True)
        dk = OS.rope_apply(dk, cos, sin, inverse=True)
    torch.cuda.synchronize()
    got = host(dqkv)
    errs = [rel_err(got[:, :d].reshape(B, S, H, hd), dq),
            rel_err(got[:, d:d + dkv].reshape(B, S, Hkv, hd), dk),
            rel_err(got[:, d + dkv:].reshape(B, S, Hkv, hd), dv)]
    print(f"gqa errors: dq {errs[0]:.2e} dk {errs[1]:.2e} dv {errs[2]:.2e}", flush=True)
    for i, e in enumerate(errs):
        assert e <= tol, ("dq", "dk", "dv")[i]


@pytest.mark.parametrize("dt", [lc.LC_FP16, lc.LC_BF16], ids=["fp16", "bf16"])
@pytest.mark.parametrize("H,Hkv", [(4, 1), (4, 2), (2, 2)])
def test_gqa_attention_matrix_cores(H, Hkv, dt):
    gqa_case(2, 256, H, Hkv, 128, dt, 21, True)


@pytest.mark.parametrize("rope", [False, True])
def test_gqa_attention_half_full_last_block(rope):
    gqa_case(1, 384, 4, 2, 128, lc.LC_FP16, 24, rope)


@pytest.mark.parametrize("H,Hkv", [(4, 2), (6, 3)])
def test_gqa_attention_fp32(H, Hkv):
    gqa_case(2, 64, H, Hkv, 32, lc.LC_FP32, 22, True)


# ---------------------------------------------------------------- per-head q/k norm

@pytest.mark.parametrize("x_dt,d_dt,w_dt,hd", [(lc.LC_FP16, lc.LC_BF16, lc.LC_BF16, 128),
                                               (lc.LC_FP32, lc.LC_FP32, lc.LC_FP32, 32),
                                               (lc.LC_FP32, lc.LC_FP32, lc.LC_FP32, 64)],
                         ids=["bf16_stage", "fp32_hd32", "fp32_hd64"])
def test_qk_norm_rope(x_dt, d_dt, w_dt, hd):
    """RMSNorm over each q and k head row, gains qn / kn, then RoPE (forward);
    the backward maps the gradient at the normalised rows to the raw rows and
    sums the gain gradients, against the oracle's RMSNorm and RoPE."""
    banner(f"q/k norm x={x_dt} d={d_dt} hd={hd}")
    rng = np.random.default_rng(23)
    B, S, H, Hkv = 2, 24, 4, 2
    T = B * S
    d, dkv = H * hd, Hkv * hd
    ld = d + 2 * dkv + 8  # a padded row, v columns untouched
    eps = 1e-6
    x, xd = typed(rng.standard_normal((T, ld)) * 3.0, x_dt)
    gq, gqd = typed(1.0 + 0.1 * rng.standard_normal(hd), w_dt)
    gk, gkd = typed(1.0 + 0.1 * rng.standard_normal(hd), w_dt)
    cos, sin = OS.rope_tables(S, hd, 10000.0)
    raw = torch.empty((T, d + dkv), dtype=TORCH_DT[x_dt], device=DEV)
    rstd = torch.empty(T * (H + Hkv), dtype=torch.float32, device=DEV)
    lc.lc_qk_norm_rope_forward(T, H, Hkv, hd, S, eps, xd, ld, raw, rstd, gqd, gkd, x_dt, w_dt,
                               f32(cos), f32(sin))
    torch.cuda.synchronize()
    xq = x[:, :d].reshape(B, S, H, hd).astype(np.float64)
    xk = x[:, d:d + dkv].reshape(B, S, Hkv, hd).astype(np.float64)
    yq, rq = OS.rmsnorm_forward(xq, gq.astype(np.float64), eps)
    yk, rk = OS.rmsnorm_forward(xk, gk.astype(np.float64), eps)
    zq, zk = OS.rope_apply(yq, cos, sin), OS.rope_apply(yk, cos, sin)
    got = host(xd)
    tol = ROUND_TOL[x_dt] + 1e-5
    assert rel_err(got[:, :d].reshape(B, S, H, hd), zq) <= tol
    assert rel_err(got[:, d:d + dkv].reshape(B, S, Hkv, hd), zk) <= tol
    assert np.array_equal(got[:, d + dkv:], x[:, d + dkv:])  # v and padding untouched
    assert np.array_equal(host(raw), x[:, :d + dkv])
    r_ref = np.concatenate([rq.reshape(T, H), rk.reshape(T, Hkv)], axis=1)
    assert rel_err(host(rstd).reshape(T, H + Hkv), r_ref) <= 1e-5
    # backward: dy at the normalised (unrotated) rows, in place
    dy, dyd = typed(rng.standard_normal((T, ld)), d_dt)
    dg = torch.full((2 * hd,), 0.5, dtype=torch.float32, device=DEV)
    sb = lc.lc_qk_norm_scratch_bytes(T, hd)
    scratch = torch.empty(sb, dtype=torch.uint8, device=DEV)
    lc.lc_qk_norm_rope_backward(T, H, Hkv, hd, S, eps, raw, rstd, gqd, gkd, x_dt, w_dt, dyd, ld,
                                d_dt, dg[:hd], dg[hd:], scratch, sb)
    torch.cuda.synchronize()
    xr = host(raw)  # the kernel's own raw rows and rstd: the reference uses them too
    rr = host(rstd).reshape(T, H + Hkv)
    dxq, dgq = OS.rmsnorm_backward(dy[:, :d].reshape(T, H, hd).astype(np.float64),
                                   xr[:, :d].reshape(T, H, hd), rr[:, :H, None],
                                   gq.astype(np.float64))
    dxk, dgk = OS.rmsnorm_backward(dy[:, d:d + dkv].reshape(T, Hkv, hd).astype(np.float64),
                                   xr[:, d:].reshape(T, Hkv, hd), rr[:, H:, None],
                                   gk.astype(np.float64))
    got = host(dyd)
    tol = ROUND_TOL[d_dt] + 1e-5
    assert rel_err(got[:, :d].reshape(T, H, hd), dxq) <= tol
    assert rel_err(got[:, d:d + dkv].reshape(T, Hkv, hd), dxk) <= tol
    assert np.array_equal(got[:, d + dkv:], dy[:, d + dkv:])
    gg = host(dg)
    assert rel_err(gg[:hd], 0.5 + dgq) <= 1e-5 and rel_err(gg[hd:], 0.5 + dgk) <= 1e-5
    # the same call twice gives the same bits (fixed reduction order)
    dyd2 = torch.from_numpy(dy).to(TORCH_DT[d_dt]).to(DEV)
    dg2 = torch.full((2 * hd,), 0.5, dtype=torch.float32, device=DEV)
    lc.lc_qk_norm_rope_backward(T, H, Hkv, hd, S, eps, raw, rstd, gqd, gkd, x_dt, w_dt, dyd2, ld,
                                d_dt, dg2[:hd], dg2[hd:], scratch, sb)
    torch.cuda.synchronize()
    assert torch.equal(dyd2, dyd) and torch.equal(dg2, dg)


# ---------------------------------------------------------------- full-size AdamW shard

def test_adam_full_size_shard_sampled_bit_exact():
    """The 1.6e9-element shard in the benchmark's launch (two steps, bf16
    gradient, bf16 cast): a sample of elements, including the first and the
    last ones (the tail past the last 8-element block), taken before each
    step and checked bit for bit against the oracle's AdamW on them."""
    cfg = synth.ADAM_1P6B
    n = cfg.n
    banner(f"adam full-size shard n={n}")
    g = torch.Generator(device=DEV)
    g.manual_seed(11)
    p = torch.randn(n, generator=g, device=DEV).mul_(cfg.p_std)
    m = torch.zeros_like(p)
    v = torch.zeros_like(p)
    gr = torch.randn(n, generator=g, device=DEV).mul_(cfg.g_std).to(torch.bfloat16)
    out = torch.empty(n, dtype=torch.bfloat16, device=DEV)
    rng = np.random.default_rng(31)
    idx = np.unique(np.concatenate([np.arange(16), np.arange(n - 16, n),
                                    rng.integers(0, n, 200_000)]))
    it = torch.from_numpy(idx).to(DEV)
    for step in (1, 2):
        p0, m0, v0 = (host32(t[it]) for t in (p, m, v))
        g0 = gr[it].float().cpu().numpy()
        lc.shard_adam_step(p, m, v, gr, lc.LC_BF16, out, n, cfg.lr, cfg.beta1, cfg.beta2,
                           cfg.eps, cfg.weight_decay, step)
        torch.cuda.synchronize()
        pr, mr, vr = OP.adamw(p0, m0, v0, g0, cfg.lr, cfg.beta1, cfg.beta2, cfg.eps,
                              cfg.weight_decay, step)
        for got, ref, name in ((p, pr, "p"), (m, mr, "m"), (v, vr, "v")):
            assert np.array_equal(host32(got[it]).view(np.uint32), ref.view(np.uint32)), name
        assert np.array_equal(out[it].cpu().view(torch.int16).numpy().view(np.uint16),
                              OP.bf16_rne_bits(pr)), "bf16 cast"
    del p, m, v, gr, out
    torch.cuda.empty_cache()


def host32(t):
    return t.detach().float().cpu().numpy().astype(np.float32)


# ---------------------------------------------------------------- 64-bit coverage

N64 = (1 << 31) + 17   # element indices and byte offsets past 2^31 and 2^32
PAD = 64               # canary words after each buffer


def _index_field(n, shift, bits, dtype, chunk=1 << 28):
    """t[i] = (i >> shift) & (2^bits - 1) as `dtype` (exact), built in chunks."""
    out = torch.empty(n + PAD, dtype=dtype, device=DEV)
    for a in range(0, n, chunk):
        b = min(n, a + chunk)
        i = torch.arange(a, b, dtype=torch.int64, device=DEV)
        out[a:b] = ((i >> shift) & ((1 << bits) - 1)).to(dtype)
    return out


def _all_equal_field(t, n, shift, bits, chunk=1 << 28):
    for a in range(0, n, chunk):
        b = min(n, a + chunk)
        i = torch.arange(a, b, dtype=torch.int64, device=DEV)
        want = ((i >> shift) & ((1 << bits) - 1)).to(torch.float32)
        if not torch.equal(t[a:b], want):
            bad = torch.nonzero(t[a:b] != want)[0].item() + a
            return bad
    return -1


@pytest.mark.parametrize("gdt", ["f32", "bf16"])
def test_accumulate_coverage_past_2_pow_31(gdt):
    """n = 2^31 + 17: the bucket zeroed by the fill kernel, then one
    accumulate of g[i] = a bit field of i, for fields that together name
    every index (fp32: 20 + 12 bits; bf16, exact up to 256: four bytes).
    Every element must equal its own index's field (each updated exactly
    once, from its own g) and the canary words after G stay untouched."""
    n = N64
    fields = [(0, 20), (20, 12)] if gdt == "f32" else [(0, 8), (8, 8), (16, 8), (24, 8)]
    tdt = torch.float32 if gdt == "f32" else torch.bfloat16
    G = torch.full((n + PAD,), 7.0, dtype=torch.float32, device=DEV)
    for shift, bits in fields:
        banner(f"accumulate n=2^31+17 g={gdt} field {shift}:{bits}")
        g = _index_field(n, shift, bits, tdt)
        g[n:] = 3.0
        lc.lc_zero_fill_f32(G, n)
        lc.chunk_accumulate_grad(G, g, lc.LC_BF16 if gdt == "bf16" else lc.LC_FP32, n)
        torch.cuda.synchronize()
        bad = _all_equal_field(G, n, shift, bits)
        assert bad < 0, f"element {bad} holds {G[bad].item()}"
        assert torch.all(G[n:] == 7.0)
        del g
    del G
    torch.cuda.empty_cache()


def test_adam_coverage_past_2_pow_31():
    """n = 2^31 + 17, bf16 gradient and bf16 cast. (1) Coverage: g = m = v = 0
    and weight decay 0.1 make the step p' = fl(p * c_wd) exactly (m' = v' = 0,
    the update term 0), so with p[i] a bit field of i every element of p and
    of the cast must hold its own index's value; two fields name every index.
    (2) Random p, m, v, g: elements at the head, the tail and around 2^31,
    plus a random sample, bit for bit against the oracle's AdamW. Canary
    words after every buffer stay untouched."""
    n = N64
    lr, b1, b2, eps, wd = 3e-4, 0.9, 0.95, 1e-8, 0.1
    c_wd = torch.tensor(np.float32(1.0 - lr * wd), device=DEV)
    m = torch.zeros(n + PAD, dtype=torch.float32, device=DEV)
    v = torch.zeros(n + PAD, dtype=torch.float32, device=DEV)
    g = torch.zeros(n + PAD, dtype=torch.bfloat16, device=DEV)
    out = torch.full((n + PAD,), 5.0, dtype=torch.bfloat16, device=DEV)
    for shift, bits in ((0, 20), (20, 12)):
        banner(f"adam n=2^31+17 coverage field {shift}:{bits}")
        p = _index_field(n, shift, bits, torch.float32)
        p[n:] = 9.0
        m.zero_(), v.zero_(), g.zero_()
        lc.shard_adam_step(p, m, v, g, lc.LC_BF16, out, n, lr, b1, b2, eps, wd, 1)
        torch.cuda.synchronize()
        for a in range(0, n, 1 << 28):
            b = min(n, a + (1 << 28))
            i = torch.arange(a, b, dtype=torch.int64, device=DEV)
            want = ((i >> shift) & ((1 << bits) - 1)).to(torch.float32) * c_wd
            assert torch.equal(p[a:b], want), (shift, a)
            assert torch.equal(out[a:b], want.to(torch.bfloat16)), (shift, a)
        assert torch.all(m[:n] == 0) and torch.all(v[:n] == 0)
        for t, c in ((p, 9.0), (m, 0.0), (v, 0.0), (out, 5.0)):
            assert torch.all(t[n:] == c)
        del p
    banner("adam n=2^31+17 sampled bit-exact")
    gen = torch.Generator(device=DEV)
    gen.manual_seed(12)
    p = torch.randn(n + PAD, generator=gen, device=DEV).mul_(0.02)
    m.normal_(0.0, 1e-3, generator=gen)
    v.normal_(0.0, 1e-3, generator=gen).square_()
    g.copy_(torch.randn(n + PAD, generator=gen, device=DEV).mul_(1e-3).to(torch.bfloat16))
    canary = [t[n:].clone() for t in (p, m, v, g, out)]
    # contiguous windows inside [0, n) read by plain slicing: the head, the
    # tail (which crosses 2^31: n - 64 = 2^31 - 47), just below 2^31, and
    # random places
    rng = np.random.default_rng(32)
    W = 64
    starts = sorted({0, n - W, (1 << 31) - 2 * W} |
                    {int(a) for a in rng.integers(0, n - W + 1, 400)})
    assert all(0 <= a and a + W <= n for a in starts)

    def windows(t):
        return np.concatenate([t[a:a + W].float().cpu().numpy() for a in starts])

    p0, m0, v0, g0 = (windows(t) for t in (p, m, v, g))
    for name, a in (("p", p0), ("m", m0), ("v", v0), ("g", g0)):
        assert np.all(np.isfinite(a)), f"non-finite {name} input at {np.nonzero(~np.isfinite(a))[0][:8]}"
    lc.shard_adam_step(p, m, v, g, lc.LC_BF16, out, n, lr, b1, b2, eps, wd, 7)
    torch.cuda.synchronize()
    pr, mr, vr = OP.adamw(p0, m0, v0, g0, lr, b1, b2, eps, wd, 7)
    pos = np.concatenate([np.arange(a, a + W) for a in starts])
    bad = {}
    for got, ref, name in ((p, pr, "p"), (m, mr, "m"), (v, vr, "v")):
        diff = windows(got).astype(np.float32).view(np.uint32) != ref.view(np.uint32)
        bad[name] = (int(diff[pos < (1 << 31)].sum()), int(diff[pos >= (1 << 31)].sum()))
    ob = np.concatenate([out[a:a + W].cpu().view(torch.int16).numpy().view(np.uint16)
                         for a in starts])
    bad["out"] = int((ob != OP.bf16_rne_bits(pr)).sum())
    print(f"mismatches (below 2^31, from 2^31) over {pos.size} elements: {bad}", flush=True)
    assert all(b == (0, 0) for k, b in bad.items() if k != "out") and bad["out"] == 0, bad
    for t, c in zip((p, m, v, g, out), canary):
        assert torch.equal(t[n:], c)
    del p, m, v, g, out
    torch.cuda.empty_cache()
