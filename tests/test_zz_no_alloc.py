"""The RMSNorm backward entry point that allocates nothing
(lc_rmsnorm_backward_noalloc) against the one that takes a caller's scratch
(lc_rmsnorm_backward), through the C-ABI: two calls in a row on one GPU, the
second smaller, each bit for bit equal (same kernels, same reduction order)
and within the RMSNorm tolerance of the oracle; sizes beyond the fixed array
are refused before anything is enqueued."""
import numpy as np
import pytest
import torch

from oracle import stage as OS
from paper_2606_11169_amd import libchunk as lc
from paper_2606_11169_amd.runner import require_gpu
from tests.gpu_util import DEV, banner, host, rel_err

pytestmark = pytest.mark.gpu

BF16, FP32 = lc.LC_BF16, lc.LC_FP32


def _case(rng, T, d):
    x = torch.from_numpy(rng.standard_normal((T, d)).astype(np.float32)).to(DEV)
    g = torch.from_numpy((1 + 0.1 * rng.standard_normal(d)).astype(np.float32)).to(DEV)
    g = g.to(torch.bfloat16)
    dn = torch.from_numpy(rng.standard_normal((T, d)).astype(np.float32)).to(DEV)
    dres = torch.from_numpy(rng.standard_normal((T, d)).astype(np.float32)).to(DEV)
    rstd = torch.empty(T, dtype=torch.float32, device=DEV)
    n = torch.empty((T, d), dtype=torch.bfloat16, device=DEV)
    lc.lc_rmsnorm_forward(T, d, x, g, 1e-5, n, rstd, FP32, BF16, BF16)
    dg0 = torch.from_numpy(rng.standard_normal(d).astype(np.float32)).to(DEV)
    return x, g, dn, dres, rstd, dg0


def _outputs(T, d):
    return (torch.full((T, d), float("nan"), dtype=torch.float32, device=DEV),
            torch.full((T, d), float("nan"), dtype=torch.bfloat16, device=DEV))


def test_rmsnorm_backward_noalloc_matches_the_scratch_entry_point():
    require_gpu()
    rng = np.random.default_rng(51)
    for T, d in ((16384, 4096), (300, 512)):   # the fixed array's limit, then smaller
        banner(f"rmsnorm backward no-alloc T={T} d={d}")
        x, g, dn, dres, rstd, dg0 = _case(rng, T, d)
        sb = lc.lc_rmsnorm_scratch_bytes(T, d)
        scratch = torch.empty(sb, dtype=torch.uint8, device=DEV)
        dx_a, cp_a = _outputs(T, d)
        dg_a = dg0.clone()
        lc.lc_rmsnorm_backward(T, d, dn, x, rstd, g, dres, dx_a, dg_a, scratch, sb, FP32, FP32,
                               BF16, FP32, FP32, dx_copy=cp_a)
        dx_b, cp_b = _outputs(T, d)
        dg_b = dg0.clone()
        lc.lc_rmsnorm_backward_noalloc(T, d, dn, x, rstd, g, dres, dx_b, dg_b, FP32, FP32, BF16,
                                       FP32, FP32, dx_copy=cp_b)
        torch.cuda.synchronize()
        assert torch.equal(dx_a, dx_b) and torch.equal(cp_a, cp_b)
        assert torch.equal(dg_a, dg_b)
        # and the oracle's RMSNorm backward (the entry point's own tolerance)
        dx_ref, dg_ref = OS.rmsnorm_backward(host(dn), host(x), host(rstd)[:, None], host(g))
        assert rel_err(host(dx_b), host(dres) + dx_ref) <= 1e-5
        assert rel_err(host(dg_b), host(dg0) + dg_ref) <= 1e-5
        del scratch


def test_rmsnorm_backward_noalloc_refuses_sizes_beyond_its_array():
    require_gpu()
    T, d = 16384 + 16, 4096   # one 16-row block more than the array holds
    banner(f"rmsnorm backward no-alloc refusal T={T} d={d}")
    x = torch.zeros((T, d), dtype=torch.float32, device=DEV)
    g = torch.ones(d, dtype=torch.bfloat16, device=DEV)
    rstd = torch.ones(T, dtype=torch.float32, device=DEV)
    dx = torch.full((T, d), 3.0, dtype=torch.float32, device=DEV)
    dg = torch.full((d,), 5.0, dtype=torch.float32, device=DEV)
    with pytest.raises(lc.LibchunkError) as e:
        lc.lc_rmsnorm_backward_noalloc(T, d, x, x, rstd, g, None, dx, dg, FP32, FP32, BF16,
                                       FP32, FP32)
    assert e.value.status == lc.LC_ERR_WORKSPACE and "fixed" in str(e.value)
    torch.cuda.synchronize()
    assert torch.all(dx == 3.0) and torch.all(dg == 5.0)   # nothing ran
    # without a gain gradient no scratch is needed, whatever the size
    lc.lc_rmsnorm_backward_noalloc(T, d, x, x, rstd, g, None, dx, None, FP32, FP32, BF16,
                                   FP32, FP32)
    torch.cuda.synchronize()
    assert torch.all(dx == 0.0)
