"""Argument checking of the op entry points (include/libchunk_ops.h and the
buffer calls of include/libchunk.h), without a GPU.

Every call below breaks one documented rule and must return its status from
the host-side checks, before anything is enqueued; addresses are aligned
fakes that are never dereferenced. Zero-length buffer calls are no-ops that
return LC_OK without touching the device. The module runs only on hosts
without a GPU: there a check that stopped firing reaches the launch, which
fails with LC_ERR_HIP and the test reports it; on a GPU host the same call
would launch a kernel on the fake addresses.
"""
import pytest
import torch

from paper_2606_11169_amd import libchunk as lc

pytestmark = pytest.mark.skipif(torch.cuda.device_count() > 0,
                                reason="fake device addresses: host-only checks")

A = 1 << 24          # 16-byte aligned fake device addresses, never read
B = 2 << 24
Cc = 3 << 24
D = 4 << 24
E = 5 << 24
BF16, FP16, FP32 = lc.LC_BF16, lc.LC_FP16, lc.LC_FP32


def status_of(fn, *a, **k):
    try:
        fn(*a, **k)
    except lc.LibchunkError as e:
        return e.status
    return lc.LC_OK


def gemm(**over):
    args = dict(dtype=BF16, epilogue=lc.LC_EPI_STORE, M=256, N=256, K=256, A=A, lda=256,
                a_kmajor=1, B=B, ldb=256, b_kmajor=1, Cm=Cc, ldc=256)
    args.update(over)
    return status_of(lc.lc_gemm, **args)


@pytest.mark.parametrize("over,want", [
    (dict(K=0), lc.LC_ERR_INVALID_ARG),
    (dict(A=None), lc.LC_ERR_INVALID_ARG),
    (dict(A=A + 8), lc.LC_ERR_INVALID_ARG),
    (dict(epilogue=9), lc.LC_ERR_INVALID_ARG),
    (dict(lda=128), lc.LC_ERR_INVALID_ARG),
    (dict(ldc=128), lc.LC_ERR_INVALID_ARG),
    (dict(N=260, ldc=264), lc.LC_ERR_UNSUPPORTED),
    (dict(dtype=FP16), lc.LC_ERR_INVALID_ARG),
    (dict(epilogue=lc.LC_EPI_RESIDUAL, R=None), lc.LC_ERR_INVALID_ARG),
    (dict(group_mode=lc.LC_GROUP_ROWS, n_groups=0, group_offsets=D), lc.LC_ERR_INVALID_ARG),
    (dict(group_mode=lc.LC_GROUP_ROWS, n_groups=65, group_offsets=D), lc.LC_ERR_INVALID_ARG),
    (dict(group_mode=lc.LC_GROUP_ROWS, n_groups=2, group_offsets=D,
          epilogue=lc.LC_EPI_RESIDUAL, R=E, ldr=256), lc.LC_ERR_UNSUPPORTED),
    # an operand spanning 2 GiB: the buffer offsets are 32-bit
    (dict(M=32768, K=32768, lda=32768, ldb=32768), lc.LC_ERR_UNSUPPORTED),
], ids=["K0", "nullA", "unalignedA", "epilogue", "lda", "ldc", "N%8", "dtype", "residual",
        "groups0", "groups65", "grouped_residual", "2GiB"])
def test_gemm_argument_errors(over, want):
    assert gemm(**over) == want


def test_rmsnorm_argument_errors():
    fwd = dict(T=16, d=256, x=A, g=B, eps=1e-5, n=Cc, rstd=D, x_dtype=FP32, w_dtype=BF16,
               out_dtype=BF16)
    assert status_of(lc.lc_rmsnorm_forward, **{**fwd, "T": 0}) == lc.LC_ERR_INVALID_ARG
    assert status_of(lc.lc_rmsnorm_forward, **{**fwd, "d": 100}) == lc.LC_ERR_UNSUPPORTED
    assert status_of(lc.lc_rmsnorm_forward, **{**fwd, "x": None}) == lc.LC_ERR_INVALID_ARG
    assert status_of(lc.lc_rmsnorm_forward, **{**fwd, "x_dtype": 7}) == lc.LC_ERR_INVALID_ARG
    need = lc.lc_rmsnorm_scratch_bytes(16, 256)
    bwd = dict(T=16, d=256, dn=A, x=B, rstd=Cc, g=D, dres=None, dx=E, dg_accum=E + (1 << 20),
               scratch=E + (2 << 20), scratch_bytes=need - 4, dn_dtype=FP32, x_dtype=FP32,
               w_dtype=BF16, dres_dtype=FP32, out_dtype=FP32)
    assert status_of(lc.lc_rmsnorm_backward, **bwd) == lc.LC_ERR_WORKSPACE


def attn_fwd(**over):
    a = dict(dtype=FP16, o_dtype=BF16, B=1, S=256, H=4, hd=128, q=A, k=A + 1024, v=A + 2048,
             ld_qkv=3 * 512, o=B, ld_o=512, lse=Cc)
    a.update(over)
    return status_of(lc.lc_attention_forward, **a)


def test_attention_argument_errors():
    assert attn_fwd(hd=64, ld_qkv=768, ld_o=256) == lc.LC_ERR_UNSUPPORTED  # matrix cores: 128
    assert attn_fwd(S=200) == lc.LC_ERR_UNSUPPORTED                         # S % 128
    assert attn_fwd(Hkv=3) == lc.LC_ERR_INVALID_ARG                         # does not divide H
    assert attn_fwd(ld_qkv=256) == lc.LC_ERR_INVALID_ARG                    # ld < H*hd
    assert attn_fwd(o_dtype=FP16) == lc.LC_ERR_UNSUPPORTED
    assert attn_fwd(dtype=FP32, o_dtype=FP32, hd=130, ld_o=520) == lc.LC_ERR_UNSUPPORTED
    assert attn_fwd(q=None) == lc.LC_ERR_INVALID_ARG
    need = lc.lc_attention_scratch_bytes(1, 256, 4, 2)
    assert need > lc.lc_attention_scratch_bytes(1, 256, 4)  # the grouped dk/dv shares
    st = status_of(lc.lc_attention_backward, FP16, BF16, 1, 256, 4, 128, A, A + 1024,
                   A + 1536, 2048, B, Cc, 512, D, E, E + 1024, E + 1536, 2048, None, None,
                   E + (1 << 20), need - 256, Hkv=2)
    assert st == lc.LC_ERR_WORKSPACE


def test_qk_norm_argument_errors():
    fwd = dict(T=8, H=4, Hkv=2, hd=128, seq_len=8, eps=1e-6, qk=A, ld=1024, raw=B, rstd=Cc,
               gq=D, gk=D + 256, x_dtype=FP16, w_dtype=BF16, rope_cos=E, rope_sin=E + 4096)
    assert status_of(lc.lc_qk_norm_rope_forward, **{**fwd, "hd": 48}) == lc.LC_ERR_UNSUPPORTED
    assert status_of(lc.lc_qk_norm_rope_forward, **{**fwd, "x_dtype": BF16}) == lc.LC_ERR_INVALID_ARG
    assert status_of(lc.lc_qk_norm_rope_forward, **{**fwd, "ld": 512}) == lc.LC_ERR_INVALID_ARG
    assert status_of(lc.lc_qk_norm_rope_forward, **{**fwd, "rope_cos": None}) == lc.LC_ERR_INVALID_ARG
    need = lc.lc_qk_norm_scratch_bytes(8, 128)
    assert need == 2 * 2 * 128 * 4  # two 4-token blocks of q and k gain partials
    bwd = dict(T=8, H=4, Hkv=2, hd=128, seq_len=8, eps=1e-6, raw=B, rstd=Cc, gq=D, gk=D + 256,
               x_dtype=FP16, w_dtype=BF16, dqk=A, ld_d=1024, d_dtype=BF16, dgq=E, dgk=E + 512,
               scratch=E + 4096, scratch_bytes=need - 4)
    assert status_of(lc.lc_qk_norm_rope_backward, **bwd) == lc.LC_ERR_WORKSPACE
    assert status_of(lc.lc_qk_norm_rope_backward, **{**bwd, "dgq": None}) == lc.LC_ERR_INVALID_ARG


def test_buffer_call_errors_and_empty_calls():
    assert status_of(lc.chunk_accumulate_grad, A, A, FP32, 1024) == lc.LC_ERR_INVALID_ARG
    assert status_of(lc.chunk_accumulate_grad, A + 4, B, FP32, 1024) == lc.LC_ERR_INVALID_ARG
    assert status_of(lc.chunk_accumulate_grad, A, B, 7, 1024) == lc.LC_ERR_INVALID_ARG
    assert status_of(lc.chunk_accumulate_grad, A, B, FP32, 0) == lc.LC_OK
    adam = (A, B, Cc, D, BF16, E, 1024, 1e-3, 0.9, 0.999, 1e-8, 0.0)
    assert status_of(lc.shard_adam_step, *adam, 0) == lc.LC_ERR_INVALID_ARG  # step >= 1
    assert status_of(lc.shard_adam_step, A, None, Cc, D, BF16, E, 1024, 1e-3, 0.9, 0.999, 1e-8,
                     0.0, 1) == lc.LC_ERR_INVALID_ARG
    assert status_of(lc.shard_adam_step, A, B, Cc, D, 9, E, 1024, 1e-3, 0.9, 0.999, 1e-8, 0.0,
                     1) == lc.LC_ERR_INVALID_ARG
    assert status_of(lc.shard_adam_step, A, B, Cc, D, BF16, E, 0, 1e-3, 0.9, 0.999, 1e-8, 0.0,
                     1) == lc.LC_OK
    assert status_of(lc.lc_zero_fill_f32, A + 4, 16) == lc.LC_ERR_INVALID_ARG
    assert status_of(lc.lc_zero_fill_f32, A, 0) == lc.LC_OK


def test_moe_argument_errors():
    assert status_of(lc.lc_moe_route, 16, 64, 1, A, B, Cc, D, BF16, BF16) == lc.LC_ERR_INVALID_ARG
    assert status_of(lc.lc_moe_route, 16, 64, 65, A, B, Cc, D, BF16, BF16) == lc.LC_ERR_INVALID_ARG
    assert status_of(lc.lc_moe_route, 16, 60, 4, A, B, Cc, D, BF16, BF16) == lc.LC_ERR_UNSUPPORTED
    assert status_of(lc.lc_moe_dispatch, 16, 4, None, B, Cc, D, E, E + 4096) == lc.LC_ERR_INVALID_ARG
