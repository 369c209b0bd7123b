"""ctypes binding of libchunk (include/libchunk.h, include/libchunk_ops.h).

Argument marshalling only: every function forwards to the C entry point of
the same name; all computation happens in the HIP kernels behind it. Device
buffers are passed as integers (device addresses) or as torch tensors (their
data_ptr()); streams as integers (a hipStream_t) or torch streams. A negative
status raises LibchunkError carrying lc_last_error().

The shared library must have been built (``python -m
paper_2606_11169_amd.build``); importing works without it, the first call
raises.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import List, Sequence, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "_lib", "libchunk.so")

LC_OK = 0
LC_ERR_INVALID_ARG = -1
LC_ERR_UNSUPPORTED = -2
LC_ERR_BAD_ORDER = -3
LC_ERR_STASH_FULL = -4
LC_ERR_STATE = -5
LC_ERR_WORKSPACE = -6
LC_ERR_HIP = -7
STATUS_NAMES = {0: "OK", -1: "INVALID_ARG", -2: "UNSUPPORTED", -3: "BAD_ORDER",
                -4: "STASH_FULL", -5: "STATE", -6: "WORKSPACE", -7: "HIP"}

LC_FP32, LC_BF16, LC_FP16 = 0, 1, 2
LC_PASS_F, LC_PASS_B, LC_PASS_BI, LC_PASS_BW = 0, 1, 2, 3
LC_ORDER_WITH_NEXT = 0x100
(LC_T_WQ, LC_T_WK, LC_T_WV, LC_T_WO, LC_T_G1, LC_T_W1, LC_T_W3, LC_T_W2, LC_T_G2,
 LC_T_WR, LC_T_QN, LC_T_KN) = range(12)
(LC_EPI_STORE, LC_EPI_STORE_F32, LC_EPI_ACCUM_F32, LC_EPI_RESIDUAL, LC_EPI_ROPE,
 LC_EPI_SWIGLU, LC_EPI_SWIGLU_BWD) = range(7)
LC_GROUP_NONE, LC_GROUP_ROWS, LC_GROUP_K = 0, 1, 2


class LibchunkError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"libchunk {STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class lc_stage_desc(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("head_dim", C.c_int32), ("d_ff", C.c_int32), ("n_experts", C.c_int32),
                ("top_k", C.c_int32), ("d_ff_expert", C.c_int32), ("seq_len", C.c_int32),
                ("micro_batch", C.c_int32), ("rms_eps", C.c_float), ("rope_base", C.c_float),
                ("causal", C.c_int32), ("compute_dtype", C.c_int32),
                ("n_kv_heads", C.c_int32), ("qk_norm", C.c_int32)]


class lc_order_entry(C.Structure):
    _fields_ = [("mb", C.c_int32), ("pass_", C.c_int32)]


class lc_order(C.Structure):
    _fields_ = [("num_microbatches", C.c_int32), ("n_entries", C.c_int32),
                ("entries", C.POINTER(lc_order_entry))]


class lc_microbatch_desc(C.Structure):
    _fields_ = [("mb", C.c_int32), ("reserved", C.c_int32), ("x", C.c_void_p),
                ("y", C.c_void_p), ("dy", C.c_void_p), ("dx", C.c_void_p)]


class lc_param_bufs(C.Structure):
    _fields_ = [("w", C.c_void_p), ("grad", C.c_void_p)]


class lc_zero_bufs(C.Structure):
    _fields_ = [("level", C.c_int32), ("n_w_shards", C.c_int32), ("grad_shard", C.c_void_p),
                ("shard_offset", C.c_size_t), ("shard_len", C.c_size_t),
                ("grad_full", C.c_void_p), ("w_shards", C.POINTER(C.c_void_p)),
                ("w_shard_lens", C.POINTER(C.c_size_t)), ("w_full", C.c_void_p)]


class lc_adam_hparams(C.Structure):
    _fields_ = [("lr", C.c_float), ("beta1", C.c_float), ("beta2", C.c_float),
                ("eps", C.c_float), ("weight_decay", C.c_float), ("reserved", C.c_int32),
                ("step", C.c_int64)]


class lc_gemm_args(C.Structure):
    _fields_ = [("dtype", C.c_int32), ("epilogue", C.c_int32),
                ("c_dtype", C.c_int32), ("r_dtype", C.c_int32), ("aux_dtype", C.c_int32),
                ("reserved0", C.c_int32),
                ("M", C.c_int64), ("N", C.c_int64), ("K", C.c_int64),
                ("A", C.c_void_p), ("lda", C.c_int64), ("a_kmajor", C.c_int32),
                ("b_kmajor", C.c_int32), ("B", C.c_void_p), ("ldb", C.c_int64),
                ("C", C.c_void_p), ("ldc", C.c_int64),
                ("R", C.c_void_p), ("ldr", C.c_int64),
                ("aux0", C.c_void_p), ("aux1", C.c_void_p), ("ld_aux", C.c_int64),
                ("rope_cos", C.c_void_p), ("rope_sin", C.c_void_p),
                ("rope_seq", C.c_int32), ("rope_cols", C.c_int32), ("head_dim", C.c_int32),
                ("reserved1", C.c_int32),
                ("group_mode", C.c_int32), ("n_groups", C.c_int32),
                ("group_offsets", C.c_void_p), ("group_stride_b", C.c_int64),
                ("group_stride_c", C.c_int64)]


class lc_moe_args(C.Structure):
    _fields_ = [("T", C.c_int64), ("d", C.c_int32), ("E", C.c_int32),
                ("n_dtype", C.c_int32), ("w_dtype", C.c_int32),
                ("n", C.c_void_p), ("wr", C.c_void_p), ("sel", C.c_void_p), ("w", C.c_void_p),
                ("offsets", C.c_void_p), ("perm", C.c_void_p), ("wrow", C.c_void_p),
                ("rowpos", C.c_void_p)]


class lc_norm_args(C.Structure):
    _fields_ = [("T", C.c_int64), ("d", C.c_int64), ("eps", C.c_float),
                ("x_dtype", C.c_int32), ("w_dtype", C.c_int32), ("out_dtype", C.c_int32),
                ("dn_dtype", C.c_int32), ("dres_dtype", C.c_int32),
                ("x", C.c_void_p), ("g", C.c_void_p), ("n", C.c_void_p), ("rstd", C.c_void_p),
                ("dn", C.c_void_p), ("dres", C.c_void_p), ("dx", C.c_void_p),
                ("dx_copy", C.c_void_p), ("dg_accum", C.c_void_p),
                ("scratch", C.c_void_p), ("scratch_bytes", C.c_size_t)]


class lc_attn_args(C.Structure):
    _fields_ = [("dtype", C.c_int32), ("o_dtype", C.c_int32),
                ("B", C.c_int32), ("S", C.c_int32), ("H", C.c_int32), ("hd", C.c_int32),
                ("q", C.c_void_p), ("k", C.c_void_p), ("v", C.c_void_p), ("ld_qkv", C.c_int64),
                ("o", C.c_void_p), ("ld_o", C.c_int64), ("lse", C.c_void_p),
                ("dout", C.c_void_p), ("dq", C.c_void_p), ("dk", C.c_void_p), ("dv", C.c_void_p),
                ("ld_dqkv", C.c_int64), ("rope_cos", C.c_void_p), ("rope_sin", C.c_void_p),
                ("scratch", C.c_void_p), ("scratch_bytes", C.c_size_t),
                ("Hkv", C.c_int32), ("reserved", C.c_int32),
                ("qkv_bf16", C.c_void_p), ("ld_qkv_bf16", C.c_int64)]


class lc_qknorm_args(C.Structure):
    _fields_ = [("T", C.c_int64), ("H", C.c_int32), ("Hkv", C.c_int32), ("hd", C.c_int32),
                ("seq_len", C.c_int32), ("eps", C.c_float), ("x_dtype", C.c_int32),
                ("w_dtype", C.c_int32), ("d_dtype", C.c_int32), ("qk", C.c_void_p),
                ("ld", C.c_int64), ("raw", C.c_void_p), ("rstd", C.c_void_p),
                ("gq", C.c_void_p), ("gk", C.c_void_p), ("rope_cos", C.c_void_p),
                ("rope_sin", C.c_void_p), ("dqk", C.c_void_p), ("ld_d", C.c_int64),
                ("dgq", C.c_void_p), ("dgk", C.c_void_p), ("store_dg", C.c_int32),
                ("reserved", C.c_int32), ("scratch", C.c_void_p), ("scratch_bytes", C.c_size_t)]


# name -> (restype, argtypes)
_SIGS = {
    "lc_last_error": (C.c_char_p, []),
    "lc_param_count": (C.c_int, [C.POINTER(lc_stage_desc), C.POINTER(C.c_size_t)]),
    "lc_param_offset": (C.c_int, [C.POINTER(lc_stage_desc), C.c_int32, C.c_int32, C.c_int32,
                                  C.POINTER(C.c_size_t), C.POINTER(C.c_int64)]),
    "lc_order_1f1b": (C.c_int, [C.c_int32, C.c_int32, C.c_int32, C.POINTER(lc_order_entry),
                                C.c_int32, C.POINTER(C.c_int32)]),
    "lc_order_1f1b_overlap": (C.c_int, [C.c_int32, C.c_int32, C.c_int32,
                                        C.POINTER(lc_order_entry), C.c_int32,
                                        C.POINTER(C.c_int32)]),
    "lc_order_1f1b_split": (C.c_int, [C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                      C.POINTER(lc_order_entry), C.c_int32,
                                      C.POINTER(C.c_int32)]),
    "lc_order_1f1b_split_overlap": (C.c_int, [C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                              C.POINTER(lc_order_entry), C.c_int32,
                                              C.POINTER(C.c_int32)]),
    "lc_order_validate": (C.c_int, [C.POINTER(lc_order), C.c_int32, C.POINTER(C.c_int32)]),
    "lc_order_validate_split": (C.c_int, [C.POINTER(lc_order), C.c_int32, C.c_int32,
                                          C.POINTER(C.c_int32), C.POINTER(C.c_int32)]),
    "lc_workspace_bytes": (C.c_int, [C.POINTER(lc_stage_desc), C.c_int32, C.POINTER(C.c_size_t)]),
    "lc_workspace_bytes_split": (C.c_int, [C.POINTER(lc_stage_desc), C.c_int32, C.c_int32,
                                           C.POINTER(C.c_size_t)]),
    "lc_stage_create": (C.c_int, [C.POINTER(lc_stage_desc), C.c_void_p, C.c_size_t, C.c_int32,
                                  C.c_void_p, C.POINTER(C.c_void_p)]),
    "lc_stage_create_split": (C.c_int, [C.POINTER(lc_stage_desc), C.c_void_p, C.c_size_t,
                                        C.c_int32, C.c_int32, C.c_void_p,
                                        C.POINTER(C.c_void_p)]),
    "lc_stage_destroy": (C.c_int, [C.c_void_p]),
    "chunk_forward": (C.c_int, [C.c_void_p, C.POINTER(lc_param_bufs),
                                C.POINTER(lc_microbatch_desc), C.c_void_p]),
    "chunk_backward": (C.c_int, [C.c_void_p, C.POINTER(lc_param_bufs),
                                 C.POINTER(lc_microbatch_desc), C.c_void_p]),
    "chunk_backward_input": (C.c_int, [C.c_void_p, C.POINTER(lc_param_bufs),
                                       C.POINTER(lc_microbatch_desc), C.c_void_p]),
    "chunk_backward_weight": (C.c_int, [C.c_void_p, C.POINTER(lc_param_bufs),
                                        C.POINTER(lc_microbatch_desc), C.c_void_p]),
    "lc_run_order": (C.c_int, [C.c_void_p, C.POINTER(lc_param_bufs), C.POINTER(lc_order),
                               C.POINTER(lc_microbatch_desc), C.c_void_p]),
    "lc_run_order_zero": (C.c_int, [C.c_void_p, C.POINTER(lc_param_bufs),
                                    C.POINTER(lc_zero_bufs), C.POINTER(lc_order),
                                    C.POINTER(lc_microbatch_desc), C.c_void_p]),
    "lc_zero_fill_f32": (C.c_int, [C.c_void_p, C.c_size_t, C.c_void_p]),
    "lc_run_order_overlap": (C.c_int, [C.c_void_p, C.POINTER(lc_param_bufs),
                                       C.POINTER(lc_order), C.POINTER(lc_microbatch_desc),
                                       C.c_void_p, C.c_void_p]),
    "chunk_accumulate_grad": (C.c_int, [C.c_void_p, C.c_void_p, C.c_int32, C.c_size_t,
                                        C.c_void_p]),
    "shard_adam_step": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32,
                                  C.c_void_p, C.c_size_t, C.POINTER(lc_adam_hparams),
                                  C.c_void_p]),
    "lc_gemm": (C.c_int, [C.POINTER(lc_gemm_args), C.c_void_p]),
    "lc_rmsnorm_forward": (C.c_int, [C.POINTER(lc_norm_args), C.c_void_p]),
    "lc_rmsnorm_backward": (C.c_int, [C.POINTER(lc_norm_args), C.c_void_p]),
    "lc_rmsnorm_scratch_bytes": (C.c_size_t, [C.c_int64, C.c_int64]),
    "lc_rmsnorm_backward_noalloc": (C.c_int, [C.POINTER(lc_norm_args), C.c_void_p]),
    "lc_attention_forward": (C.c_int, [C.POINTER(lc_attn_args), C.c_void_p]),
    "lc_attention_backward": (C.c_int, [C.POINTER(lc_attn_args), C.c_void_p]),
    "lc_attention_scratch_bytes": (C.c_size_t, [C.c_int32, C.c_int32, C.c_int32]),
    "lc_attention_scratch_bytes_kv": (C.c_size_t, [C.c_int32, C.c_int32, C.c_int32, C.c_int32]),
    "lc_qk_norm_rope_forward": (C.c_int, [C.POINTER(lc_qknorm_args), C.c_void_p]),
    "lc_qk_norm_rope_backward": (C.c_int, [C.POINTER(lc_qknorm_args), C.c_void_p]),
    "lc_qk_norm_scratch_bytes": (C.c_size_t, [C.c_int64, C.c_int32]),
    "lc_cast_bf16": (C.c_int, [C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]),
    "lc_moe_route": (C.c_int, [C.POINTER(lc_moe_args), C.c_void_p]),
    "lc_moe_dispatch": (C.c_int, [C.POINTER(lc_moe_args), C.c_void_p]),
    "lc_stage_timer_enable": (C.c_int, [C.c_void_p, C.c_int32]),
    "lc_stage_timer_read": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32,
                                      C.c_void_p]),
    "lc_stage_moe_routing": (C.c_int, [C.c_void_p, C.c_int32, C.c_int32, C.c_void_p,
                                       C.c_void_p]),
}

EXPORTED = tuple(_SIGS)
_lib = None


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2606_11169_amd.build`")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(st: int) -> int:
    if st < 0:
        raise LibchunkError(st, lib().lc_last_error().decode(errors="replace"))
    return st


def ptr(x) -> int:
    """Device address of a torch tensor, or an int / None passed through."""
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


def stream_ptr(s) -> int:
    if s is None:
        return 0
    if isinstance(s, int):
        return s
    return int(s.cuda_stream)


def _vp(x):
    return C.c_void_p(ptr(x) or None)


# ------------------------------------------------------------------ host-only

def make_desc(n_layers, d_model, n_heads, head_dim, d_ff, seq_len, micro_batch, bf16,
              n_experts=0, top_k=0, d_ff_expert=0, rms_eps=1e-5, rope_base=10000.0,
              causal=1, n_kv_heads=0, qk_norm=False) -> lc_stage_desc:
    return lc_stage_desc(n_layers, d_model, n_heads, head_dim, d_ff, n_experts, top_k,
                         d_ff_expert, seq_len, micro_batch, rms_eps, rope_base, causal,
                         LC_BF16 if bf16 else LC_FP32, n_kv_heads, 1 if qk_norm else 0)


def desc_of_config(cfg) -> lc_stage_desc:
    """The descriptor of a synth.StageConfig."""
    return make_desc(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.head_dim, cfg.d_ff,
                     cfg.seq_len, cfg.micro_batch, cfg.bf16, n_experts=cfg.n_experts,
                     top_k=cfg.top_k, d_ff_expert=cfg.d_ff_expert, rms_eps=cfg.rms_eps,
                     rope_base=cfg.rope_base, n_kv_heads=cfg.n_kv_heads, qk_norm=cfg.qk_norm)


def lc_param_count(desc: lc_stage_desc) -> int:
    n = C.c_size_t()
    _check(lib().lc_param_count(C.byref(desc), C.byref(n)))
    return n.value


def lc_param_offset(desc, layer, tensor_id, expert=0) -> Tuple[int, Tuple[int, int]]:
    off = C.c_size_t()
    shape = (C.c_int64 * 2)()
    _check(lib().lc_param_offset(C.byref(desc), layer, tensor_id, expert, C.byref(off), shape))
    return off.value, (shape[0], shape[1])


def lc_order_1f1b(M, P, s) -> List[Tuple[int, int]]:
    buf = (lc_order_entry * max(1, 2 * M))()
    n = C.c_int32()
    _check(lib().lc_order_1f1b(M, P, s, buf, 2 * M, C.byref(n)))
    return [(buf[i].mb, buf[i].pass_) for i in range(n.value)]


def lc_order_1f1b_overlap(M, P, s) -> List[Tuple[int, int]]:
    buf = (lc_order_entry * max(1, 2 * M))()
    n = C.c_int32()
    _check(lib().lc_order_1f1b_overlap(M, P, s, buf, 2 * M, C.byref(n)))
    return [(buf[i].mb, buf[i].pass_) for i in range(n.value)]


def lc_order_1f1b_split(M, P, s, w_delay) -> List[Tuple[int, int]]:
    buf = (lc_order_entry * max(1, 3 * M))()
    n = C.c_int32()
    _check(lib().lc_order_1f1b_split(M, P, s, w_delay, buf, 3 * M, C.byref(n)))
    return [(buf[i].mb, buf[i].pass_) for i in range(n.value)]


def lc_order_1f1b_split_overlap(M, P, s, w_delay) -> List[Tuple[int, int]]:
    buf = (lc_order_entry * max(1, 3 * M))()
    n = C.c_int32()
    _check(lib().lc_order_1f1b_split_overlap(M, P, s, w_delay, buf, 3 * M, C.byref(n)))
    return [(buf[i].mb, buf[i].pass_) for i in range(n.value)]


def make_order(entries: Sequence[Tuple[int, int]], M: int):
    arr = (lc_order_entry * max(1, len(entries)))(*[lc_order_entry(m, p) for m, p in entries])
    o = lc_order(M, len(entries), C.cast(arr, C.POINTER(lc_order_entry)))
    o._keep = arr
    return o


def lc_order_validate(entries, M, max_in_flight) -> Tuple[int, int]:
    """Returns (status, peak) without raising for Order errors."""
    o = make_order(entries, M)
    pk = C.c_int32()
    st = lib().lc_order_validate(C.byref(o), max_in_flight, C.byref(pk))
    if st not in (LC_OK, LC_ERR_BAD_ORDER, LC_ERR_STASH_FULL):
        _check(st)
    return st, pk.value


def lc_order_validate_split(entries, M, max_in_flight, max_w_pending) -> Tuple[int, int, int]:
    """Returns (status, peak, peak_w) without raising for Order errors."""
    o = make_order(entries, M)
    pk, pkw = C.c_int32(), C.c_int32()
    st = lib().lc_order_validate_split(C.byref(o), max_in_flight, max_w_pending, C.byref(pk),
                                       C.byref(pkw))
    if st not in (LC_OK, LC_ERR_BAD_ORDER, LC_ERR_STASH_FULL):
        _check(st)
    return st, pk.value, pkw.value


def lc_workspace_bytes(desc, max_in_flight, max_w_pending=0) -> int:
    n = C.c_size_t()
    _check(lib().lc_workspace_bytes_split(C.byref(desc), max_in_flight, max_w_pending,
                                          C.byref(n)))
    return n.value


def lc_rmsnorm_scratch_bytes(T, d) -> int:
    return int(lib().lc_rmsnorm_scratch_bytes(T, d))


def lc_attention_scratch_bytes(B, S, H, Hkv=0) -> int:
    if Hkv:
        return int(lib().lc_attention_scratch_bytes_kv(B, S, H, Hkv))
    return int(lib().lc_attention_scratch_bytes(B, S, H))


def lc_qk_norm_scratch_bytes(T, hd) -> int:
    return int(lib().lc_qk_norm_scratch_bytes(T, hd))


# ------------------------------------------------------------------ stage

class Stage:
    """Owns an lc_stage handle (host memory); the workspace belongs to the caller."""

    def __init__(self, desc, workspace, ws_bytes, max_in_flight, stream=None, max_w_pending=0):
        h = C.c_void_p()
        _check(lib().lc_stage_create_split(C.byref(desc), _vp(workspace), ws_bytes,
                                           max_in_flight, max_w_pending,
                                           C.c_void_p(stream_ptr(stream) or None), C.byref(h)))
        self.handle = h
        self.desc = desc

    def close(self):
        if self.handle:
            lib().lc_stage_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def lc_stage_create(desc, workspace, ws_bytes, max_in_flight, stream=None,
                    max_w_pending=0) -> Stage:
    return Stage(desc, workspace, ws_bytes, max_in_flight, stream, max_w_pending)


def _mb(mb, x=None, y=None, dy=None, dx=None):
    return lc_microbatch_desc(mb, 0, _vp(x), _vp(y), _vp(dy), _vp(dx))


def chunk_forward(stage: Stage, w, grad, mb, x, y, stream=None):
    pb = lc_param_bufs(_vp(w), _vp(grad))
    d = _mb(mb, x=x, y=y)
    return _check(lib().chunk_forward(stage.handle, C.byref(pb), C.byref(d),
                                      C.c_void_p(stream_ptr(stream) or None)))


def chunk_backward(stage: Stage, w, grad, mb, dy, dx, stream=None):
    pb = lc_param_bufs(_vp(w), _vp(grad))
    d = _mb(mb, dy=dy, dx=dx)
    return _check(lib().chunk_backward(stage.handle, C.byref(pb), C.byref(d),
                                       C.c_void_p(stream_ptr(stream) or None)))


def chunk_backward_input(stage: Stage, w, mb, dy, dx, stream=None):
    pb = lc_param_bufs(_vp(w), _vp(None))
    d = _mb(mb, dy=dy, dx=dx)
    return _check(lib().chunk_backward_input(stage.handle, C.byref(pb), C.byref(d),
                                             C.c_void_p(stream_ptr(stream) or None)))


def chunk_backward_weight(stage: Stage, w, grad, mb, stream=None):
    pb = lc_param_bufs(_vp(w), _vp(grad))
    d = _mb(mb)
    return _check(lib().chunk_backward_weight(stage.handle, C.byref(pb), C.byref(d),
                                              C.c_void_p(stream_ptr(stream) or None)))


def lc_run_order(stage: Stage, w, grad, entries, xs, ys, dys, dxs, stream=None,
                 aux_stream=None):
    """Runs an Order; with aux_stream given, through lc_run_order_overlap."""
    M = len(xs)
    o = make_order(entries, M)
    arr = (lc_microbatch_desc * M)(*[_mb(i, xs[i], ys[i], dys[i], dxs[i]) for i in range(M)])
    pb = lc_param_bufs(_vp(w), _vp(grad))
    s0 = C.c_void_p(stream_ptr(stream) or None)
    if aux_stream is None:
        return _check(lib().lc_run_order(stage.handle, C.byref(pb), C.byref(o), arr, s0))
    return _check(lib().lc_run_order_overlap(stage.handle, C.byref(pb), C.byref(o), arr, s0,
                                             C.c_void_p(stream_ptr(aux_stream) or None)))


def lc_run_order_zero(stage: Stage, w, level, grad_shard, shard_offset, shard_len, grad_full,
                      entries, xs, ys, dys, dxs, w_shards=(), w_full=None, stream=None):
    """lc_run_order with ZeRO-2/3 buffers (w_shards: device tensors or
    addresses, in bucket order, with their element counts taken from
    .numel() for tensors, or (address, count) pairs)."""
    M = len(xs)
    o = make_order(entries, M)
    arr = (lc_microbatch_desc * M)(*[_mb(i, xs[i], ys[i], dys[i], dxs[i]) for i in range(M)])
    pb = lc_param_bufs(_vp(w), None)
    ptrs, lens = [], []
    for sh in w_shards:
        if isinstance(sh, tuple):
            ptrs.append(ptr(sh[0]))
            lens.append(int(sh[1]))
        else:
            ptrs.append(ptr(sh))
            lens.append(int(sh.numel()))
    pa = (C.c_void_p * max(1, len(ptrs)))(*[p or None for p in ptrs])
    la = (C.c_size_t * max(1, len(lens)))(*lens)
    z = lc_zero_bufs(level, len(ptrs), _vp(grad_shard), shard_offset, shard_len, _vp(grad_full),
                     C.cast(pa, C.POINTER(C.c_void_p)), C.cast(la, C.POINTER(C.c_size_t)),
                     _vp(w_full))
    return _check(lib().lc_run_order_zero(stage.handle, C.byref(pb), C.byref(z), C.byref(o), arr,
                                          C.c_void_p(stream_ptr(stream) or None)))


def lc_zero_fill_f32(buf, n, stream=None):
    return _check(lib().lc_zero_fill_f32(_vp(buf), n, C.c_void_p(stream_ptr(stream) or None)))


# ------------------------------------------------------------------ buffers

def chunk_accumulate_grad(accum, g, g_dtype, n, stream=None):
    return _check(lib().chunk_accumulate_grad(_vp(accum), _vp(g), g_dtype, n,
                                              C.c_void_p(stream_ptr(stream) or None)))


def shard_adam_step(master, m, v, grad, grad_dtype, out_bf16, n, lr, beta1, beta2, eps,
                    weight_decay, step, stream=None):
    hp = lc_adam_hparams(lr, beta1, beta2, eps, weight_decay, 0, step)
    return _check(lib().shard_adam_step(_vp(master), _vp(m), _vp(v), _vp(grad), grad_dtype,
                                        _vp(out_bf16), n, C.byref(hp),
                                        C.c_void_p(stream_ptr(stream) or None)))


def lc_cast_bf16(inp, out, n, stream=None):
    return _check(lib().lc_cast_bf16(_vp(inp), _vp(out), n,
                                     C.c_void_p(stream_ptr(stream) or None)))


# ------------------------------------------------------------------ ops

def lc_gemm(dtype, epilogue, M, N, K, A, lda, a_kmajor, B, ldb, b_kmajor, Cm, ldc, R=None,
            ldr=0, aux0=None, aux1=None, ld_aux=0, rope_cos=None, rope_sin=None, rope_seq=0,
            rope_cols=0, head_dim=0, c_dtype=None, r_dtype=None, aux_dtype=None, stream=None,
            group_mode=0, n_groups=0, group_offsets=None, group_stride_b=0, group_stride_c=0):
    """C = A.B^T with an epilogue (lc_gemm_args); c/r/aux dtypes default to `dtype`."""
    a = lc_gemm_args()
    a.dtype, a.epilogue = dtype, epilogue
    a.c_dtype = dtype if c_dtype is None else c_dtype
    a.r_dtype = dtype if r_dtype is None else r_dtype
    a.aux_dtype = dtype if aux_dtype is None else aux_dtype
    a.M, a.N, a.K = M, N, K
    a.A, a.lda, a.a_kmajor = ptr(A) or None, lda, int(a_kmajor)
    a.B, a.ldb, a.b_kmajor = ptr(B) or None, ldb, int(b_kmajor)
    a.C, a.ldc = ptr(Cm) or None, ldc
    a.R, a.ldr = ptr(R) or None, ldr
    a.aux0, a.aux1, a.ld_aux = ptr(aux0) or None, ptr(aux1) or None, ld_aux
    a.rope_cos, a.rope_sin = ptr(rope_cos) or None, ptr(rope_sin) or None
    a.rope_seq, a.rope_cols, a.head_dim = rope_seq, rope_cols, head_dim
    a.group_mode, a.n_groups = group_mode, n_groups
    a.group_offsets = ptr(group_offsets) or None
    a.group_stride_b, a.group_stride_c = group_stride_b, group_stride_c
    return _check(lib().lc_gemm(C.byref(a), C.c_void_p(stream_ptr(stream) or None)))


def _fill(struct, **kw):
    for k, v in kw.items():
        if isinstance(v, (int, float)) or v is None:
            setattr(struct, k, v if not (k in _PTR_FIELDS and v == 0) else None)
        else:
            setattr(struct, k, ptr(v))
    return struct


_PTR_FIELDS = {"x", "g", "n", "rstd", "dn", "dres", "dx", "dx_copy", "dg_accum", "scratch", "q",
               "qkv_bf16",
               "k", "v", "o", "lse", "dout", "dq", "dk", "dv", "rope_cos", "rope_sin", "qk",
               "raw", "gq", "gk", "dqk", "dgq", "dgk"}


def lc_rmsnorm_forward(T, d, x, g, eps, n, rstd, x_dtype, w_dtype, out_dtype, stream=None):
    a = _fill(lc_norm_args(), T=T, d=d, eps=eps, x=x, g=g, n=n, rstd=rstd, x_dtype=x_dtype,
              w_dtype=w_dtype, out_dtype=out_dtype)
    return _check(lib().lc_rmsnorm_forward(C.byref(a), C.c_void_p(stream_ptr(stream) or None)))


def lc_rmsnorm_backward(T, d, dn, x, rstd, g, dres, dx, dg_accum, scratch, scratch_bytes,
                        dn_dtype, x_dtype, w_dtype, dres_dtype, out_dtype, dx_copy=None,
                        stream=None):
    a = _fill(lc_norm_args(), T=T, d=d, dn=dn, x=x, rstd=rstd, g=g, dres=dres, dx=dx,
              dx_copy=dx_copy, dg_accum=dg_accum, scratch=scratch, scratch_bytes=scratch_bytes,
              dn_dtype=dn_dtype, x_dtype=x_dtype, w_dtype=w_dtype, dres_dtype=dres_dtype,
              out_dtype=out_dtype)
    return _check(lib().lc_rmsnorm_backward(C.byref(a), C.c_void_p(stream_ptr(stream) or None)))


def lc_rmsnorm_backward_noalloc(T, d, dn, x, rstd, g, dres, dx, dg_accum, dn_dtype, x_dtype,
                                w_dtype, dres_dtype, out_dtype, dx_copy=None, stream=None):
    """lc_rmsnorm_backward with the library's fixed scratch array (no scratch
    argument, nothing allocated)."""
    a = _fill(lc_norm_args(), T=T, d=d, dn=dn, x=x, rstd=rstd, g=g, dres=dres, dx=dx,
              dx_copy=dx_copy, dg_accum=dg_accum, dn_dtype=dn_dtype, x_dtype=x_dtype,
              w_dtype=w_dtype, dres_dtype=dres_dtype, out_dtype=out_dtype)
    return _check(lib().lc_rmsnorm_backward_noalloc(C.byref(a),
                                                    C.c_void_p(stream_ptr(stream) or None)))


def lc_attention_forward(dtype, o_dtype, B, S, H, hd, q, k, v, ld_qkv, o, ld_o, lse, stream=None,
                         Hkv=0):
    a = _fill(lc_attn_args(), dtype=dtype, o_dtype=o_dtype, B=B, S=S, H=H, hd=hd, q=q, k=k, v=v,
              ld_qkv=ld_qkv, o=o, ld_o=ld_o, lse=lse, Hkv=Hkv)
    return _check(lib().lc_attention_forward(C.byref(a), C.c_void_p(stream_ptr(stream) or None)))


def lc_attention_backward(dtype, o_dtype, B, S, H, hd, q, k, v, ld_qkv, o, dout, ld_o, lse, dq,
                          dk, dv, ld_dqkv, rope_cos, rope_sin, scratch, scratch_bytes,
                          stream=None, Hkv=0, qkv_bf16=None, ld_qkv_bf16=0):
    a = _fill(lc_attn_args(), dtype=dtype, o_dtype=o_dtype, B=B, S=S, H=H, hd=hd, q=q, k=k, v=v,
              ld_qkv=ld_qkv, o=o, ld_o=ld_o, lse=lse, dout=dout, dq=dq, dk=dk, dv=dv,
              ld_dqkv=ld_dqkv, rope_cos=rope_cos, rope_sin=rope_sin, scratch=scratch,
              scratch_bytes=scratch_bytes, Hkv=Hkv, qkv_bf16=qkv_bf16, ld_qkv_bf16=ld_qkv_bf16)
    return _check(lib().lc_attention_backward(C.byref(a), C.c_void_p(stream_ptr(stream) or None)))


def lc_qk_norm_rope_forward(T, H, Hkv, hd, seq_len, eps, qk, ld, raw, rstd, gq, gk, x_dtype,
                            w_dtype, rope_cos, rope_sin, stream=None):
    a = _fill(lc_qknorm_args(), T=T, H=H, Hkv=Hkv, hd=hd, seq_len=seq_len, eps=eps, qk=qk, ld=ld,
              raw=raw, rstd=rstd, gq=gq, gk=gk, x_dtype=x_dtype, w_dtype=w_dtype,
              rope_cos=rope_cos, rope_sin=rope_sin)
    return _check(lib().lc_qk_norm_rope_forward(C.byref(a),
                                                C.c_void_p(stream_ptr(stream) or None)))


def lc_qk_norm_rope_backward(T, H, Hkv, hd, seq_len, eps, raw, rstd, gq, gk, x_dtype, w_dtype,
                             dqk, ld_d, d_dtype, dgq, dgk, scratch, scratch_bytes, store_dg=0,
                             stream=None):
    a = _fill(lc_qknorm_args(), T=T, H=H, Hkv=Hkv, hd=hd, seq_len=seq_len, eps=eps, raw=raw,
              rstd=rstd, gq=gq, gk=gk, x_dtype=x_dtype, w_dtype=w_dtype, dqk=dqk, ld_d=ld_d,
              d_dtype=d_dtype, dgq=dgq, dgk=dgk, scratch=scratch, scratch_bytes=scratch_bytes,
              store_dg=store_dg)
    return _check(lib().lc_qk_norm_rope_backward(C.byref(a),
                                                 C.c_void_p(stream_ptr(stream) or None)))


def lc_moe_route(T, d, E, n, wr, sel, w, n_dtype, w_dtype, stream=None):
    """Router: top-2 experts and renormalised gate weights per token."""
    a = _fill(lc_moe_args(), T=T, d=d, E=E, n_dtype=n_dtype, w_dtype=w_dtype)
    a.n, a.wr, a.sel, a.w = ptr(n) or None, ptr(wr) or None, ptr(sel) or None, ptr(w) or None
    return _check(lib().lc_moe_route(C.byref(a), C.c_void_p(stream_ptr(stream) or None)))


def lc_moe_dispatch(T, E, sel, w, offsets, perm, wrow, rowpos, stream=None):
    """Stable grouping of the (token, expert) pairs by expert."""
    a = _fill(lc_moe_args(), T=T, d=8, E=E, n_dtype=LC_BF16, w_dtype=LC_BF16)
    a.sel, a.w = ptr(sel) or None, ptr(w) or None
    a.offsets, a.perm = ptr(offsets) or None, ptr(perm) or None
    a.wrow, a.rowpos = ptr(wrow) or None, ptr(rowpos) or None
    return _check(lib().lc_moe_dispatch(C.byref(a), C.c_void_p(stream_ptr(stream) or None)))


def lc_stage_timer_enable(stage, max_launches):
    """Brackets the stage's next `max_launches` weight-gradient product launches
    with HIP events on their streams (0 turns timing off)."""
    return _check(lib().lc_stage_timer_enable(stage.handle, C.c_int32(max_launches)))


def lc_stage_timer_read(stage, cap):
    """Waits for the timed launches and returns (durations in ms, FLOP per
    launch, number timed since the last read); restarts the count."""
    ms = (C.c_float * max(cap, 1))()
    fl = (C.c_double * max(cap, 1))()
    n = C.c_int32(0)
    _check(lib().lc_stage_timer_read(stage.handle, ms, fl, C.c_int32(cap), C.byref(n)))
    k = min(cap, n.value)
    return list(ms[:k]), list(fl[:k]), n.value


def lc_stage_moe_routing(stage, mb, layer, sel_out, stream=None):
    """Copies the routing of a stashed microbatch's layer into `sel_out` [T, 2] int32."""
    return _check(lib().lc_stage_moe_routing(stage.handle, C.c_int32(mb), C.c_int32(layer),
                                             C.c_void_p(ptr(sel_out)),
                                             C.c_void_p(stream_ptr(stream) or None)))
