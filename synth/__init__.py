"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This module holds the workload shapes, the canonical flat parameter layout
and the random-number recipe. It contains none of the method's arithmetic:
no normalisation, attention, projection, gradient or optimizer step. Both
the CPU oracle and the HIP path consume exactly the values produced here.

Recipe (the paper measures Qwen3 decoder training but prints no layer
definition, dataset or precision; these stand-ins follow the workload
shapes of the pipeline-stage experiments, Piper Section 6):
  * activations X and upstream gradients dY ~ N(0, 1);
  * projection, FFN and router matrices ~ N(0, 0.02);
  * RMSNorm gains = 1 (random gains only where a test asks for them);
  * for bf16-compute workloads every draw is rounded to the nearest bf16
    value (round-to-nearest-even), so both sides see identical inputs.
Each tensor has its own stream: numpy's PCG64 seeded with (seed, tensor id),
so any tensor can be regenerated on its own.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Tuple

import numpy as np

# ---------------------------------------------------------------------------
# Workloads
# ---------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class StageConfig:
    """Shape of one pipeline stage (one Chunk per microbatch and pass)."""
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ff: int
    seq_len: int
    micro_batch: int
    num_microbatches: int
    bf16: bool
    n_experts: int = 0
    top_k: int = 0
    d_ff_expert: int = 0
    rms_eps: float = 1e-5
    rope_base: float = 10000.0
    n_kv_heads: int = 0    # key/value heads (grouped-query attention); 0 = n_heads
    qk_norm: bool = False  # per-head RMSNorm of q and k before RoPE (Qwen3)
    pp_size: int = 2       # pipeline depth used to build the 1F1B Order
    pp_rank: int = 0       # this stage's index in the pipeline
    # AdamW hyper-parameters applied after the last backward of a step
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    adam_eps: float = 1e-8
    weight_decay: float = 0.0

    @property
    def tokens(self) -> int:
        return self.micro_batch * self.seq_len

    @property
    def moe(self) -> bool:
        return self.n_experts > 0

    @property
    def kv_heads(self) -> int:
        return self.n_kv_heads or self.n_heads


@dataclasses.dataclass(frozen=True)
class AdamShardConfig:
    name: str
    n: int
    lr: float
    beta1: float
    beta2: float
    eps: float
    weight_decay: float
    p_std: float
    g_std: float


TINY_FP32 = StageConfig(
    name="tiny_fp32_2L_d128", n_layers=2, d_model=128, n_heads=4, head_dim=32,
    d_ff=344, seq_len=64, micro_batch=2, num_microbatches=4, bf16=False,
    pp_size=2, pp_rank=0, lr=1e-3, beta1=0.9, beta2=0.999, adam_eps=1e-8,
    weight_decay=0.0)

LLAMA_2K = StageConfig(
    name="llama_8L_d2048_s2048", n_layers=8, d_model=2048, n_heads=16,
    head_dim=128, d_ff=5632, seq_len=2048, micro_batch=1, num_microbatches=8,
    bf16=True, pp_size=4, pp_rank=0)

STAGE_7B = StageConfig(
    name="stage7b_4L_d4096_s4096", n_layers=4, d_model=4096, n_heads=32,
    head_dim=128, d_ff=11008, seq_len=4096, micro_batch=1,
    num_microbatches=16, bf16=True, pp_size=8, pp_rank=0,
    lr=3e-4, beta1=0.9, beta2=0.95, adam_eps=1e-8, weight_decay=0.1)

MOE_2K = StageConfig(
    name="moe_4L_d2048_e8_s2048", n_layers=4, d_model=2048, n_heads=16,
    head_dim=128, d_ff=0, seq_len=2048, micro_batch=2, num_microbatches=8,
    bf16=True, n_experts=8, top_k=2, d_ff_expert=1408, pp_size=4, pp_rank=0)

ADAM_1P6B = AdamShardConfig(
    name="adam_shard_1p6e9", n=1_600_000_000, lr=3e-4, beta1=0.9, beta2=0.95,
    eps=1e-8, weight_decay=0.1, p_std=0.02, g_std=1e-3)

# Qwen3-8B-shaped stage: 4 layers of d 4096, 32 query heads and 8 key/value
# heads of 128, per-head q/k RMSNorm, SwiGLU 12288
QWEN3_STAGE = StageConfig(
    name="qwen3_4L_d4096_kv8_s4096", n_layers=4, d_model=4096, n_heads=32,
    head_dim=128, d_ff=12288, seq_len=4096, micro_batch=1, num_microbatches=16,
    bf16=True, n_kv_heads=8, qk_norm=True, rms_eps=1e-6, rope_base=1000000.0,
    pp_size=8, pp_rank=0, lr=3e-4, beta1=0.9, beta2=0.95, adam_eps=1e-8,
    weight_decay=0.1)

STAGES = {c.name: c for c in (TINY_FP32, LLAMA_2K, STAGE_7B, MOE_2K, QWEN3_STAGE)}


def scaled(cfg: StageConfig, **kw) -> StageConfig:
    """A copy of `cfg` with some fields replaced (small parity cases)."""
    return dataclasses.replace(cfg, **kw)


# ---------------------------------------------------------------------------
# Canonical flat parameter layout (one bucket per stage)
# ---------------------------------------------------------------------------

# tensor ids inside one layer, in layout order
DENSE_TENSORS = ("wq", "wk", "wv", "wo", "g1", "w1", "w3", "w2", "g2")


def layout(cfg: StageConfig) -> List[Tuple[str, int, Tuple[int, ...]]]:
    """[(name, offset, shape)] of every parameter tensor in the flat bucket.

    Per layer l: Wq [d, d], Wk, Wv [kv_heads * hd, d], Wo [d, d]; g1 [d];
    with qk_norm the q and k gains qn, kn [hd]; then either the dense FFN
    W1 (gate) [f, d], W3 (up) [f, d], W2 (down) [d, f], or the MoE block
    Wr [E, d] followed by W1_e, W3_e [fe, d], W2_e [d, fe] per expert e;
    then g2 [d]. Weights are [out, in] row-major.
    """
    d, f = cfg.d_model, cfg.d_ff
    dkv = cfg.kv_heads * cfg.head_dim
    out = []
    off = 0

    def add(name, shape):
        nonlocal off
        out.append((name, off, tuple(shape)))
        off += int(np.prod(shape))

    for l in range(cfg.n_layers):
        add(f"L{l}.wq", (d, d))
        add(f"L{l}.wk", (dkv, d))
        add(f"L{l}.wv", (dkv, d))
        add(f"L{l}.wo", (d, d))
        add(f"L{l}.g1", (d,))
        if cfg.qk_norm:
            add(f"L{l}.qn", (cfg.head_dim,))
            add(f"L{l}.kn", (cfg.head_dim,))
        if cfg.moe:
            fe = cfg.d_ff_expert
            add(f"L{l}.wr", (cfg.n_experts, d))
            for e in range(cfg.n_experts):
                add(f"L{l}.e{e}.w1", (fe, d))
                add(f"L{l}.e{e}.w3", (fe, d))
                add(f"L{l}.e{e}.w2", (d, fe))
        else:
            add(f"L{l}.w1", (f, d))
            add(f"L{l}.w3", (f, d))
            add(f"L{l}.w2", (d, f))
        add(f"L{l}.g2", (d,))
    return out


def param_count(cfg: StageConfig) -> int:
    name, off, shape = layout(cfg)[-1]
    return off + int(np.prod(shape))


# ---------------------------------------------------------------------------
# Random draws
# ---------------------------------------------------------------------------

TID_X = 100_000
TID_DY = 200_000
TID_ADAM = 300_000


def _rng(seed: int, tid: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tid])))


def normal(seed: int, tid: int, n: int, std: float) -> np.ndarray:
    """n draws of N(0, std^2) as float32 (tensor `tid` of run `seed`)."""
    a = _rng(seed, tid).standard_normal(n, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    return a


def round_bf16(a: np.ndarray) -> np.ndarray:
    """float32 array -> float32 array holding the nearest bf16 values (RNE).

    Uses torch's own float->bfloat16 conversion (a library routine), so the
    input recipe does not depend on either side's cast.
    """
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 array of bf16-representable values -> uint16 bit patterns."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    return (a.view(np.uint32) >> 16).astype(np.uint16)


def stage_params(cfg: StageConfig, seed: int = 0,
                 random_gains: bool = False) -> np.ndarray:
    """The flat parameter bucket (float32 values; bf16 values for bf16
    workloads) in the canonical layout."""
    n = param_count(cfg)
    w = np.empty(n, dtype=np.float32)
    for tid, (name, off, shape) in enumerate(layout(cfg)):
        sz = int(np.prod(shape))
        if name.endswith((".g1", ".g2", ".qn", ".kn")):
            if random_gains:
                w[off:off + sz] = 1.0 + normal(seed, tid, sz, 0.1)
            else:
                w[off:off + sz] = 1.0
        else:
            w[off:off + sz] = normal(seed, tid, sz, 0.02)
    if cfg.bf16:
        w = round_bf16(w)
    return w


def unflatten(cfg: StageConfig, flat: np.ndarray) -> Dict[str, np.ndarray]:
    """Views of the flat bucket as named tensors."""
    return {name: flat[off:off + int(np.prod(shape))].reshape(shape)
            for name, off, shape in layout(cfg)}


def flatten(cfg: StageConfig, tensors: Dict[str, np.ndarray],
            dtype=np.float64) -> np.ndarray:
    """Named tensors -> flat bucket in the canonical layout."""
    out = np.zeros(param_count(cfg), dtype=dtype)
    for name, off, shape in layout(cfg):
        out[off:off + int(np.prod(shape))] = np.asarray(tensors[name]).reshape(-1)
    return out


def activation(cfg: StageConfig, seed: int, mb: int, which: str) -> np.ndarray:
    """X[mb] (which='x') or dY[mb] (which='dy'), shape [b, S, d], ~N(0,1)."""
    tid = (TID_X if which == "x" else TID_DY) + mb
    a = normal(seed, tid, cfg.tokens * cfg.d_model, 1.0)
    if cfg.bf16:
        a = round_bf16(a)
    return a.reshape(cfg.micro_batch, cfg.seq_len, cfg.d_model)


def adam_inputs(n: int, seed: int = 0, p_std: float = 0.02,
                g_std: float = 1e-3, state: str = "zero"):
    """(p fp32, m fp32, v fp32, g as bf16 values in fp32) for an Adam shard.

    state='zero' gives m = v = 0 (a first step); state='warm' gives
    m ~ N(0, 1e-3) and v = N(0, 1e-3)^2 (a later step).
    """
    p = normal(seed, TID_ADAM + 0, n, p_std)
    g = round_bf16(normal(seed, TID_ADAM + 1, n, g_std))
    if state == "zero":
        m = np.zeros(n, np.float32)
        v = np.zeros(n, np.float32)
    else:
        m = normal(seed, TID_ADAM + 2, n, 1e-3)
        v = np.square(normal(seed, TID_ADAM + 3, n, 1e-3))
    return p, m, v, g
