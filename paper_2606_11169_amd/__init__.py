"""libchunk: one device's share of Piper's data-parallel training hot path on
AMD Instinct MI355X (gfx950): Chunk forward/backward of a decoder pipeline
stage over a microbatch Order, fp32 gradient accumulation, and a fused AdamW
shard step, behind a C ABI (include/libchunk.h, include/libchunk_ops.h).

`libchunk` is the ctypes binding; `runner` drives a stage with PyTorch
device memory; `build` compiles the HIP library in-tree.
"""
from . import libchunk  # noqa: F401
