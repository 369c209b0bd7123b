"""Device-side driver of one pipeline stage through the libchunk C-ABI.

Allocates the caller-owned device memory the library expects (weights in the
compute dtype, the fp32 gradient bucket, fp32 master/m/v for the optimizer,
the workspace, and per-microbatch X/Y/dY/dX) with PyTorch, and calls the
entry points. PyTorch is used for memory and streams only.
"""
from __future__ import annotations

from typing import List, Optional, Sequence, Tuple

import numpy as np
import torch

from . import libchunk as lc


def require_gpu():
    if not torch.cuda.is_available():
        raise RuntimeError("libchunk needs a ROCm GPU (torch.cuda.is_available() is False)")
    lc.lib()  # fails loudly when the HIP library is missing


def to_device(a: np.ndarray, bf16: bool, device="cuda") -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    if bf16:
        t = t.to(torch.bfloat16)
    return t.to(device)


class StageRunner:
    """One stage on one GPU: weights, gradient bucket, workspace, microbatches."""

    def __init__(self, desc: lc.lc_stage_desc, flat_params: np.ndarray, max_in_flight: int,
                 device="cuda", stream: Optional[torch.cuda.Stream] = None,
                 max_w_pending: int = 0):
        require_gpu()
        self.desc = desc
        self.bf16 = desc.compute_dtype == lc.LC_BF16
        self.dtype = torch.bfloat16 if self.bf16 else torch.float32
        self.device = device
        self.stream = stream or torch.cuda.current_stream()
        self.n_params = lc.lc_param_count(desc)
        assert flat_params.size == self.n_params
        self.w = to_device(flat_params, self.bf16, device)
        self.grad = torch.zeros(self.n_params, dtype=torch.float32, device=device)
        self.ws_bytes = lc.lc_workspace_bytes(desc, max_in_flight, max_w_pending)
        self.ws = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=device)
        base = self.ws.data_ptr()
        self.ws_ptr = (base + 255) // 256 * 256
        self.max_in_flight = max_in_flight
        self.stage = lc.lc_stage_create(desc, self.ws_ptr, self.ws_bytes, max_in_flight,
                                        self.stream, max_w_pending)
        self.T = desc.micro_batch * desc.seq_len
        self.master = None

    # -------------------------------------------------------------- microbatches
    def alloc_microbatches(self, Xs: Sequence[np.ndarray], dYs: Sequence[np.ndarray]):
        self.X = [to_device(x, self.bf16, self.device) for x in Xs]
        self.dY = [to_device(d, self.bf16, self.device) for d in dYs]
        self.Y = [torch.empty_like(x) for x in self.X]
        self.dX = [torch.empty_like(x) for x in self.X]

    def alloc_random_microbatches(self, M: int, seed: int = 0):
        """N(0,1) activations generated on the device (benchmark inputs)."""
        g = torch.Generator(device=self.device)
        g.manual_seed(seed)
        shape = (self.desc.micro_batch, self.desc.seq_len, self.desc.d_model)
        self.X = [torch.randn(shape, generator=g, device=self.device).to(self.dtype)
                  for _ in range(M)]
        self.dY = [torch.randn(shape, generator=g, device=self.device).to(self.dtype)
                   for _ in range(M)]
        self.Y = [torch.empty_like(x) for x in self.X]
        self.dX = [torch.empty_like(x) for x in self.X]

    def forward(self, mb: int):
        lc.chunk_forward(self.stage, self.w, self.grad, mb, self.X[mb], self.Y[mb], self.stream)

    def backward(self, mb: int):
        lc.chunk_backward(self.stage, self.w, self.grad, mb, self.dY[mb], self.dX[mb],
                          self.stream)

    def backward_input(self, mb: int):
        lc.chunk_backward_input(self.stage, self.w, mb, self.dY[mb], self.dX[mb], self.stream)

    def backward_weight(self, mb: int):
        lc.chunk_backward_weight(self.stage, self.w, self.grad, mb, self.stream)

    def moe_routing(self, mb: int, layer: int) -> np.ndarray:
        """The experts chosen for each token of a stashed microbatch's layer, [T, 2]."""
        out = torch.empty((self.T, 2), dtype=torch.int32, device=self.device)
        lc.lc_stage_moe_routing(self.stage, mb, layer, out, self.stream)
        torch.cuda.synchronize()
        return out.cpu().numpy()

    def run_order(self, entries: Sequence[Tuple[int, int]], aux_stream=None):
        """Enqueues an Order on self.stream; overlapped pairs use aux_stream
        when one is given."""
        lc.lc_run_order(self.stage, self.w, self.grad, entries, self.X, self.Y, self.dY, self.dX,
                        self.stream, aux_stream)

    def run_order_zero(self, entries, level, grad_shard, shard_offset, grad_full,
                       w_shards=(), w_full=None):
        """Enqueues an Order with ZeRO-2 (level 2) or ZeRO-3 (level 3)
        buffers: each backward's full gradient goes to grad_full and its
        slice [shard_offset, shard_offset + grad_shard.numel()) is added into
        grad_shard; at level 3 the weights are gathered from w_shards into
        w_full before every entry."""
        lc.lc_run_order_zero(self.stage, self.w, level, grad_shard, shard_offset,
                             grad_shard.numel(), grad_full, entries, self.X, self.Y, self.dY,
                             self.dX, w_shards, w_full, self.stream)

    # -------------------------------------------------------------- optimizer
    def init_optimizer(self, flat_params: np.ndarray):
        """fp32 master weights and zero Adam moments. An fp32 stage's compute
        weights are the master weights themselves (updated in place)."""
        if self.bf16:
            self.master = torch.from_numpy(np.ascontiguousarray(flat_params, np.float32)).to(
                self.device)
        else:
            self.master = self.w
        self.m = torch.zeros_like(self.master)
        self.v = torch.zeros_like(self.master)
        self.step_count = 0

    def adam_step(self, lr, beta1, beta2, eps, weight_decay):
        """AdamW over the whole bucket (this GPU's shard), writing the new bf16
        compute weights in the same pass."""
        self.step_count += 1
        out = self.w if self.bf16 else None
        lc.shard_adam_step(self.master, self.m, self.v, self.grad, lc.LC_FP32, out,
                           self.n_params, lr, beta1, beta2, eps, weight_decay, self.step_count,
                           self.stream)

    def zero_grad(self):
        """G = +0 before the first backward of a step (the library's fill
        kernel, enqueued on the stage's stream)."""
        lc.lc_zero_fill_f32(self.grad, self.n_params, self.stream)

    def close(self):
        self.stage.close()


def random_stage(desc: lc.lc_stage_desc, max_in_flight: int, seed: int = 0, device="cuda",
                 stream=None, max_w_pending: int = 0) -> StageRunner:
    """A StageRunner with weights drawn on the device: matrices ~ N(0, 0.02)
    in the compute dtype, RMSNorm gains (and q/k norm gains) = 1 (benchmark
    inputs)."""
    require_gpu()
    r = StageRunner.__new__(StageRunner)
    r.desc = desc
    r.bf16 = desc.compute_dtype == lc.LC_BF16
    r.dtype = torch.bfloat16 if r.bf16 else torch.float32
    r.device = device
    r.stream = stream or torch.cuda.current_stream()
    r.n_params = lc.lc_param_count(desc)
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    master = torch.randn(r.n_params, generator=g, device=device, dtype=torch.float32)
    master.mul_(0.02)
    gains = (lc.LC_T_G1, lc.LC_T_G2) + ((lc.LC_T_QN, lc.LC_T_KN) if desc.qk_norm else ())
    for l in range(desc.n_layers):
        for t in gains:
            off, (n, _) = lc.lc_param_offset(desc, l, t)
            master[off:off + n] = 1.0
    r.w = master.to(r.dtype) if r.bf16 else master
    r.master = master
    r.m = torch.zeros_like(master)
    r.v = torch.zeros_like(master)
    r.step_count = 0
    r.grad = torch.zeros(r.n_params, dtype=torch.float32, device=device)
    r.ws_bytes = lc.lc_workspace_bytes(desc, max_in_flight, max_w_pending)
    r.ws = torch.empty(r.ws_bytes + 256, dtype=torch.uint8, device=device)
    r.ws_ptr = (r.ws.data_ptr() + 255) // 256 * 256
    r.max_in_flight = max_in_flight
    r.stage = lc.lc_stage_create(desc, r.ws_ptr, r.ws_bytes, max_in_flight, r.stream,
                                 max_w_pending)
    r.T = desc.micro_batch * desc.seq_len
    return r
