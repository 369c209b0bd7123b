"""Whole-stage parity of the HIP path (lc_run_order / chunk_forward /
chunk_backward / shard_adam_step) with the oracle.

* tiny fp32 stage (2 layers, d 128, 4 microbatches in 1F1B, one AdamW step):
  Y, dX, every gradient tensor and the updated p, m, v within 1e-4
* small bf16 stage spanning several tiles: within 2e-2
* Order invariance (1F1B vs GPipe: bitwise identical), run-to-run
  determinism, and the accumulated gradient equal, bit for bit, to the
  sequential fp32 sum of the per-microbatch gradients
* the 7B-shaped, Qwen3-8B-shaped and 8-layer d-2048 Llama-style stages at
  full size: outputs on a prefix of the sequence against the oracle run on
  that prefix (causality makes the prefix self-contained), with dY zero
  beyond the prefix so the full-size backward (dX, every gradient) is
  checked too; dX beyond the prefix must be exactly 0
* split backwards (Bi/Bw), overlapped pairs on two streams and the ZeRO-2/3
  paths: bit-identical to the plain Order, and against the oracle
* a NaN in one input token: propagated (causally) into Y, dX, the gradient and
  the AdamW update, never skipped; everything it cannot reach bit-identical
* the weight-gradient timing hook: one event pair per product, results unchanged
"""
import numpy as np
import pytest
import torch

import synth
from oracle import optim as OP
from oracle import order as OO
from oracle import stage as OS
from paper_2606_11169_amd import libchunk as lc
from paper_2606_11169_amd.runner import StageRunner, require_gpu
from tests.gpu_util import banner, gpu_routes, host, oracle_order_with_routes, rel_err

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


def desc_of(cfg):
    return lc.desc_of_config(cfg)


PASS = {"F": lc.LC_PASS_F, "B": lc.LC_PASS_B, "Bi": lc.LC_PASS_BI, "Bw": lc.LC_PASS_BW}


def to_c(entries):
    """Oracle Order -> C entries; a nested pair's first entry carries
    LC_ORDER_WITH_NEXT."""
    out = []
    for e in entries:
        if isinstance(e, list):
            for k, (mb, ps) in enumerate(e):
                out.append((mb, PASS[ps] | (lc.LC_ORDER_WITH_NEXT if k < len(e) - 1 else 0)))
        else:
            out.append((e[0], PASS[e[1]]))
    return out


def inputs(cfg, seed=0):
    flat = synth.stage_params(cfg, seed)
    M = cfg.num_microbatches
    Xs = [synth.activation(cfg, seed, mb, "x") for mb in range(M)]
    dYs = [synth.activation(cfg, seed, mb, "dy") for mb in range(M)]
    return flat, Xs, dYs


def gpu_run(cfg, order, flat, Xs, dYs, max_in_flight=None, max_w_pending=0, aux_stream=None):
    r = StageRunner(desc_of(cfg), flat, max_in_flight or cfg.num_microbatches,
                    max_w_pending=max_w_pending)
    r.alloc_microbatches(Xs, dYs)
    r.run_order(to_c(order), aux_stream)
    torch.cuda.synchronize()
    return r


def report(errs, k=6):
    top = sorted(errs.items(), key=lambda kv: -kv[1])[:k]
    print("worst tensors: " + ", ".join(f"{n}={e:.2e}" for n, e in top), flush=True)


def per_tensor_errors(cfg, got, ref):
    out = {}
    for name, off, shape in synth.layout(cfg):
        sz = int(np.prod(shape))
        out[name] = rel_err(got[off:off + sz], ref[off:off + sz])
    return out


SMALL_BF16 = synth.StageConfig(
    name="small_bf16", n_layers=2, d_model=256, n_heads=2, head_dim=128, d_ff=512, seq_len=256,
    micro_batch=2, num_microbatches=3, bf16=True, pp_size=3, pp_rank=0)
# Qwen3-style variant (per-head q/k RMSNorm, grouped-query attention)
QWEN_BF16 = synth.StageConfig(
    name="qwen_bf16", n_layers=2, d_model=512, n_heads=4, head_dim=128, d_ff=512, seq_len=256,
    micro_batch=2, num_microbatches=3, bf16=True, n_kv_heads=2, qk_norm=True, rms_eps=1e-6,
    rope_base=1000000.0, pp_size=3, pp_rank=0)
QWEN_FP32 = synth.StageConfig(
    name="qwen_fp32", n_layers=2, d_model=128, n_heads=4, head_dim=32, d_ff=344, seq_len=64,
    micro_batch=2, num_microbatches=4, bf16=False, n_kv_heads=2, qk_norm=True, rms_eps=1e-6,
    pp_size=2, pp_rank=0)


# 384 tokens: a half-full last 256-row block of the attention kernels after a
# full one (forward, dK/dV and dQ partial-block masking)
SMALL_BF16_S384 = synth.scaled(SMALL_BF16, name="small_bf16_s384", seq_len=384,
                               num_microbatches=2, pp_size=2)


@pytest.mark.parametrize("cfg,tol", [(synth.TINY_FP32, 1e-4), (SMALL_BF16, 2e-2),
                                     (QWEN_FP32, 1e-4), (QWEN_BF16, 2e-2),
                                     (SMALL_BF16_S384, 2e-2)],
                         ids=["tiny_fp32", "small_bf16", "qwen_fp32", "qwen_bf16",
                              "small_bf16_s384"])
def test_stage_matches_oracle(cfg, tol):
    banner(f"stage {cfg.name}")
    flat, Xs, dYs = inputs(cfg)
    order = OO.one_f_one_b(cfg.num_microbatches, cfg.pp_size, cfg.pp_rank)
    r = gpu_run(cfg, order, flat, Xs, dYs)
    Ys, dXs, G = OS.run_order(cfg, flat, Xs, dYs, order)
    for mb in range(cfg.num_microbatches):
        print(f"mb {mb}: Y err {rel_err(host(r.Y[mb]), Ys[mb]):.2e}, "
              f"dX err {rel_err(host(r.dX[mb]), dXs[mb]):.2e}")
        assert rel_err(host(r.Y[mb]), Ys[mb]) <= tol, f"Y[{mb}]"
        assert rel_err(host(r.dX[mb]), dXs[mb]) <= tol, f"dX[{mb}]"
    Gg = host(r.grad)
    errs = per_tensor_errors(cfg, Gg, G)
    report(errs)
    worst = max(errs, key=errs.get)
    assert errs[worst] <= tol, (worst, errs[worst])
    # one AdamW step on the accumulated gradient
    r.init_optimizer(flat)
    r.adam_step(cfg.lr, cfg.beta1, cfg.beta2, cfg.adam_eps, cfg.weight_decay)
    torch.cuda.synchronize()
    g_ref = G.astype(np.float32)
    z = np.zeros_like(flat)
    p_ref, m_ref, v_ref = OP.adamw(flat, z, z, g_ref, cfg.lr, cfg.beta1, cfg.beta2,
                                   cfg.adam_eps, cfg.weight_decay, 1)
    assert rel_err(host(r.m), m_ref) <= tol
    assert rel_err(host(r.v), v_ref) <= 2 * tol
    # at t = 1 the update is ~ -lr*sign(g), so an element whose gradient is
    # within the tolerated error of 0 may move either way. Such elements are
    # the ones with |g_ref| <= tol * max|g_ref| over their tensor: p is
    # compared on all others, and every sign disagreement must lie among them
    keep = adam_comparable(cfg, G, tol)
    flips = np.sign(Gg.astype(np.float32)) != np.sign(g_ref)
    print(f"adam: {int((~keep).sum())} of {keep.size} elements near zero gradient excluded, "
          f"{int(flips.sum())} sign disagreements")
    assert not np.any(flips & keep), "a gradient sign differs where |g_ref| is not near 0"
    assert rel_err(host(r.master)[keep], p_ref[keep]) <= tol
    r.close()


def adam_comparable(cfg, G, tol):
    """Elements whose reference gradient is not within tol * max|G| of its
    tensor from zero: there the first AdamW step's direction is fixed."""
    keep = np.ones(G.size, bool)
    for name, off, shape in synth.layout(cfg):
        sz = int(np.prod(shape))
        g = np.abs(G[off:off + sz])
        keep[off:off + sz] = g > tol * np.max(g)
    return keep


def test_order_invariance_determinism_and_exact_accumulation():
    cfg = SMALL_BF16
    banner("order invariance / determinism")
    flat, Xs, dYs = inputs(cfg, seed=3)
    M = cfg.num_microbatches
    a = gpu_run(cfg, OO.one_f_one_b(M, 3, 0), flat, Xs, dYs)
    b = gpu_run(cfg, OO.gpipe(M), flat, Xs, dYs)
    c = gpu_run(cfg, OO.one_f_one_b(M, 3, 0), flat, Xs, dYs)
    for r in (b, c):
        assert torch.equal(a.grad, r.grad)
        for mb in range(M):
            assert torch.equal(a.Y[mb], r.Y[mb]) and torch.equal(a.dX[mb], r.dX[mb])
    # each microbatch alone into a zeroed bucket, then a sequential fp32 sum
    acc = np.zeros(a.n_params, np.float32)
    for mb in range(M):
        one = gpu_run(cfg, [(0, "F"), (0, "B")], flat, [Xs[mb]], [dYs[mb]], max_in_flight=1)
        acc = OP.accumulate(acc, host(one.grad).astype(np.float32))
        one.close()
    assert np.array_equal(acc.view(np.uint32), host(a.grad).astype(np.float32).view(np.uint32))
    for r in (a, b, c):
        r.close()


def test_weight_gradient_timer_brackets_every_product():
    """lc_stage_timer_enable/read: one event pair per weight-gradient product
    in launch order (layers top down: W2, W1;W3, Wo, Wq;Wk;Wv), each with its
    2 M N K; timing leaves the gradient bit-identical; the count restarts on
    read and stops at the capacity."""
    cfg = SMALL_BF16
    banner("weight-gradient timer")
    flat, Xs, dYs = inputs(cfg, seed=5)
    M, nl = cfg.num_microbatches, cfg.n_layers
    order = OO.one_f_one_b(M, 3, 0)
    ref = gpu_run(cfg, order, flat, Xs, dYs)
    r = StageRunner(desc_of(cfg), flat, M)
    r.alloc_microbatches(Xs, dYs)
    launches = 4 * nl * M
    lc.lc_stage_timer_enable(r.stage, launches + 3)
    r.run_order(to_c(order))
    torch.cuda.synchronize()
    ms, fl, n = lc.lc_stage_timer_read(r.stage, launches + 3)
    assert n == launches and len(ms) == launches
    assert torch.equal(ref.grad, r.grad)
    T, D, F = cfg.tokens, cfg.d_model, cfg.d_ff
    QC = D + 2 * cfg.head_dim * cfg.kv_heads
    per_layer = [2.0 * D * F * T, 2.0 * 2 * F * D * T, 2.0 * D * D * T, 2.0 * QC * D * T]
    assert fl == per_layer * (nl * M)
    assert all(0.0 < t < 1e3 for t in ms)
    assert lc.lc_stage_timer_read(r.stage, 4)[2] == 0
    lc.lc_stage_timer_enable(r.stage, 5)
    r.zero_grad()
    r.run_order(to_c(order))
    torch.cuda.synchronize()
    ms, fl, n = lc.lc_stage_timer_read(r.stage, 2)
    assert n == 5 and len(ms) == 2 and fl == per_layer[:2]
    assert torch.equal(ref.grad, r.grad)
    lc.lc_stage_timer_enable(r.stage, 0)
    for x in (ref, r):
        x.close()


def test_non_finite_values_propagate_without_skipping():
    """NaN is neither masked nor skipped: a NaN in one element of one token's
    input makes every later position of that sequence NaN in Y (the token's
    normalised row is all NaN and causal attention carries it forward), leaves
    the positions before the token's 64-key block and the other sequence of the
    microbatch bit-identical, leaves the other microbatches bit-identical, and
    reaches the gradient; AdamW then turns exactly the parameters whose
    gradient is NaN into NaN and updates the rest."""
    cfg = SMALL_BF16
    banner("NaN propagation")
    flat, Xs, dYs = inputs(cfg, seed=6)
    M = cfg.num_microbatches
    order = OO.one_f_one_b(M, 3, 0)
    ref = gpu_run(cfg, order, flat, Xs, dYs)
    p = 150  # token of sequence 0; its 64-key block starts at 128
    bad = [x.copy() for x in Xs]
    bad[1][0, p, 7] = np.nan  # activations are [micro_batch, seq_len, d_model]
    r = gpu_run(cfg, order, flat, bad, dYs)
    assert torch.isnan(r.Y[1][0, p:].float()).all()
    assert torch.equal(r.Y[1][0, :128], ref.Y[1][0, :128])
    assert torch.equal(r.Y[1][1], ref.Y[1][1])  # the microbatch's other sequence
    for mb in (0, 2):
        assert torch.equal(r.Y[mb], ref.Y[mb]) and torch.equal(r.dX[mb], ref.dX[mb])
    assert torch.isnan(r.dX[1][0, p].float()).all()
    g_nan = torch.isnan(r.grad)
    assert g_nan.any() and not torch.isnan(ref.grad).any()
    r.init_optimizer(flat)
    r.adam_step(1e-3, 0.9, 0.95, 1e-8, 0.1)
    torch.cuda.synchronize()
    assert torch.equal(torch.isnan(r.master), g_nan)
    assert torch.equal(torch.isnan(r.w.float()), g_nan)
    assert torch.isfinite(r.master[~g_nan]).all()
    for x in (ref, r):
        x.close()


def test_stage_error_paths_have_no_side_effects():
    cfg = SMALL_BF16
    banner("stage error paths")
    flat, Xs, dYs = inputs(cfg, seed=4)
    r = StageRunner(desc_of(cfg), flat, 2)
    r.alloc_microbatches(Xs, dYs)
    with pytest.raises(lc.LibchunkError) as e:
        r.backward(0)
    assert e.value.status == lc.LC_ERR_STATE
    r.forward(0)
    with pytest.raises(lc.LibchunkError) as e:
        r.forward(0)
    assert e.value.status == lc.LC_ERR_STATE
    r.forward(1)
    with pytest.raises(lc.LibchunkError) as e:
        r.forward(2)
    assert e.value.status == lc.LC_ERR_STASH_FULL
    r.backward(0)
    r.backward(1)
    with pytest.raises(lc.LibchunkError) as e:
        r.run_order(to_c(OO.parse("F1 F0 B0 B1 B2 F2")))
    assert e.value.status == lc.LC_ERR_BAD_ORDER
    with pytest.raises(lc.LibchunkError) as e:
        r.run_order(to_c(OO.gpipe(3)))
    assert e.value.status == lc.LC_ERR_STASH_FULL
    torch.cuda.synchronize()
    r.close()


@pytest.mark.parametrize("cfg,tol", [(synth.TINY_FP32, 1e-4), (SMALL_BF16, 2e-2),
                                     (QWEN_BF16, 2e-2)],
                         ids=["tiny_fp32", "small_bf16", "qwen_bf16"])
def test_split_backward_matches_full_backward_and_oracle(cfg, tol):
    """Bi + Bw (PASS values of Section 4.1): with the Bw entries in
    microbatch order, adjacent or deferred, every output and the gradient are
    bit-identical to the plain Order's; Bw in another order changes the
    gradient by rounding only (checked against the oracle)."""
    banner(f"split backward {cfg.name}")
    flat, Xs, dYs = inputs(cfg, seed=6)
    M, P, s = cfg.num_microbatches, cfg.pp_size, cfg.pp_rank
    ref = gpu_run(cfg, OO.one_f_one_b(M, P, s), flat, Xs, dYs)
    for wd in (0, 1, M):
        order = OO.one_f_one_b_split(M, P, s, wd)
        r = gpu_run(cfg, order, flat, Xs, dYs, max_w_pending=min(wd + 1, M))
        print(f"w_delay {wd}: {' '.join(f'{p}{m}' for m, p in order)}", flush=True)
        assert torch.equal(r.grad, ref.grad), f"w_delay {wd}"
        for mb in range(M):
            assert torch.equal(r.Y[mb], ref.Y[mb]) and torch.equal(r.dX[mb], ref.dX[mb])
        r.close()
    rev = [(m, "F") for m in range(M)] + [(m, "Bi") for m in range(M)] + \
          [(m, "Bw") for m in reversed(range(M))]
    r = gpu_run(cfg, rev, flat, Xs, dYs, max_w_pending=M)
    _, dXs, G = OS.run_order(cfg, flat, Xs, dYs, rev)
    errs = per_tensor_errors(cfg, host(r.grad), G)
    report(errs)
    assert max(errs.values()) <= tol
    for mb in range(M):
        assert torch.equal(r.dX[mb], ref.dX[mb])
        assert rel_err(host(r.dX[mb]), dXs[mb]) <= tol
    r.close()
    ref.close()


SPLIT_PAIRS = {
    3: "F0 [F1 Bi0] [F2 Bw0] Bi1 [Bi2 Bw1] Bw2",
    4: "F0 [F1 Bi0] [F2 Bw0] [F3 Bi1] [Bi2 Bw1] [Bi3 Bw2] Bw3",
}


@pytest.mark.parametrize("cfg", [synth.TINY_FP32, SMALL_BF16], ids=["tiny_fp32", "small_bf16"])
def test_overlapped_pairs_on_two_streams_are_bit_identical(cfg):
    """Nested pairs of the Order (Section 4.1) run on two streams with event
    waits on cross-stream edges only: 1F1B with its steady-state (F, B)
    pairs nested, and a split Order with (F, Bi), (F, Bw) and (Bi, Bw)
    pairs, give the flat 1F1B Order's outputs and gradient bit for bit, on
    two streams and with both streams the same."""
    banner(f"overlapped pairs {cfg.name}")
    flat, Xs, dYs = inputs(cfg, seed=8)
    M, P, s = cfg.num_microbatches, cfg.pp_size, cfg.pp_rank
    tol = 2e-2 if cfg.bf16 else 1e-4
    ref = gpu_run(cfg, OO.one_f_one_b(M, P, s), flat, Xs, dYs)
    aux = torch.cuda.Stream()
    cases = [(OO.one_f_one_b_overlap(M, P, s), 0), (OO.parse(SPLIT_PAIRS[M]), 2)]
    for order, wp in cases:
        assert OO.validate(order, M, M, max_w_pending=wp or M)[0] == "OK"
        assert any(isinstance(e, list) for e in order)
        # the oracle runs the same nested Order (its pairs in sequence)
        r = gpu_run(cfg, order, flat, Xs, dYs, max_w_pending=wp, aux_stream=aux)
        Ys, dXs, G = OS.run_order(cfg, flat, Xs, dYs, order)
        errs = per_tensor_errors(cfg, host(r.grad), G)
        for mb in range(M):
            errs[f"Y{mb}"] = rel_err(host(r.Y[mb]), Ys[mb])
            errs[f"dX{mb}"] = rel_err(host(r.dX[mb]), dXs[mb])
        report(errs)
        assert max(errs.values()) <= tol, (order, max(errs, key=errs.get))
        r.close()
        for stream in (aux, None):
            r = gpu_run(cfg, order, flat, Xs, dYs, max_w_pending=wp,
                        aux_stream=stream if stream is not None else torch.cuda.current_stream())
            torch.cuda.synchronize()
            assert torch.equal(r.grad, ref.grad), (order, stream)
            for mb in range(M):
                assert torch.equal(r.Y[mb], ref.Y[mb]) and torch.equal(r.dX[mb], ref.dX[mb])
            r.close()
    ref.close()


SMALL_MOE_ZERO = synth.StageConfig(
    name="small_moe_zero", n_layers=2, d_model=256, n_heads=2, head_dim=128, d_ff=0,
    seq_len=256, micro_batch=2, num_microbatches=3, bf16=True, n_experts=4, top_k=2,
    d_ff_expert=128, pp_size=3, pp_rank=0)


@pytest.mark.parametrize("cfg", [synth.TINY_FP32, SMALL_BF16, QWEN_BF16, SMALL_MOE_ZERO],
                         ids=["tiny_fp32", "small_bf16", "qwen_bf16", "small_moe"])
def test_zero_paths_give_the_accumulated_gradient_slices(cfg):
    """ZeRO-2/3 on one GPU (each backward into a temporary full gradient,
    then this rank's slice added into its persistent shard; at level 3 the
    weights gathered from shards before every entry): for each of three
    ranks' shards, the shard equals its slice of the plain Order's gradient
    bit for bit, and Y, dX are unchanged; also with split backwards."""
    banner(f"zero paths {cfg.name}")
    flat, Xs, dYs = inputs(cfg, seed=9)
    M, P, s = cfg.num_microbatches, cfg.pp_size, cfg.pp_rank
    tol = 2e-2 if cfg.bf16 else 1e-4
    ref = gpu_run(cfg, OO.one_f_one_b(M, P, s), flat, Xs, dYs)
    n = ref.n_params
    bounds = [0, (n // 3) // 4 * 4, (2 * n // 3) // 4 * 4 + 4, n]
    orders = [(OO.one_f_one_b(M, P, s), 0), (OO.one_f_one_b_split(M, P, s, 1), 2)]
    # the oracle's gradient: the three ranks' shards together must be it (a
    # mixture-of-experts stage's oracle takes the GPU's routing, as near-ties
    # may route either way)
    if cfg.moe:
        routes = gpu_routes(cfg, flat, Xs, dYs)
        _, _, G_ref = oracle_order_with_routes(cfg, flat, Xs, dYs, orders[0][0], routes)
    else:
        _, _, G_ref = OS.run_order(cfg, flat, Xs, dYs, orders[0][0])
    for level in (2, 3):
        for order, wp in orders:
            shards = []
            for rank in range(3):
                off, end = bounds[rank], bounds[rank + 1]
                r = StageRunner(desc_of(cfg), flat, M, max_w_pending=wp)
                r.alloc_microbatches(Xs, dYs)
                shard = torch.zeros(end - off, dtype=torch.float32, device="cuda")
                full = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda")
                w_shards, w_full = (), None
                if level == 3:
                    w_shards = [r.w[bounds[i]:bounds[i + 1]].clone() for i in range(3)]
                    w_full = torch.full_like(r.w, float("nan"))
                    r.w.fill_(float("nan"))  # ignored at level 3
                r.run_order_zero(to_c(order), level, shard, off, full, w_shards, w_full)
                torch.cuda.synchronize()
                assert torch.equal(shard, ref.grad[off:end]), (level, rank, wp)
                assert torch.all(r.grad == 0)  # params->grad is not touched
                for mb in range(M):
                    assert torch.equal(r.Y[mb], ref.Y[mb]) and torch.equal(r.dX[mb], ref.dX[mb])
                shards.append(host(shard))
                r.close()
            errs = per_tensor_errors(cfg, np.concatenate(shards), G_ref)
            report(errs, 3)
            assert max(errs.values()) <= tol, (level, wp, max(errs, key=errs.get))
    # ZeRO-3 with every weight shard already at its place in w_full (an
    # in-place gather): the same shard as the plain Order's slice
    r = StageRunner(desc_of(cfg), flat, M)
    r.alloc_microbatches(Xs, dYs)
    w_full = r.w.clone()
    r.w.fill_(float("nan"))
    shard = torch.zeros(bounds[2] - bounds[1], dtype=torch.float32, device="cuda")
    full = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda")
    r.run_order_zero(to_c(orders[0][0]), 3, shard, bounds[1], full,
                     [w_full[bounds[i]:bounds[i + 1]] for i in range(3)], w_full)
    torch.cuda.synchronize()
    assert torch.equal(shard, ref.grad[bounds[1]:bounds[2]])
    r.close()
    # bad layouts are rejected before anything is enqueued, and the stage
    # still runs an Order afterwards
    r = StageRunner(desc_of(cfg), flat, M)
    r.alloc_microbatches(Xs, dYs)
    shard = torch.zeros(8, dtype=torch.float32, device="cuda")
    full = torch.zeros(n + 64, dtype=torch.float32, device="cuda")
    wbuf = torch.empty(n + 64, dtype=r.w.dtype, device="cuda")
    order = to_c(OO.one_f_one_b(M, P, s))
    for bad in (dict(level=2, grad_shard=shard, shard_offset=2),
                dict(level=2, grad_shard=shard, shard_offset=n - 4),
                dict(level=4, grad_shard=shard, shard_offset=0),
                dict(level=3, grad_shard=shard, shard_offset=0,
                     w_shards=[r.w[:n // 2]], w_full=torch.empty_like(r.w)),
                # the shard is a view into the temporary full gradient
                dict(level=2, grad_shard=full[16:24], shard_offset=0, msg="overlap"),
                dict(level=2, grad_shard=full[n:n + 8], shard_offset=0, full=full[4:n + 4],
                     msg="overlap"),
                # a weight shard inside w_full, away from its own place
                dict(level=3, grad_shard=shard, shard_offset=0, w_full=wbuf[:n],
                     w_shards=[wbuf[8:8 + n // 2], r.w[n // 2:]], msg="overlap"),
                dict(level=3, grad_shard=shard, shard_offset=0, w_full=wbuf[:n],
                     w_shards=[r.w[:n // 2], wbuf[n // 2 + 8:n + 8]], msg="overlap")):
        with pytest.raises(lc.LibchunkError) as e:
            r.run_order_zero(order, bad["level"], bad["grad_shard"], bad["shard_offset"],
                             bad.get("full", full[:n]), bad.get("w_shards", ()), bad.get("w_full"))
        assert e.value.status == lc.LC_ERR_INVALID_ARG
        assert bad.get("msg", "") in str(e.value), str(e.value)
    torch.cuda.synchronize()
    r.run_order(order)
    torch.cuda.synchronize()
    assert torch.equal(r.grad, ref.grad)
    r.close()
    ref.close()


def test_split_backward_error_paths():
    cfg = SMALL_BF16
    banner("split backward error paths")
    flat, Xs, dYs = inputs(cfg, seed=7)
    r = StageRunner(desc_of(cfg), flat, 2)  # no weight-pass slots
    r.alloc_microbatches(Xs, dYs)
    r.forward(0)
    with pytest.raises(lc.LibchunkError) as e:
        r.backward_input(0)
    assert e.value.status == lc.LC_ERR_STASH_FULL
    with pytest.raises(lc.LibchunkError) as e:
        r.run_order(to_c(OO.parse("F0 Bi0 Bw0 F1 B1 F2 B2")))
    assert e.value.status == lc.LC_ERR_STASH_FULL  # rejected before any launch
    r.backward(0)
    r.close()
    r = StageRunner(desc_of(cfg), flat, 2, max_w_pending=1)
    r.alloc_microbatches(Xs, dYs)
    with pytest.raises(lc.LibchunkError) as e:
        r.backward_input(0)
    assert e.value.status == lc.LC_ERR_STATE
    r.forward(0)
    r.forward(1)
    with pytest.raises(lc.LibchunkError) as e:
        r.backward_weight(0)
    assert e.value.status == lc.LC_ERR_STATE
    r.backward_input(0)
    for call in (lambda: r.backward_input(0), lambda: r.backward(0)):
        with pytest.raises(lc.LibchunkError) as e:
            call()
        assert e.value.status == lc.LC_ERR_STATE
    with pytest.raises(lc.LibchunkError) as e:
        r.backward_input(1)
    assert e.value.status == lc.LC_ERR_STASH_FULL  # the one weight slot is taken
    with pytest.raises(lc.LibchunkError) as e:
        r.forward(2)
    assert e.value.status == lc.LC_ERR_STASH_FULL  # microbatch 0 still holds its stash
    r.backward_weight(0)
    r.backward(1)
    with pytest.raises(lc.LibchunkError) as e:
        r.backward_weight(0)
    assert e.value.status == lc.LC_ERR_STATE
    torch.cuda.synchronize()
    r.close()


@pytest.mark.parametrize("cfg,tol", [(synth.STAGE_7B, 2e-2),
                                     (synth.scaled(synth.STAGE_7B, bf16=False), 1e-4),
                                     (synth.QWEN3_STAGE, 2e-2), (synth.LLAMA_2K, 2e-2)],
                         ids=["stage7b_bf16", "stage7b_fp32", "qwen3_bf16", "llama2k_bf16"])
def test_full_size_stage_on_a_prefix(cfg, tol):
    P = 128
    banner(f"full-size {cfg.name} prefix {P}")
    flat = synth.stage_params(cfg, 0)
    X = synth.activation(cfg, 0, 0, "x")
    dY = synth.activation(cfg, 0, 0, "dy")
    dY[:, P:] = 0.0
    r = StageRunner(desc_of(cfg), flat, 1)
    r.alloc_microbatches([X], [dY])
    r.forward(0)
    r.backward(0)
    torch.cuda.synchronize()
    Yg = host(r.Y[0])
    dXg = host(r.dX[0])
    Gg = host(r.grad)
    r.close()
    del r
    torch.cuda.empty_cache()
    layers = OS.layer_params(cfg, flat)
    Yp, caches = OS.stage_forward(cfg, layers, X[:, :P])
    dXp, Gp = OS.stage_backward(cfg, layers, caches, dY[:, :P])
    print(f"Y prefix err {rel_err(Yg[:, :P], Yp):.2e}, dX prefix err {rel_err(dXg[:, :P], dXp):.2e}")
    assert rel_err(Yg[:, :P], Yp) <= tol
    assert rel_err(dXg[:, :P], dXp) <= tol
    assert np.all(dXg[:, P:] == 0.0)
    errs = per_tensor_errors(cfg, Gg, Gp)
    report(errs, 12)
    worst = max(errs, key=errs.get)
    assert errs[worst] <= tol, (worst, errs[worst])


FULL_LENGTH = [
    synth.scaled(synth.STAGE_7B, name="stage7b_1L_s4096", n_layers=1, num_microbatches=1),
    synth.scaled(synth.QWEN3_STAGE, name="qwen3_1L_s4096", n_layers=1, num_microbatches=1),
    synth.scaled(synth.LLAMA_2K, name="llama_2L_s2048", n_layers=2, num_microbatches=1),
]


@pytest.mark.parametrize("cfg", FULL_LENGTH, ids=["stage7b_1L", "qwen3_1L", "llama2k_2L"])
def test_full_length_layers(cfg):
    """Layers of the benchmark shapes over whole sequences (4096 tokens for
    the 7B- and Qwen3-shaped layers, 2048 for the Llama-style ones) with dY
    nonzero everywhere: Y, dX and every gradient tensor against the oracle
    at every position, so the long key loops of attention, its heavy-first
    block order and the long-context terms of every weight gradient are all
    compared. The margin to the 2e-2 tolerance is printed."""
    tol = 2e-2
    banner(f"full-length {cfg.name}")
    flat = synth.stage_params(cfg, 0)
    X = synth.activation(cfg, 0, 0, "x")
    dY = synth.activation(cfg, 0, 0, "dy")
    r = StageRunner(desc_of(cfg), flat, 1)
    r.alloc_microbatches([X], [dY])
    r.forward(0)
    r.backward(0)
    torch.cuda.synchronize()
    Yg, dXg, Gg = host(r.Y[0]), host(r.dX[0]), host(r.grad)
    r.close()
    del r
    torch.cuda.empty_cache()
    banner(f"full-length {cfg.name}: oracle")
    layers = OS.layer_params(cfg, flat)
    Yr, caches = OS.stage_forward(cfg, layers, X)
    dXr, Gr = OS.stage_backward(cfg, layers, caches, dY)
    errs = per_tensor_errors(cfg, Gg, Gr)
    errs["Y"] = rel_err(Yg, Yr)
    errs["dX"] = rel_err(dXg, dXr)
    report(errs, 12)
    worst = max(errs, key=errs.get)
    print(f"margin: worst {worst} {errs[worst]:.2e} = {errs[worst] / tol:.0%} of {tol}", flush=True)
    assert errs[worst] <= tol, (worst, errs[worst])


@pytest.mark.parametrize("cfg", [synth.STAGE_7B, synth.MOE_2K], ids=["7b", "moe"])
def test_full_size_split_backward_is_bit_identical(cfg):
    """The 7B-shaped and the mixture-of-experts stage at full size, two
    microbatches: the split Order (Bi0 Bi1 Bw0 Bw1, two weight passes
    pending) gives the plain Order's dX and gradient bit for bit."""
    from paper_2606_11169_amd.runner import random_stage
    banner(f"full-size split backward {cfg.name}")
    P = cfg.pp_size
    got = []
    for order, wp in ((OO.one_f_one_b(2, P, 0), 0), (OO.one_f_one_b_split(2, P, 0, 1), 2)):
        r = random_stage(desc_of(cfg), 2, seed=1, max_w_pending=wp)
        r.alloc_random_microbatches(2, seed=2)
        r.run_order(to_c(order))
        torch.cuda.synchronize()
        got.append((r.grad.clone(), [t.clone() for t in r.dX], [t.clone() for t in r.Y]))
        r.close()
        del r
        torch.cuda.empty_cache()
    (ga, dxa, ya), (gb, dxb, yb) = got
    assert torch.isfinite(ga).all() and ga.abs().max() > 0
    assert torch.equal(ga, gb)
    for mb in range(2):
        assert torch.equal(dxa[mb], dxb[mb]) and torch.equal(ya[mb], yb[mb])


def test_full_size_overlapped_pair_is_bit_identical():
    """The 7B-shaped stage: F0 [F1 B0] B1 with the pair on two streams gives
    the flat Order's dX, Y and gradient bit for bit."""
    from paper_2606_11169_amd.runner import random_stage
    cfg = synth.STAGE_7B
    banner("full-size overlapped pair")
    got = []
    aux = torch.cuda.Stream()
    for order, stream in ((OO.parse("F0 F1 B0 B1"), None), (OO.parse("F0 [F1 B0] B1"), aux)):
        r = random_stage(desc_of(cfg), 2, seed=1)
        r.alloc_random_microbatches(2, seed=2)
        r.run_order(to_c(order), stream)
        torch.cuda.synchronize()
        got.append((r.grad.clone(), [t.clone() for t in r.dX], [t.clone() for t in r.Y]))
        r.close()
        del r
        torch.cuda.empty_cache()
    (ga, dxa, ya), (gb, dxb, yb) = got
    assert torch.isfinite(ga).all() and ga.abs().max() > 0
    assert torch.equal(ga, gb)
    for mb in range(2):
        assert torch.equal(dxa[mb], dxb[mb]) and torch.equal(ya[mb], yb[mb])
