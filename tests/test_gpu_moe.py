"""Parity of the mixture-of-experts path (router, dispatch, grouped expert
products, the whole MoE stage) with the oracle.

* router: the selected experts agree with the oracle's top-2 of its float64
  softmax on the same bf16 inputs except where the two candidates' oracle
  probabilities are within 1e-4 (near-ties fp32 logits may order either
  way); gate weights within 1e-5; the zero-router closed form (ties to
  experts 0 and 1, weights exactly 1/2)
* dispatch: offsets, permutation, row positions and row weights bit-exact
  against the oracle's grouping of the GPU's own routing (integer work)
* grouped products: integer-valued operands make every sum exact, so each
  group's rows / k range are compared bit for bit, with empty groups and
  groups that end inside a tile
* MoE stage: Y, dX and every gradient tensor within 2e-2 of the oracle run
  with the GPU's routing as a routing override (the gate weights still come
  from the oracle's own logits); the GPU routing differs from the oracle's
  own routing only at near-ties (probability gap below 1e-2)
"""
import numpy as np
import pytest
import torch

import synth
from oracle import stage as OS
from paper_2606_11169_amd import libchunk as lc
from paper_2606_11169_amd.runner import StageRunner, require_gpu
from tests.gpu_util import (DEV, banner, bf16, check_routing_near_ties, f32, gpu_routes, host,
                            oracle_order_with_routes, rel_err)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


def bf16_round(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16).float().numpy()


def i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(DEV)


def random_routing(rng, T, E):
    sel = np.stack([rng.choice(E, size=2, replace=False) for _ in range(T)]).astype(np.int32)
    w0 = rng.uniform(0.5, 1.0, size=T).astype(np.float32)
    return sel, np.stack([w0, 1.0 - w0], axis=1).astype(np.float32)


# ---------------------------------------------------------------- router

@pytest.mark.parametrize("T,d,E", [(1000, 256, 8), (129, 512, 2), (64, 128, 64)])
def test_router_matches_oracle(T, d, E):
    banner(f"moe route T={T} d={d} E={E}")
    rng = np.random.default_rng(T + d + E)
    n = bf16_round(rng.standard_normal((T, d)))
    wr = bf16_round(0.02 * rng.standard_normal((E, d)))
    sel = torch.empty((T, 2), dtype=torch.int32, device=DEV)
    w = torch.empty((T, 2), dtype=torch.float32, device=DEV)
    lc.lc_moe_route(T, d, E, bf16(n), bf16(wr), sel, w, lc.LC_BF16, lc.LC_BF16)
    torch.cuda.synchronize()
    gs, gw = sel.cpu().numpy(), host(w)
    _, pi, osel, ow = OS.moe_route(n.astype(np.float64), wr.astype(np.float64), 2)
    assert np.all(gs[:, 0] != gs[:, 1])
    rows = np.arange(T)
    same = np.all(gs == osel, axis=1)
    for t in np.nonzero(~same)[0]:
        gap = np.max(np.abs(pi[t, gs[t]] - pi[t, osel[t]]))
        assert gap < 1e-4, f"token {t}: GPU {gs[t]} vs oracle {osel[t]}, probability gap {gap}"
    assert np.max(np.abs(gw[same] - ow[same])) <= 1e-5
    assert same.mean() > 0.99
    del rows


def test_router_zero_weights_tie_to_lowest_experts():
    banner("moe route zero router")
    T, d, E = 300, 256, 8
    n = bf16_round(np.random.default_rng(1).standard_normal((T, d)))
    sel = torch.empty((T, 2), dtype=torch.int32, device=DEV)
    w = torch.empty((T, 2), dtype=torch.float32, device=DEV)
    lc.lc_moe_route(T, d, E, bf16(n), bf16(np.zeros((E, d))), sel, w, lc.LC_BF16, lc.LC_BF16)
    torch.cuda.synchronize()
    assert np.all(sel.cpu().numpy() == np.array([0, 1]))
    assert np.all(host(w) == 0.5)


# ---------------------------------------------------------------- dispatch

@pytest.mark.parametrize("T,E", [(1, 2), (1000, 8), (3000, 8), (2500, 64), (1024, 3)])
def test_dispatch_bit_exact(T, E):
    banner(f"moe dispatch T={T} E={E}")
    rng = np.random.default_rng(7 * T + E)
    sel, w = random_routing(rng, T, E)
    off = torch.full((E + 1,), -7, dtype=torch.int32, device=DEV)
    perm = torch.full((2 * T,), -7, dtype=torch.int32, device=DEV)
    wrow = torch.full((2 * T,), -7.0, dtype=torch.float32, device=DEV)
    rowpos = torch.full((T, 2), -7, dtype=torch.int32, device=DEV)
    lc.lc_moe_dispatch(T, E, i32(sel), f32(w), off, perm, wrow, rowpos)
    torch.cuda.synchronize()
    ooff, operm, orowpos = OS.moe_dispatch(sel, E)
    assert np.array_equal(off.cpu().numpy(), ooff)
    assert np.array_equal(perm.cpu().numpy(), operm)
    assert np.array_equal(rowpos.cpu().numpy(), orowpos)
    slot = np.zeros(2 * T, np.int64)
    for k in range(2):
        slot[orowpos[:, k]] = k
    want = w[operm, slot]
    assert np.array_equal(wrow.cpu().numpy().view(np.uint32), want.view(np.uint32))


def test_dispatch_skips_invalid_pairs():
    """A repeated or out-of-range expert is not placed (rowpos -1); the rows
    past the placed ones read token 0 with weight 0."""
    banner("moe dispatch invalid pairs")
    T, E = 5, 4
    sel = np.array([[0, 1], [2, 2], [3, 9], [1, 0], [-1, 3]], np.int32)
    w = np.full((T, 2), 0.5, np.float32)
    off = torch.empty(E + 1, dtype=torch.int32, device=DEV)
    perm = torch.full((2 * T,), -7, dtype=torch.int32, device=DEV)
    wrow = torch.full((2 * T,), -7.0, dtype=torch.float32, device=DEV)
    rowpos = torch.full((T, 2), -7, dtype=torch.int32, device=DEV)
    lc.lc_moe_dispatch(T, E, i32(sel), f32(w), off, perm, wrow, rowpos)
    torch.cuda.synchronize()
    assert off.cpu().numpy().tolist() == [0, 2, 4, 5, 7]
    assert perm.cpu().numpy().tolist() == [0, 3, 0, 3, 1, 2, 4, 0, 0, 0]
    assert rowpos.cpu().numpy().tolist() == [[0, 2], [4, -1], [5, -1], [3, 1], [-1, 6]]
    assert host(wrow).tolist()[7:] == [0.0, 0.0, 0.0]


# ---------------------------------------------------------------- grouped products

def ints(rng, shape, lo=-8, hi=8):
    return rng.integers(lo, hi + 1, size=shape).astype(np.float32)


@pytest.mark.parametrize("b_kmajor", [True, False], ids=["NT", "NN"])
def test_grouped_rows_bit_exact(b_kmajor):
    banner(f"grouped rows b_kmajor={b_kmajor}")
    rng = np.random.default_rng(3)
    sizes = [300, 0, 17, 512, 256, 1]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    G, R, N, K = len(sizes), int(off[-1]) + 40, 264, 200
    A = ints(rng, (R, K))
    Bs = [ints(rng, (N, K)) for _ in range(G)]
    stride = N * K
    Bflat = np.concatenate([(b if b_kmajor else b.T.copy()).ravel() for b in Bs])
    C = torch.full((R, N), -1.0, dtype=torch.float32, device=DEV)
    lc.lc_gemm(lc.LC_BF16, lc.LC_EPI_STORE_F32, R, N, K, bf16(A), K, 1, bf16(Bflat),
               K if b_kmajor else N, int(b_kmajor), C, N, group_mode=lc.LC_GROUP_ROWS,
               n_groups=G, group_offsets=i32(off), group_stride_b=stride)
    torch.cuda.synchronize()
    got = host(C)
    for g in range(G):
        rows = slice(off[g], off[g + 1])
        want = A[rows].astype(np.int64) @ Bs[g].astype(np.int64).T
        assert np.array_equal(got[rows], want.astype(np.float64)), f"group {g}"
    assert np.all(got[off[-1]:] == -1.0)  # rows past the last group untouched


def test_grouped_swiglu_rows_matches_per_group():
    banner("grouped rows swiglu")
    rng = np.random.default_rng(4)
    sizes = [130, 0, 400]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    G, R, F, D = len(sizes), int(off[-1]), 128, 256
    A = bf16_round(rng.standard_normal((R, D)))
    W = [bf16_round(0.05 * rng.standard_normal((2 * F, D))) for _ in range(G)]
    act = torch.empty((R, F), dtype=torch.bfloat16, device=DEV)
    gate = torch.empty((R, F), dtype=torch.float32, device=DEV)
    up = torch.empty_like(gate)
    lc.lc_gemm(lc.LC_BF16, lc.LC_EPI_SWIGLU, R, F, D, bf16(A), D, 1,
               bf16(np.concatenate([w.ravel() for w in W])), D, 1, act, F, aux0=gate, aux1=up,
               ld_aux=F, aux_dtype=lc.LC_FP32, group_mode=lc.LC_GROUP_ROWS, n_groups=G,
               group_offsets=i32(off), group_stride_b=2 * F * D)
    torch.cuda.synchronize()
    for g in range(G):
        rows = slice(off[g], off[g + 1])
        gt = A[rows].astype(np.float64) @ W[g][:F].T.astype(np.float64)
        u = A[rows].astype(np.float64) @ W[g][F:].T.astype(np.float64)
        if sizes[g] == 0:
            continue
        assert rel_err(host(gate)[rows], gt) <= 1e-5
        assert rel_err(host(up)[rows], u) <= 1e-5
        a = gt / (1.0 + np.exp(-gt)) * u
        assert rel_err(host(act)[rows], a) <= 1e-2


def test_grouped_k_bit_exact():
    banner("grouped k")
    rng = np.random.default_rng(5)
    sizes = [70, 0, 300, 1, 257]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    G, Ktot, M, N = len(sizes), int(off[-1]) + 9, 264, 136
    A = ints(rng, (Ktot, M))   # A(m, k) = A[k, m]
    B = ints(rng, (Ktot, N))   # B(n, k) = B[k, n]
    C0 = ints(rng, (G, M, N), -1000, 1000)
    C = f32(C0.reshape(-1))
    lc.lc_gemm(lc.LC_BF16, lc.LC_EPI_ACCUM_F32, M, N, Ktot, bf16(A), M, 0, bf16(B), N, 0, C, N,
               group_mode=lc.LC_GROUP_K, n_groups=G, group_offsets=i32(off),
               group_stride_c=M * N)
    torch.cuda.synchronize()
    got = host(C).reshape(G, M, N)
    for g in range(G):
        ks = slice(off[g], off[g + 1])
        want = C0[g] + (A[ks].astype(np.int64).T @ B[ks].astype(np.int64))
        assert np.array_equal(got[g], want.astype(np.float64)), f"group {g}"


# ---------------------------------------------------------------- stage

SMALL_MOE = synth.StageConfig(
    name="small_moe", n_layers=2, d_model=256, n_heads=2, head_dim=128, d_ff=0, seq_len=256,
    micro_batch=2, num_microbatches=2, bf16=True, n_experts=4, top_k=2, d_ff_expert=128,
    pp_size=2, pp_rank=0)


def desc_of(cfg):
    return lc.desc_of_config(cfg)


# Qwen3-MoE-style attention on a mixture-of-experts stage: grouped-query
# attention (4 query heads over 2 key/value heads) with per-head q/k RMSNorm
SMALL_MOE_QK = synth.StageConfig(
    name="small_moe_qk", n_layers=2, d_model=512, n_heads=4, head_dim=128, d_ff=0, seq_len=256,
    micro_batch=2, num_microbatches=2, bf16=True, n_experts=4, top_k=2, d_ff_expert=128,
    n_kv_heads=2, qk_norm=True, rms_eps=1e-6, rope_base=1000000.0, pp_size=2, pp_rank=0)


@pytest.mark.parametrize("cfg", [SMALL_MOE, SMALL_MOE_QK], ids=["mha", "gqa_qknorm"])
def test_moe_stage_matches_oracle_with_gpu_routing(cfg):
    banner(f"moe stage {cfg.name}")
    M = cfg.num_microbatches
    flat = synth.stage_params(cfg, 0)
    Xs = [synth.activation(cfg, 0, mb, "x") for mb in range(M)]
    dYs = [synth.activation(cfg, 0, mb, "dy") for mb in range(M)]
    r = StageRunner(desc_of(cfg), flat, M)
    r.alloc_microbatches(Xs, dYs)
    routes = []
    for mb in range(M):
        r.forward(mb)
        routes.append([r.moe_routing(mb, l) for l in range(cfg.n_layers)])
    for mb in range(M):
        r.backward(mb)
    torch.cuda.synchronize()
    layers = OS.layer_params(cfg, flat)
    G = np.zeros(synth.param_count(cfg))
    errs = {}
    near_tie_mismatches = 0
    for mb in range(M):
        Y, caches = OS.stage_forward(cfg, layers, Xs[mb], route_overrides=routes[mb])
        for l in range(cfg.n_layers):
            pi = caches[l]["moe"]["pi"]
            own = np.argsort(-pi, axis=1, kind="stable")[:, :2]
            g = routes[mb][l]
            diff = ~np.all(own == g, axis=1)
            for t in np.nonzero(diff)[0]:
                gap = np.max(np.abs(pi[t, g[t]] - pi[t, own[t]]))
                assert gap < 1e-2, f"mb {mb} layer {l} token {t}: routing gap {gap}"
            near_tie_mismatches += int(diff.sum())
        dX, gmb = OS.stage_backward(cfg, layers, caches, dYs[mb])
        G += gmb
        errs[f"Y{mb}"] = rel_err(host(r.Y[mb]), Y)
        errs[f"dX{mb}"] = rel_err(host(r.dX[mb]), dX)
    got = host(r.grad)
    for name, off, shape in synth.layout(cfg):
        sz = int(np.prod(shape))
        errs[name] = rel_err(got[off:off + sz], G[off:off + sz])
    top = sorted(errs.items(), key=lambda kv: -kv[1])[:6]
    print("worst tensors: " + ", ".join(f"{n}={e:.2e}" for n, e in top)
          + f"; routing differs from the oracle's own at {near_tie_mismatches} near-ties",
          flush=True)
    assert max(errs.values()) <= 2e-2
    r.close()


def test_moe_stage_with_an_expert_that_receives_no_tokens():
    """Router rows u, -u, 0, 0 in every layer: each token picks the positive
    one of experts 0 and 1, then expert 2 (experts 2 and 3 tie at logit 0,
    the lower index wins), so expert 3 gets no rows. Its weight gradients and
    its router row's gradient are exactly zero, and every output and gradient
    matches the oracle given the GPU's routing (the oracle's own routing
    agrees except where u.n2 is within rounding of 0). Split backwards give
    the same gradient and dX bit for bit."""
    cfg = SMALL_MOE
    banner("moe stage with an unused expert")
    M, E, d = cfg.num_microbatches, cfg.n_experts, cfg.d_model
    flat = synth.stage_params(cfg, 2)
    named = synth.unflatten(cfg, flat)
    rng = np.random.default_rng(41)
    for l in range(cfg.n_layers):
        u = bf16_round(rng.standard_normal(d) / np.sqrt(d))
        wr = named[f"L{l}.wr"]
        wr[:] = 0.0
        wr[0], wr[1] = u, -u
    flat = synth.flatten(cfg, named, dtype=np.float32)
    Xs = [synth.activation(cfg, 2, mb, "x") for mb in range(M)]
    dYs = [synth.activation(cfg, 2, mb, "dy") for mb in range(M)]
    r = StageRunner(desc_of(cfg), flat, M)
    r.alloc_microbatches(Xs, dYs)
    routes = []
    for mb in range(M):
        r.forward(mb)
        routes.append([r.moe_routing(mb, l) for l in range(cfg.n_layers)])
    for mb in range(M):
        r.backward(mb)
    torch.cuda.synchronize()
    for mb in range(M):
        for l in range(cfg.n_layers):
            sel = routes[mb][l]
            assert np.all(sel[:, 1] == 2) and np.all(np.isin(sel[:, 0], (0, 1))), (mb, l)
    # the same microbatches with split backwards (all Bi, then all Bw): the
    # unused expert's grouped weight products run over empty groups there too
    rs = StageRunner(desc_of(cfg), flat, M, max_w_pending=M)
    rs.alloc_microbatches(Xs, dYs)
    for mb in range(M):
        rs.forward(mb)
    for mb in range(M):
        rs.backward_input(mb)
    for mb in range(M):
        rs.backward_weight(mb)
    torch.cuda.synchronize()
    assert torch.equal(rs.grad, r.grad)
    for mb in range(M):
        assert torch.equal(rs.dX[mb], r.dX[mb])
    rs.close()
    got = host(r.grad)
    gg = synth.unflatten(cfg, got)
    for l in range(cfg.n_layers):
        for t in ("w1", "w3", "w2"):
            assert np.all(gg[f"L{l}.e3.{t}"] == 0.0), (l, t)
            assert np.any(gg[f"L{l}.e2.{t}"] != 0.0), (l, t)
        assert np.all(gg[f"L{l}.wr"][3] == 0.0) and np.any(gg[f"L{l}.wr"][2] != 0.0)
    layers = OS.layer_params(cfg, flat)
    G = np.zeros(synth.param_count(cfg))
    errs = {}
    for mb in range(M):
        Y, caches = OS.stage_forward(cfg, layers, Xs[mb], route_overrides=routes[mb])
        for l in range(cfg.n_layers):
            pi = caches[l]["moe"]["pi"]
            own = np.argsort(-pi, axis=1, kind="stable")[:, :2]
            for t in np.nonzero(~np.all(own == routes[mb][l], axis=1))[0]:
                assert abs(pi[t, 0] - pi[t, 1]) < 1e-2, (mb, l, t)
        dX, gmb = OS.stage_backward(cfg, layers, caches, dYs[mb])
        G += gmb
        errs[f"Y{mb}"] = rel_err(host(r.Y[mb]), Y)
        errs[f"dX{mb}"] = rel_err(host(r.dX[mb]), dX)
    for name, off, shape in synth.layout(cfg):
        sz = int(np.prod(shape))
        if np.any(G[off:off + sz] != 0.0):
            errs[name] = rel_err(got[off:off + sz], G[off:off + sz])
        else:
            assert np.all(got[off:off + sz] == 0.0), name
    top = sorted(errs.items(), key=lambda kv: -kv[1])[:6]
    print("worst tensors: " + ", ".join(f"{n}={e:.2e}" for n, e in top), flush=True)
    assert max(errs.values()) <= 2e-2
    r.close()


def test_moe_overlapped_pair_on_two_streams_is_bit_identical():
    """A mixture-of-experts stage with its (F1, B0) pair nested and run on two
    streams gives the flat Order's outputs and gradient bit for bit."""
    cfg = SMALL_MOE
    banner(f"moe overlapped pair {cfg.name}")
    M = cfg.num_microbatches
    flat = synth.stage_params(cfg, 1)
    Xs = [synth.activation(cfg, 1, mb, "x") for mb in range(M)]
    dYs = [synth.activation(cfg, 1, mb, "dy") for mb in range(M)]
    F, B, NX = lc.LC_PASS_F, lc.LC_PASS_B, lc.LC_ORDER_WITH_NEXT
    aux = torch.cuda.Stream()
    runs = []
    for order, stream in (([(0, F), (1, F), (0, B), (1, B)], None),
                          ([(0, F), (1, F | NX), (0, B), (1, B)], aux)):
        r = StageRunner(desc_of(cfg), flat, M)
        r.alloc_microbatches(Xs, dYs)
        r.run_order(order, stream)
        torch.cuda.synchronize()
        runs.append(r)
    a, b = runs
    assert torch.equal(a.grad, b.grad)
    for mb in range(M):
        assert torch.equal(a.Y[mb], b.Y[mb]) and torch.equal(a.dX[mb], b.dX[mb])
    # and against the oracle running the same nested Order, given the GPU's
    # routing (a forward per microbatch on a fresh stage reads it back)
    oracle_order = [(0, "F"), [(1, "F"), (0, "B")], (1, "B")]
    check_order_against_oracle(cfg, flat, Xs, dYs, oracle_order, b)
    for r in runs:
        r.close()


def check_order_against_oracle(cfg, flat, Xs, dYs, order, run, tol=2e-2):
    """Y, dX and every gradient tensor of a GPU run of `order` against the
    oracle executing the same Order (its nested pairs in sequence; Bw adds
    the gradient Bi computed), with the GPU's routing as the override."""
    routes = gpu_routes(cfg, flat, Xs, dYs)
    Ys, dXs, G = oracle_order_with_routes(cfg, flat, Xs, dYs, order, routes)
    M = len(Xs)
    errs = {}
    got = host(run.grad)
    for name, off, shape in synth.layout(cfg):
        sz = int(np.prod(shape))
        errs[name] = rel_err(got[off:off + sz], G[off:off + sz])
    for mb in range(M):
        errs[f"Y{mb}"] = rel_err(host(run.Y[mb]), Ys[mb])
        errs[f"dX{mb}"] = rel_err(host(run.dX[mb]), dXs[mb])
    top = sorted(errs.items(), key=lambda kv: -kv[1])[:4]
    print("vs oracle, worst: " + ", ".join(f"{n}={e:.2e}" for n, e in top), flush=True)
    assert max(errs.values()) <= tol, max(errs, key=errs.get)


@pytest.mark.parametrize("w_delay", [0, 1, 2])
def test_moe_split_backward_is_bit_identical(w_delay):
    """A mixture-of-experts stage under 1F1B with split backwards (Bi, then Bw
    w_delay backwards later): the Bi passes leave the routed dy rows, the
    experts' [dgate | dup] and the router logit gradients in weight-pass
    slots, the Bw passes add the expert, router and attention weight
    gradients; outputs and gradient equal the plain 1F1B Order's bit for
    bit. The split pairs of the overlapped split Order on two streams give
    the same bits too."""
    cfg = SMALL_MOE
    banner(f"moe split backward {cfg.name} w_delay {w_delay}")
    M = cfg.num_microbatches
    flat = synth.stage_params(cfg, 2)
    Xs = [synth.activation(cfg, 2, mb, "x") for mb in range(M)]
    dYs = [synth.activation(cfg, 2, mb, "dy") for mb in range(M)]
    P, s = 3, 0
    plain = lc.lc_order_1f1b(M, P, s)
    split = lc.lc_order_1f1b_split(M, P, s, w_delay)
    assert any(p & ~lc.LC_ORDER_WITH_NEXT == lc.LC_PASS_BW for _, p in split)
    wp = min(w_delay + 1, M)
    runs = []
    for order, mwp in ((plain, 0), (split, wp)):
        r = StageRunner(desc_of(cfg), flat, M, max_w_pending=mwp)
        r.alloc_microbatches(Xs, dYs)
        r.run_order(order)
        torch.cuda.synchronize()
        runs.append(r)
    a, b = runs
    assert torch.equal(a.grad, b.grad)
    for mb in range(M):
        assert torch.equal(a.Y[mb], b.Y[mb]) and torch.equal(a.dX[mb], b.dX[mb])
    b.close()
    # the split Order with its first adjacent (Bi, Bw) of two microbatches run
    # as an overlapped pair (Bi first), with a weight-pass slot for each
    BI, BW, NX = lc.LC_PASS_BI, lc.LC_PASS_BW, lc.LC_ORDER_WITH_NEXT
    nested = list(split)
    for i in range(len(nested) - 1):
        (m1, p1), (m2, p2) = nested[i], nested[i + 1]
        if {p1, p2} == {BI, BW} and m1 != m2:
            bi, bw = ((m1, p1), (m2, p2)) if p1 == BI else ((m2, p2), (m1, p1))
            nested[i:i + 2] = [(bi[0], BI | NX), bw]
            break
    else:
        pytest.fail(f"no adjacent (Bi, Bw) pair in {split}")
    gen = lc.lc_order_1f1b_split_overlap(M, P, s, w_delay)  # the generator's nesting
    for k, order in enumerate((nested, gen)):
        c = StageRunner(desc_of(cfg), flat, M, max_w_pending=M)
        c.alloc_microbatches(Xs, dYs)
        c.run_order(order, torch.cuda.Stream())
        torch.cuda.synchronize()
        assert torch.equal(a.grad, c.grad)
        for mb in range(M):
            assert torch.equal(a.dX[mb], c.dX[mb])
        if k == 1:
            check_order_against_oracle(cfg, flat, Xs, dYs, c_to_oracle(order), c)
        c.close()
    a.close()


def c_to_oracle(entries):
    """C Order entries -> the oracle's Order (a flagged entry and the next
    one form a nested pair)."""
    names = {lc.LC_PASS_F: "F", lc.LC_PASS_B: "B", lc.LC_PASS_BI: "Bi", lc.LC_PASS_BW: "Bw"}
    out, i = [], 0
    while i < len(entries):
        mb, p = entries[i]
        if p & lc.LC_ORDER_WITH_NEXT:
            mb2, p2 = entries[i + 1]
            out.append([(mb, names[p & ~lc.LC_ORDER_WITH_NEXT]), (mb2, names[p2])])
            i += 2
        else:
            out.append((mb, names[p]))
            i += 1
    return out


def test_full_length_moe_layer():
    """One layer of the mixture-of-experts workload (d 2048, 8 experts x
    1408, 2 x 2048 tokens) over whole sequences with dY nonzero everywhere:
    the GPU's routing agrees with the oracle's own top-2 except at near-ties,
    and Y, dX and every gradient tensor match the oracle run with the GPU's
    routing at every position."""
    cfg = synth.scaled(synth.MOE_2K, name="moe_1L_s2048", n_layers=1, num_microbatches=1)
    banner(f"full-length {cfg.name}")
    flat = synth.stage_params(cfg, 0)
    X = synth.activation(cfg, 0, 0, "x")
    dY = synth.activation(cfg, 0, 0, "dy")
    r = StageRunner(desc_of(cfg), flat, 1)
    r.alloc_microbatches([X], [dY])
    r.forward(0)
    route = [r.moe_routing(0, l) for l in range(cfg.n_layers)]
    r.backward(0)
    torch.cuda.synchronize()
    Yg, dXg, Gg = host(r.Y[0]), host(r.dX[0]), host(r.grad)
    r.close()
    del r
    torch.cuda.empty_cache()
    layers = OS.layer_params(cfg, flat)
    Yr, caches = OS.stage_forward(cfg, layers, X, route_overrides=route)
    mism = check_routing_near_ties(caches, route)
    dXr, Gr = OS.stage_backward(cfg, layers, caches, dY)
    errs = {"Y": rel_err(Yg, Yr), "dX": rel_err(dXg, dXr)}
    for name, off, shape in synth.layout(cfg):
        sz = int(np.prod(shape))
        errs[name] = rel_err(Gg[off:off + sz], Gr[off:off + sz])
    top = sorted(errs.items(), key=lambda kv: -kv[1])[:8]
    print("worst tensors: " + ", ".join(f"{n}={e:.2e}" for n, e in top)
          + f"; {mism} near-tie routing differences", flush=True)
    assert max(errs.values()) <= 2e-2


def test_full_size_moe_stage_on_a_prefix():
    """The MoE workload at full size (4 layers, d 2048, 8 experts x 1408,
    2 x 2048 tokens): outputs and gradients on a 128-token prefix of each
    sequence against the oracle run on that prefix with the GPU's routing of
    those tokens (routing is per token, and causality keeps the prefix
    self-contained); dY is zero past the prefix, so the full-size backward
    is checked too and dX past the prefix must be exactly 0."""
    cfg = synth.MOE_2K
    P, S = 128, cfg.seq_len
    banner(f"full-size {cfg.name} prefix {P}")
    flat = synth.stage_params(cfg, 0)
    X = synth.activation(cfg, 0, 0, "x")
    dY = synth.activation(cfg, 0, 0, "dy")
    dY[:, P:] = 0.0
    r = StageRunner(desc_of(cfg), flat, 1)
    r.alloc_microbatches([X], [dY])
    r.forward(0)
    route = [r.moe_routing(0, l) for l in range(cfg.n_layers)]
    r.backward(0)
    torch.cuda.synchronize()
    Yg, dXg, Gg = host(r.Y[0]), host(r.dX[0]), host(r.grad)
    r.close()
    del r
    torch.cuda.empty_cache()
    rows = np.concatenate([np.arange(b * S, b * S + P) for b in range(cfg.micro_batch)])
    override = [rt[rows] for rt in route]
    layers = OS.layer_params(cfg, flat)
    Yp, caches = OS.stage_forward(cfg, layers, X[:, :P], route_overrides=override)
    mism = check_routing_near_ties(caches, override)
    print(f"routing differs from the oracle's own top-2 at {mism} near-ties", flush=True)
    dXp, Gp = OS.stage_backward(cfg, layers, caches, dY[:, :P])
    errs = {"Y": rel_err(Yg[:, :P], Yp), "dX": rel_err(dXg[:, :P], dXp)}
    assert np.all(dXg[:, P:] == 0.0)
    for name, off, shape in synth.layout(cfg):
        sz = int(np.prod(shape))
        errs[name] = rel_err(Gg[off:off + sz], Gp[off:off + sz])
    top = sorted(errs.items(), key=lambda kv: -kv[1])[:8]
    print("worst tensors: " + ", ".join(f"{n}={e:.2e}" for n, e in top), flush=True)
    assert max(errs.values()) <= 2e-2
