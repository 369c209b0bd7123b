"""Helpers shared by the GPU tests: device transfers and error metrics."""
import sys

import numpy as np
import torch

import synth
from oracle import optim as OP
from oracle import order as OO
from oracle import stage as OS

DEV = "cuda"


def banner(msg):
    """Names the case before a GPU step, so an abort still identifies it."""
    print(f"[gpu case] {msg}", flush=True)
    sys.stdout.flush()


def f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(DEV)


def bf16(a):
    """float32 array of bf16-representable values -> bf16 device tensor (exact)."""
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16).to(DEV)


def dev(a, is_bf16):
    return bf16(a) if is_bf16 else f32(a)


def host(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def bits32(t):
    return t.detach().cpu().view(torch.int32).numpy().view(np.uint32)


def bits16(t):
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


def rel_err(got, ref):
    """max |got - ref| / max |ref| (normwise infinity error)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.max(np.abs(ref))
    return float(np.max(np.abs(got - ref)) / (den if den > 0 else 1.0))


def ints(rng, shape, lo=-8, hi=8):
    return rng.integers(lo, hi + 1, size=shape).astype(np.float32)


def bf16_round(a):
    return OP.bf16_to_f32(OP.bf16_rne_bits(np.asarray(a, np.float32)))


# ---------------------------------------------------------------- mixture of experts

def gpu_routes(cfg, flat, Xs, dYs):
    """Per microbatch and layer, the experts the GPU chooses for each token
    ([T, 2] int32), read from a fresh stage's stash after each forward."""
    from paper_2606_11169_amd import libchunk as lc
    from paper_2606_11169_amd.runner import StageRunner
    M = len(Xs)
    r = StageRunner(lc.desc_of_config(cfg), flat, M)
    r.alloc_microbatches(Xs, dYs)
    routes = []
    for mb in range(M):
        r.forward(mb)
        routes.append([r.moe_routing(mb, l) for l in range(cfg.n_layers)])
    for mb in range(M):
        r.backward(mb)
    torch.cuda.synchronize()
    r.close()
    return routes


def check_routing_near_ties(caches, routes, gap_tol=1e-2):
    """The GPU's experts per token against the oracle's own top-2 of its
    float64 softmax (on the oracle's own logits of the same inputs): every
    disagreement must be a near-tie, the two choices' oracle probabilities
    within gap_tol. Returns the number of disagreements."""
    mism = 0
    for l, c in enumerate(caches):
        pi = c["moe"]["pi"]
        own = np.argsort(-pi, axis=1, kind="stable")[:, :2]
        g = np.asarray(routes[l])
        diff = ~np.all(own == g, axis=1)
        for t in np.nonzero(diff)[0]:
            gap = np.max(np.abs(pi[t, g[t]] - pi[t, own[t]]))
            assert gap < gap_tol, f"layer {l} token {t}: GPU {g[t]}, oracle {own[t]}, gap {gap}"
        mism += int(diff.sum())
    return mism


def oracle_order_with_routes(cfg, flat, Xs, dYs, order, routes):
    """The oracle executing an Order (nested pairs in sequence; Bw adds the
    gradient its Bi computed) with the GPU's routing as the routing override
    of every forward, after checking that routing against the oracle's own
    (near-ties only). Returns (Ys, dXs, G)."""
    layers = OS.layer_params(cfg, flat)
    M = len(Xs)
    Ys, dXs, stash, held = [None] * M, [None] * M, {}, {}
    G = np.zeros(synth.param_count(cfg))
    for mb, ps in OO.flatten(order):
        if ps == "F":
            Ys[mb], stash[mb] = OS.stage_forward(cfg, layers, Xs[mb], route_overrides=routes[mb])
            check_routing_near_ties(stash[mb], routes[mb])
        elif ps in ("B", "Bi"):
            dXs[mb], g = OS.stage_backward(cfg, layers, stash.pop(mb), dYs[mb])
            if ps == "B":
                G += g
            else:
                held[mb] = g
        else:
            G += held.pop(mb)
    return Ys, dXs, G
