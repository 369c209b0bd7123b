"""Oracle: forward and backward of one transformer-decoder pipeline stage.

A Chunk in Piper is a compute node whose exec is the forward operator graph
(pass F) or the autograd graph of its backward (pass B) (Piper Section 4.1,
"IR"; the PASS dimension). The paper runs Qwen3/Llama-family decoder stages
(Section 6) but prints no layer formulas, so the layer below is the
standard pre-norm decoder block, written from the textbook definitions:

  n1 = RMSNorm(x; g1)                      rstd = 1/sqrt(mean(x^2) + eps)
  q, k, v = n1 Wq^T, n1 Wk^T, n1 Wv^T      heads use contiguous column blocks
  [Qwen3 variant: q, k <- RMSNorm over each head's hd values, gains qn, kn]
  q, k <- RoPE(q), RoPE(k)                 rotate-half pairs (i, i + hd/2)
  o = softmax(q k^T / sqrt(hd) + causal) v per (batch row, head); with
      grouped-query attention k, v have kv_heads heads and query head h
      uses key/value head h // (heads / kv_heads)
  h = x + o Wo^T
  n2 = RMSNorm(h; g2)
  dense: y = h + (silu(n2 W1^T) * (n2 W3^T)) W2^T
  MoE:   y = h + sum_{k<2} w_k FFN_{e_k}(n2), top-2 of softmax(n2 Wr^T),
         w renormalised over the two selected experts, ties to lower index

Backward is the vector-Jacobian product of L = sum(dY * Y) written out by
hand, pinned by central finite differences in float64.

All arithmetic is float64. Inputs for bf16 workloads are bf16 values
(exactly representable in float64); the oracle never rounds intermediates.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

import synth

from . import order as orders

F64 = np.float64


# ---------------------------------------------------------------------------
# RMSNorm
# ---------------------------------------------------------------------------

def rmsnorm_forward(x, g, eps):
    """n = x * rstd * g, rstd = 1/sqrt(mean_k x_k^2 + eps) over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(ms + eps)
    return x * rstd * g, rstd


def rmsnorm_backward(dn, x, rstd, g):
    """VJP of rmsnorm_forward. Returns (dx, dg).

    With xh = x*rstd: dg = sum_t dn*xh, dxh = dn*g and
    dx = rstd * (dxh - xh * mean_k(dxh_k * xh_k)).
    """
    xh = x * rstd
    dg = np.sum(dn * xh, axis=tuple(range(dn.ndim - 1)))
    dxh = dn * g
    dx = rstd * (dxh - xh * np.mean(dxh * xh, axis=-1, keepdims=True))
    return dx, dg


# ---------------------------------------------------------------------------
# Rotary position embedding (rotate-half convention)
# ---------------------------------------------------------------------------

def rope_tables(seq_len: int, head_dim: int, base: float):
    """cos/sin of p * base^(-2i/hd) for p < S, i < hd/2.

    Angles and their cos/sin are evaluated in float64 and the table is
    rounded to float32 (an fp32 angle p*theta at p ~ 4096 would lose ~2e-4
    rad); the float32-valued table is returned as float64 arrays.
    """
    half = head_dim // 2
    i = np.arange(half, dtype=F64)
    theta = base ** (-2.0 * i / head_dim)
    ang = np.arange(seq_len, dtype=F64)[:, None] * theta[None, :]
    return (np.cos(ang).astype(np.float32).astype(F64),
            np.sin(ang).astype(np.float32).astype(F64))


def rope_apply(t, cos, sin, inverse: bool = False):
    """Rotate pairs (i, i+hd/2) of t [b, S, h, hd] by +angle (or -angle).

    Positions restart at 0 for every sequence (axis 1 is the position).
    The inverse rotation is the transpose, which is also the VJP.
    """
    half = t.shape[-1] // 2
    a, b = t[..., :half], t[..., half:]
    c = cos[None, :, None, :]
    s = sin[None, :, None, :]
    if inverse:
        s = -s
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


# ---------------------------------------------------------------------------
# Causal softmax attention (plain definition, S x S per head)
# ---------------------------------------------------------------------------

def attention_probs(q2, k2):
    """P = softmax(q k^T / sqrt(hd)) with key j masked out for j > query i.

    q2, k2: [S, hd] for one (batch row, head). Returns P [S, S] with exact
    zeros above the diagonal.
    """
    S, hd = q2.shape
    s = (q2 @ k2.T) / np.sqrt(F64(hd))
    mask = np.triu(np.ones((S, S), dtype=bool), k=1)
    s = np.where(mask, -np.inf, s)
    s = s - np.max(s, axis=1, keepdims=True)
    e = np.exp(s)
    return e / np.sum(e, axis=1, keepdims=True)


def attention_forward(q, k, v):
    """o[b,i,h] = sum_{j<=i} P_ij v[b,j,h] for q, k, v of shape [b, S, h, hd]."""
    b, S, h, hd = q.shape
    o = np.empty_like(q)
    for bi in range(b):
        for hi in range(h):
            P = attention_probs(q[bi, :, hi], k[bi, :, hi])
            o[bi, :, hi] = P @ v[bi, :, hi]
    return o


def attention_backward(do, q, k, v):
    """VJP of attention_forward. Returns (dq, dk, dv).

    Per head: dv = P^T do; dP = do v^T; D_i = sum_j P_ij dP_ij;
    dS = P * (dP - D); dq = dS k / sqrt(hd); dk = dS^T q / sqrt(hd).
    """
    b, S, h, hd = q.shape
    dq, dk, dv = np.empty_like(q), np.empty_like(k), np.empty_like(v)
    sc = 1.0 / np.sqrt(F64(hd))
    for bi in range(b):
        for hi in range(h):
            q2, k2, v2, do2 = q[bi, :, hi], k[bi, :, hi], v[bi, :, hi], do[bi, :, hi]
            P = attention_probs(q2, k2)
            dv[bi, :, hi] = P.T @ do2
            dP = do2 @ v2.T
            D = np.sum(P * dP, axis=1, keepdims=True)
            dS = P * (dP - D)
            dq[bi, :, hi] = (dS @ k2) * sc
            dk[bi, :, hi] = (dS.T @ q2) * sc
    return dq, dk, dv


# ---------------------------------------------------------------------------
# SwiGLU FFN
# ---------------------------------------------------------------------------

def sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


def silu(z):
    return z * sigmoid(z)


def swiglu_ffn_forward(n, w1, w3, w2):
    """(silu(n W1^T) * (n W3^T)) W2^T; returns (out, gate, up, act)."""
    gt = n @ w1.T
    u = n @ w3.T
    a = silu(gt) * u
    return a @ w2.T, gt, u, a


def swiglu_ffn_backward(dout, n, gt, u, a, w1, w3, w2):
    """VJP of swiglu_ffn_forward. Returns (dn, dw1, dw3, dw2).

    d silu(z)/dz = s(z) (1 + z (1 - s(z))) with s the logistic sigmoid.
    """
    n2 = n.reshape(-1, n.shape[-1])
    dout2 = dout.reshape(-1, dout.shape[-1])
    gt2 = gt.reshape(-1, gt.shape[-1])
    u2 = u.reshape(-1, u.shape[-1])
    a2 = a.reshape(-1, a.shape[-1])
    da = dout2 @ w2
    dw2 = dout2.T @ a2
    s = sigmoid(gt2)
    dgt = da * u2 * s * (1.0 + gt2 * (1.0 - s))
    du = da * silu(gt2)
    dn = dgt @ w1 + du @ w3
    dw1 = dgt.T @ n2
    dw3 = du.T @ n2
    return dn.reshape(n.shape), dw1, dw3, dw2


# ---------------------------------------------------------------------------
# Top-2 MoE FFN
# ---------------------------------------------------------------------------

def moe_route(n2, wr, top_k: int):
    """Router: logits = n2 Wr^T, pi = softmax over experts, top-k experts by pi
    (ties broken toward the lower expert index), weights renormalised over
    the selected experts. Returns (logits, pi, sel [T,k], w [T,k]).
    """
    T = n2.shape[0]
    logits = n2 @ wr.T
    z = logits - np.max(logits, axis=1, keepdims=True)
    e = np.exp(z)
    pi = e / np.sum(e, axis=1, keepdims=True)
    # a stable sort on -pi keeps equal probabilities in index order
    sel = np.argsort(-pi, axis=1, kind="stable")[:, :top_k]
    ps = pi[np.arange(T)[:, None], sel]
    w = ps / np.sum(ps, axis=1, keepdims=True)
    return logits, pi, sel, w


def moe_dispatch(sel, n_experts: int):
    """Order in which the grouped expert products take their rows: the
    (token, expert) pairs grouped by expert, and within an expert by token
    (the row order in which moe_forward lists each expert's tokens).

    Returns offsets [E + 1] (offsets[e] = pairs routed to experts below e),
    perm [2T] (token of each grouped row) and rowpos [T, k] (grouped row of
    pair (t, sel[t, k])). Plain loops over the definition.
    """
    sel = np.asarray(sel)
    T, K = sel.shape
    perm, offsets = [], [0]
    rowpos = np.full((T, K), -1, dtype=np.int64)
    for e in range(n_experts):
        for t in range(T):
            for k in range(K):
                if sel[t, k] == e:
                    rowpos[t, k] = len(perm)
                    perm.append(t)
        offsets.append(len(perm))
    return np.array(offsets, np.int64), np.array(perm, np.int64), rowpos


def moe_forward(n2, p, cfg, route_override=None):
    """sum_k w_k FFN_{e_k}(n2_t) per token t; n2 is [T, d].

    `route_override` (test only) replaces the selected experts [T, k]; the
    gate weights are still taken from this oracle's own router logits.
    """
    T, d = n2.shape
    logits, pi, sel, w = moe_route(n2, p["wr"], cfg.top_k)
    if route_override is not None:
        sel = np.asarray(route_override, dtype=np.int64).reshape(T, cfg.top_k)
        ps = pi[np.arange(T)[:, None], sel]
        w = ps / np.sum(ps, axis=1, keepdims=True)
    out = np.zeros((T, d), F64)
    per_expert = {}
    for e in range(cfg.n_experts):
        rows, slot = np.nonzero(sel == e)
        if rows.size == 0:
            per_expert[e] = (rows, slot, None)
            continue
        fo, gt, u, a = swiglu_ffn_forward(n2[rows], p[f"e{e}.w1"], p[f"e{e}.w3"],
                                          p[f"e{e}.w2"])
        out[rows] += w[rows, slot][:, None] * fo
        per_expert[e] = (rows, slot, (fo, gt, u, a))
    return out, dict(pi=pi, sel=sel, w=w, per_expert=per_expert)


def moe_backward(dy, n2, p, cfg, mcache):
    """VJP of moe_forward with the routing held fixed.

    For token t and selected slot k: the expert sees dOut = w_k dy_t;
    dw_k = dy_t . FFN_{e_k}(n2_t); the selected logits get
    dl_{e_k} = w_k (dw_k - sum_j w_j dw_j) (unselected logits get 0);
    dWr = dl^T n2 and dn2 += dl Wr. Returns (dn2, grads dict).
    """
    T, d = n2.shape
    E, K = cfg.n_experts, cfg.top_k
    sel, w = mcache["sel"], mcache["w"]
    dn2 = np.zeros((T, d), F64)
    dw = np.zeros((T, K), F64)
    grads = {}
    for e in range(E):
        rows, slot, fwd = mcache["per_expert"][e]
        fe = p[f"e{e}.w1"].shape[0]
        if fwd is None:
            grads[f"e{e}.w1"] = np.zeros((fe, d), F64)
            grads[f"e{e}.w3"] = np.zeros((fe, d), F64)
            grads[f"e{e}.w2"] = np.zeros((d, fe), F64)
            continue
        fo, gt, u, a = fwd
        dw[rows, slot] = np.sum(dy[rows] * fo, axis=1)
        dout = w[rows, slot][:, None] * dy[rows]
        dn, dw1, dw3, dw2 = swiglu_ffn_backward(dout, n2[rows], gt, u, a,
                                                p[f"e{e}.w1"], p[f"e{e}.w3"],
                                                p[f"e{e}.w2"])
        np.add.at(dn2, rows, dn)
        grads[f"e{e}.w1"], grads[f"e{e}.w3"], grads[f"e{e}.w2"] = dw1, dw3, dw2
    dl = np.zeros((T, E), F64)
    inner = np.sum(w * dw, axis=1, keepdims=True)
    dl_sel = w * (dw - inner)
    for kk in range(K):
        dl[np.arange(T), sel[:, kk]] += dl_sel[:, kk]
    grads["wr"] = dl.T @ n2
    dn2 += dl @ p["wr"]
    return dn2, grads


# ---------------------------------------------------------------------------
# One decoder layer
# ---------------------------------------------------------------------------

def repeat_kv(t, groups: int):
    """[b, S, kv, hd] -> [b, S, kv * groups, hd]: head h reads kv head h // groups."""
    return np.repeat(t, groups, axis=2)


def sum_groups(t, groups: int):
    """VJP of repeat_kv: the gradients of a kv head's query heads summed."""
    b, S, h, hd = t.shape
    return t.reshape(b, S, h // groups, groups, hd).sum(axis=3)


def layer_forward(p: Dict[str, np.ndarray], x, cfg, tabs, route_override=None):
    """One pre-norm decoder layer; x is [b, S, d]. Returns (y, cache)."""
    b, S, d = x.shape
    h, hd, hkv = cfg.n_heads, cfg.head_dim, cfg.kv_heads
    cos, sin = tabs
    n1, rstd1 = rmsnorm_forward(x, p["g1"], cfg.rms_eps)
    q = (n1 @ p["wq"].T).reshape(b, S, h, hd)
    k = (n1 @ p["wk"].T).reshape(b, S, hkv, hd)
    v = (n1 @ p["wv"].T).reshape(b, S, hkv, hd)
    cache = dict(x=x, n1=n1, rstd1=rstd1, v=v)
    if cfg.qk_norm:
        qh, rq = rmsnorm_forward(q, p["qn"], cfg.rms_eps)
        kh, rk = rmsnorm_forward(k, p["kn"], cfg.rms_eps)
        cache.update(q=q, k=k, rq=rq, rk=rk)
    else:
        qh, kh = q, k
    qr = rope_apply(qh, cos, sin)
    kr = rope_apply(kh, cos, sin)
    G = h // hkv
    o = attention_forward(qr, repeat_kv(kr, G), repeat_kv(v, G)).reshape(b, S, d)
    hres = x + o @ p["wo"].T
    n2, rstd2 = rmsnorm_forward(hres, p["g2"], cfg.rms_eps)
    cache.update(qr=qr, kr=kr, o=o, h=hres, n2=n2, rstd2=rstd2)
    if cfg.moe:
        ff, mc = moe_forward(n2.reshape(b * S, d), p, cfg, route_override)
        y = hres + ff.reshape(b, S, d)
        cache["moe"] = mc
    else:
        ff, gt, u, a = swiglu_ffn_forward(n2, p["w1"], p["w3"], p["w2"])
        y = hres + ff
        cache.update(gt=gt, u=u, a=a)
    return y, cache


def layer_backward(p, cache, dy, cfg, tabs):
    """VJP of layer_forward. Returns (dx, grads) with grads keyed like p."""
    x = cache["x"]
    b, S, d = x.shape
    h, hd, hkv = cfg.n_heads, cfg.head_dim, cfg.kv_heads
    G = h // hkv
    cos, sin = tabs
    g = {}
    # FFN (the residual passes dy straight to h)
    if cfg.moe:
        dn2, gm = moe_backward(dy.reshape(b * S, d), cache["n2"].reshape(b * S, d),
                               p, cfg, cache["moe"])
        dn2 = dn2.reshape(b, S, d)
        g.update(gm)
    else:
        dn2, g["w1"], g["w3"], g["w2"] = swiglu_ffn_backward(
            dy, cache["n2"], cache["gt"], cache["u"], cache["a"],
            p["w1"], p["w3"], p["w2"])
    dxn2, g["g2"] = rmsnorm_backward(dn2, cache["h"], cache["rstd2"], p["g2"])
    dh = dy + dxn2
    # output projection
    dh2 = dh.reshape(-1, d)
    do = (dh2 @ p["wo"]).reshape(b, S, h, hd)
    g["wo"] = dh2.T @ cache["o"].reshape(-1, d)
    # attention over the repeated key/value heads, then undo the rotation
    dqr, dkr, dv = attention_backward(do, cache["qr"], repeat_kv(cache["kr"], G),
                                      repeat_kv(cache["v"], G))
    dkr, dv = sum_groups(dkr, G), sum_groups(dv, G)
    dq = rope_apply(dqr, cos, sin, inverse=True)
    dk = rope_apply(dkr, cos, sin, inverse=True)
    if cfg.qk_norm:
        dq, g["qn"] = rmsnorm_backward(dq, cache["q"], cache["rq"], p["qn"])
        dk, g["kn"] = rmsnorm_backward(dk, cache["k"], cache["rk"], p["kn"])
    dq, dk, dv = dq.reshape(-1, d), dk.reshape(-1, hkv * hd), dv.reshape(-1, hkv * hd)
    n1 = cache["n1"].reshape(-1, d)
    dn1 = (dq @ p["wq"] + dk @ p["wk"] + dv @ p["wv"]).reshape(b, S, d)
    g["wq"], g["wk"], g["wv"] = dq.T @ n1, dk.T @ n1, dv.T @ n1
    dxn1, g["g1"] = rmsnorm_backward(dn1, x, cache["rstd1"], p["g1"])
    return dh + dxn1, g


# ---------------------------------------------------------------------------
# Stage = L layers; Chunk F and Chunk B
# ---------------------------------------------------------------------------

def layer_params(cfg, flat: np.ndarray) -> List[Dict[str, np.ndarray]]:
    """Per-layer dicts of float64 views from the flat bucket."""
    named = synth.unflatten(cfg, np.asarray(flat, dtype=F64))
    layers = []
    for l in range(cfg.n_layers):
        pre = f"L{l}."
        layers.append({k[len(pre):]: v for k, v in named.items() if k.startswith(pre)})
    return layers


def stage_forward(cfg, layers, X, route_overrides=None):
    """Chunk F: Y = layer_{L-1}(...layer_0(X)). Returns (Y, caches)."""
    tabs = rope_tables(X.shape[1], cfg.head_dim, cfg.rope_base)
    x = np.asarray(X, dtype=F64)
    caches = []
    for l, p in enumerate(layers):
        ro = None if route_overrides is None else route_overrides[l]
        x, c = layer_forward(p, x, cfg, tabs, ro)
        caches.append(c)
    return x, caches


def stage_backward(cfg, layers, caches, dY):
    """Chunk B: dX and this microbatch's parameter gradients (flat, float64)."""
    S = caches[0]["x"].shape[1]
    tabs = rope_tables(S, cfg.head_dim, cfg.rope_base)
    dy = np.asarray(dY, dtype=F64)
    named = {}
    for l in reversed(range(cfg.n_layers)):
        dy, g = layer_backward(layers[l], caches[l], dy, cfg, tabs)
        for k, v in g.items():
            named[f"L{l}.{k}"] = v
    return dy, synth.flatten(cfg, named, dtype=F64)


def stage_loss(cfg, layers, X, dY, route_overrides=None) -> float:
    """L = sum(dY * Y): the scalar whose gradient Chunk B computes."""
    Y, _ = stage_forward(cfg, layers, X, route_overrides)
    return float(np.sum(np.asarray(dY, F64) * Y))


def run_order(cfg, flat_params, Xs: Sequence[np.ndarray], dYs: Sequence[np.ndarray],
              order: Sequence[Tuple[int, str]]):
    """Execute an Order of (mb, 'F'|'B'|'Bi'|'Bw') entries (Piper Section 4.1,
    Split and Order). F(mb) keeps its activations until B(mb) or Bi(mb).
    B(mb) adds the microbatch's gradient into the flat accumulator G
    (initially +0, no 1/M scaling); Bi(mb) produces dX(mb) and Bw(mb) adds the
    microbatch's gradient into G, so G receives the microbatches' gradients in
    the Order's sequence of B and Bw entries.

    Returns (Ys, dXs, G) with G in float64.
    """
    layers = layer_params(cfg, flat_params)
    M = len(Xs)
    Ys: List[Optional[np.ndarray]] = [None] * M
    dXs: List[Optional[np.ndarray]] = [None] * M
    stash = {}
    held = {}  # microbatch -> gradient computed by Bi, added by Bw
    G = np.zeros(synth.param_count(cfg), F64)
    for mb, ps in orders.flatten(order):
        if ps == "F":
            Ys[mb], stash[mb] = stage_forward(cfg, layers, Xs[mb])
        elif ps == "B":
            dXs[mb], gmb = stage_backward(cfg, layers, stash.pop(mb), dYs[mb])
            G += gmb
        elif ps == "Bi":
            dXs[mb], held[mb] = stage_backward(cfg, layers, stash.pop(mb), dYs[mb])
        else:
            G += held.pop(mb)
    return Ys, dXs, G


def prefix_forward(cfg, flat_params, X, n_tokens: int):
    """Y[:, :n] of Chunk F using only X[:, :n] (causality: positions < n never
    see later positions). Used to check full-size outputs on a prefix."""
    layers = layer_params(cfg, flat_params)
    Y, _ = stage_forward(cfg, layers, np.asarray(X)[:, :n_tokens])
    return Y
