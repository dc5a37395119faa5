"""fp64 CPU oracle of ORBIT's ViT forward and backward pass (TEST INFRASTRUCTURE).

This module is test infrastructure only. Only ``tests/``, ``__graft_entry__.smoke``
and the ``cpu_baseline`` leg of ``bench.py`` may import it; the product path
(the HIP library and its Python binding) never does, and shares no code,
constant or helper with it.

What it computes, and where the paper states it (arXiv 2404.14712):

* Sec. II (ClimaX architecture, Fig. 1): each input channel (climate variable)
  is tokenised into image patches independently; the per-variable patch
  embeddings are aggregated across variables by cross-attention; the aggregated
  tokens pass through transformer blocks, each a self-attention sub-layer and a
  feed-forward sub-layer; a final projection maps features back to image space.
* Sec. III-A: the self-attention core is softmax(Q K^T) V and the feed-forward
  core is GeLU(x A) B; Eq. (2) states that x A B equals the sum over column
  shards A_{*,k} and row shards B_{k,*} of x A_{*,k} B_{k,*}, and Eq. (3) the
  same for the gradient.
* Sec. III-B: an extra LayerNorm on the queries and keys before the scaled dot
  product (QK-LayerNorm).
* Sec. IV: 128x256 grids per variable, 48 or 91 variables; Sec. III-B: BF16
  mixed precision.

Every function is the plain definition in float64 with NumPy: a matmul is the
only library primitive used (plus ``scipy.special.erf`` for the Gaussian CDF).
Attention is materialised, the aggregation runs its full key/value projections
(no algebraic folding), and every backward is the hand-derived adjoint of the
forward written next to it. Each function states the reading it takes of
any point the paper leaves open.

Pins (tests/test_oracle_*.py): central finite differences for every backward,
a float64 PyTorch-CPU autograd cross-check (independent library code), softmax
normalisation, identical-key attention = mean of values, LayerNorm moments and
backward orthogonality, GELU closed forms and tabulated normal-CDF values,
key-bias shift invariance, identity-block and single-variable special cases,
scalar-loop brute force, and the Eq. (2)/(3) shard sums.
"""
from __future__ import annotations

import math
from typing import Dict, Tuple

import numpy as np
from scipy.special import erf

F64 = np.float64


def _f(a) -> np.ndarray:
    return np.asarray(a, dtype=F64)


def _keep(store):
    """`store` models the storage of an intermediate between two steps. The
    oracle proper passes None (exact: nothing is rounded); tests pass a
    rounding function to measure how much storing intermediates at a reduced
    precision can move each result (the precision floor of the comparison)."""
    return store if store is not None else (lambda a: a)


# ---------------------------------------------------------------------------
# Patch tokenisation (Sec. II: independent tokenisation of every variable)
# ---------------------------------------------------------------------------

def patchify(img: np.ndarray, p: int) -> np.ndarray:
    """img[B, V, Hg, Wg] -> P[B, V, L, p*p].

    Reading (paper silent on ordering): patch l = ph*(Wg/p) + pw in row-major
    order over the patch grid; pixel c = i*p + j inside a patch.
    """
    B, V, Hg, Wg = img.shape
    nh, nw = Hg // p, Wg // p
    x = _f(img).reshape(B, V, nh, p, nw, p)          # [B,V,ph,i,pw,j]
    x = x.transpose(0, 1, 2, 4, 3, 5)                # [B,V,ph,pw,i,j]
    return x.reshape(B, V, nh * nw, p * p)


def patch_embed_fwd(img, w_pe, b_pe, ve, p: int, store=None) -> np.ndarray:
    """tok[b, l, v, :] = P[b, v, l, :] @ w_pe[v] + b_pe[v] + ve[v]   (Sec. II).

    One linear map p*p -> d per variable (equal to a stride-p convolution with
    a p x p kernel), plus a learned per-variable embedding ve[v].
    Output layout tok[B, L, V, d] keeps the V x d slab of one patch contiguous.
    """
    P = patchify(img, p)                              # [B,V,L,pp]
    B, V, L, _ = P.shape
    d = w_pe.shape[2]
    tok = np.empty((B, L, V, d), F64)
    for v in range(V):
        e = P[:, v] @ _f(w_pe[v]) + _f(b_pe[v])      # [B,L,d]
        if ve is not None:
            e = e + _f(ve[v])
        tok[:, :, v, :] = e
    return _keep(store)(tok)


def patch_embed_bwd(img, dtok, p: int) -> Dict[str, np.ndarray]:
    """Adjoint of patch_embed_fwd with respect to its parameters."""
    P = patchify(img, p)
    dtok = _f(dtok)
    B, L, V, d = dtok.shape
    dw = np.empty((V, p * p, d), F64)
    db = np.empty((V, d), F64)
    for v in range(V):
        g = dtok[:, :, v, :].reshape(B * L, d)
        dw[v] = P[:, v].reshape(B * L, p * p).T @ g
        db[v] = g.sum(axis=0)
    return {"w_pe": dw, "b_pe": db, "ve": db.copy()}


# ---------------------------------------------------------------------------
# LayerNorm (pre-LN blocks; QK-LayerNorm of Sec. III-B)
# ---------------------------------------------------------------------------

def layer_norm_fwd(x, g, b, eps: float):
    """y = g * (x - mean) / sqrt(var + eps) + b over the last axis.

    Reading: biased variance (divide by the row length), affine gain/shift.
    Returns y and the cache (xhat, rstd) used by the backward.
    """
    x = _f(x)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (x - mu) * rstd
    return xhat * _f(g) + _f(b), (xhat, rstd)


def layer_norm_bwd(dy, cache, g):
    """Adjoint of layer_norm_fwd: dx, dg, db (dg, db summed over all rows)."""
    xhat, rstd = cache
    dy = _f(dy)
    gh = dy * _f(g)
    n = xhat.shape[-1]
    dx = rstd * (gh - gh.sum(axis=-1, keepdims=True) / n
                 - xhat * (gh * xhat).sum(axis=-1, keepdims=True) / n)
    red = tuple(range(dy.ndim - 1))
    return dx, (dy * xhat).sum(axis=red), dy.sum(axis=red)


# ---------------------------------------------------------------------------
# GELU (Sec. III-A feed-forward core GeLU(xA)B)
# ---------------------------------------------------------------------------

def gelu(u):
    """GELU(u) = u * Phi(u), Phi the standard normal CDF (exact erf form)."""
    u = _f(u)
    return 0.5 * u * (1.0 + erf(u / math.sqrt(2.0)))


def gelu_grad(u):
    """d GELU / du = Phi(u) + u * phi(u)."""
    u = _f(u)
    return 0.5 * (1.0 + erf(u / math.sqrt(2.0))) + u * np.exp(-0.5 * u * u) / math.sqrt(2.0 * math.pi)


# ---------------------------------------------------------------------------
# Softmax attention (Sec. III-A: softmax(Q K^T) V with 1/sqrt(d_h) scaling)
# ---------------------------------------------------------------------------

def softmax(s, axis: int = -1):
    s = _f(s)
    e = np.exp(s - s.max(axis=axis, keepdims=True))
    return e / e.sum(axis=axis, keepdims=True)


def attention_fwd(q, k, v):
    """q, k, v [..., n, d_h] -> O = softmax(q k^T / sqrt(d_h)) v, and P."""
    q, k, v = _f(q), _f(k), _f(v)
    dh = q.shape[-1]
    S = q @ np.swapaxes(k, -1, -2) / math.sqrt(dh)
    P = softmax(S, axis=-1)
    return P @ v, P


def attention_bwd(dO, q, k, v, P):
    """Adjoint of attention_fwd: dq, dk, dv."""
    dO, q, k, v = _f(dO), _f(q), _f(k), _f(v)
    dh = q.shape[-1]
    dv = np.swapaxes(P, -1, -2) @ dO
    dP = dO @ np.swapaxes(v, -1, -2)
    dS = P * (dP - (dP * P).sum(axis=-1, keepdims=True))
    dq = dS @ k / math.sqrt(dh)
    dk = np.swapaxes(dS, -1, -2) @ q / math.sqrt(dh)
    return dq, dk, dv


# ---------------------------------------------------------------------------
# Transformer block (Sec. II, Sec. III-A, Sec. III-B)
# ---------------------------------------------------------------------------

def _heads(t, H):
    """[B, L, H*dh] -> [B, H, L, dh]"""
    B, L, A = t.shape
    return t.reshape(B, L, H, A // H).transpose(0, 2, 1, 3)


def _unheads(t):
    """[B, H, L, dh] -> [B, L, H*dh]"""
    B, H, L, dh = t.shape
    return t.transpose(0, 2, 1, 3).reshape(B, L, H * dh)


def block_fwd(x, prm: Dict[str, np.ndarray], heads: int, qk_norm: int = 1, eps: float = 1e-5, store=None):
    """One pre-LN transformer block; x[B, L, d] -> y[B, L, d].

    h1 = LN1(x); [q|k|v] = h1 W_qkv + b_qkv (columns q, k, v, each head-major);
    QK-LayerNorm over each head's d_h features when qk_norm (Sec. III-B; the
    gain/shift of length d_h are shared by all heads);
    o = softmax(q k^T / sqrt(d_h)) v per head (no mask);
    x1 = x + o W_proj + b_proj;  u = LN2(x1) W_fc1 + b_fc1;
    y = x1 + GELU(u) W_fc2 + b_fc2.

    With A = heads*d_h != d and F the local MLP width this is one GPU's share
    under Eq. (2): W_qkv / W_fc1 are column shards, W_proj / W_fc2 row shards,
    and the row-shard outputs are partial sums added to the residual unreduced.
    """
    S = _keep(store)
    x = _f(x)
    p = {k_: _f(v_) for k_, v_ in prm.items()}
    A = p["w_proj"].shape[0]
    h1, c_ln1 = layer_norm_fwd(x, p["ln1_g"], p["ln1_b"], eps)
    h1 = S(h1)
    qkv = S(h1 @ p["w_qkv"] + p["b_qkv"])
    q_raw, k_raw, v_ = qkv[..., :A], qkv[..., A:2 * A], qkv[..., 2 * A:]
    q, k, v = _heads(q_raw, heads), _heads(k_raw, heads), _heads(v_, heads)
    c_qn = c_kn = None
    if qk_norm:
        q, c_qn = layer_norm_fwd(q, p["qn_g"], p["qn_b"], eps)
        k, c_kn = layer_norm_fwd(k, p["kn_g"], p["kn_b"], eps)
        q, k = S(q), S(k)
    O, P = attention_fwd(q, k, v)
    o = S(_unheads(O))
    x1 = S(x + o @ p["w_proj"] + p["b_proj"])
    h2, c_ln2 = layer_norm_fwd(x1, p["ln2_g"], p["ln2_b"], eps)
    h2 = S(h2)
    u_ = h2 @ p["w_fc1"] + p["b_fc1"]
    u = S(u_)
    g = S(gelu(u_))
    y = S(x1 + g @ p["w_fc2"] + p["b_fc2"])
    cache = dict(x=x, h1=h1, c_ln1=c_ln1, q=q, k=k, v=v, P=P, o=o, c_qn=c_qn, c_kn=c_kn,
                 x1=x1, h2=h2, c_ln2=c_ln2, u=u, g=g, heads=heads, qk_norm=qk_norm, store=store)
    return y, cache


def block_bwd(dy, cache, prm: Dict[str, np.ndarray]):
    """Adjoint of block_fwd: returns dx and the gradient of every parameter."""
    p = {k_: _f(v_) for k_, v_ in prm.items()}
    dy = _f(dy)
    c = cache
    S = _keep(c.get("store"))
    B, L, d = dy.shape
    T = B * L
    gr: Dict[str, np.ndarray] = {}
    # feed-forward sub-layer: y = x1 + GELU(u) W_fc2 + b_fc2
    gr["w_fc2"] = c["g"].reshape(T, -1).T @ dy.reshape(T, d)
    gr["b_fc2"] = dy.reshape(T, d).sum(0)
    du = S((dy @ p["w_fc2"].T) * gelu_grad(c["u"]))
    gr["w_fc1"] = c["h2"].reshape(T, d).T @ du.reshape(T, -1)
    gr["b_fc1"] = du.reshape(T, -1).sum(0)
    dh2 = S(du @ p["w_fc1"].T)
    dx1_ln, gr["ln2_g"], gr["ln2_b"] = layer_norm_bwd(dh2, c["c_ln2"], p["ln2_g"])
    dx1 = S(dy + dx1_ln)
    # attention sub-layer: x1 = x + o W_proj + b_proj
    A = p["w_proj"].shape[0]
    gr["w_proj"] = c["o"].reshape(T, A).T @ dx1.reshape(T, d)
    gr["b_proj"] = dx1.reshape(T, d).sum(0)
    do = S(dx1 @ p["w_proj"].T)
    dq, dk, dv = attention_bwd(_heads(do, c["heads"]), c["q"], c["k"], c["v"], c["P"])
    dq, dk, dv = S(dq), S(dk), S(dv)
    if c["qk_norm"]:
        dq, gr["qn_g"], gr["qn_b"] = layer_norm_bwd(dq, c["c_qn"], p["qn_g"])
        dk, gr["kn_g"], gr["kn_b"] = layer_norm_bwd(dk, c["c_kn"], p["kn_g"])
    else:
        for n_ in ("qn_g", "qn_b", "kn_g", "kn_b"):
            gr[n_] = np.zeros_like(p[n_])
    dqkv = S(np.concatenate([_unheads(dq), _unheads(dk), _unheads(dv)], axis=-1))
    gr["w_qkv"] = c["h1"].reshape(T, d).T @ dqkv.reshape(T, 3 * A)
    gr["b_qkv"] = dqkv.reshape(T, 3 * A).sum(0)
    dh1 = S(dqkv @ p["w_qkv"].T)
    dx_ln, gr["ln1_g"], gr["ln1_b"] = layer_norm_bwd(dh1, c["c_ln1"], p["ln1_g"])
    return S(dx1 + dx_ln), gr


# ---------------------------------------------------------------------------
# Cross-attention variable aggregation (Sec. II)
# ---------------------------------------------------------------------------

def agg_fwd(tok, prm: Dict[str, np.ndarray], heads: int, store=None):
    """tok[B, L, V, d] -> z[B, L, d]: one learned query attends over the V
    variable tokens of each patch (multi-head attention semantics).

    q = q0 W_q + b_q;  K = X W_k + b_k;  Vv = X W_v + b_v   (X = tok[b, l]);
    a_h = softmax_v(q_h . K_{v,h} / sqrt(d_h));  zh_h = sum_v a_{h,v} Vv_{v,h};
    z = concat_h(zh) W_o + b_o + pos[l].
    The key/value projections are computed in full (no folding).
    """
    X = _f(tok)
    p = {k_: _f(v_) for k_, v_ in prm.items()}
    B, L, V, d = X.shape
    A = p["w_q"].shape[1]
    dh = A // heads
    q = p["q0"] @ p["w_q"] + p["b_q"]                      # [A]
    K = X @ p["w_k"] + p["b_k"]                            # [B,L,V,A]
    Vv = X @ p["w_v"] + p["b_v"]
    qh = q.reshape(heads, dh)
    Kh = K.reshape(B, L, V, heads, dh)
    Vh = Vv.reshape(B, L, V, heads, dh)
    s = np.einsum("hc,blvhc->blhv", qh, Kh) / math.sqrt(dh)
    a = softmax(s, axis=-1)                                 # [B,L,H,V]
    S = _keep(store)
    zh = S(np.einsum("blhv,blvhc->blhc", a, Vh).reshape(B, L, A))
    z = zh @ p["w_o"] + p["b_o"]
    if "pos" in p and p["pos"] is not None:
        z = z + p["pos"][None, :, :]
    cache = dict(X=X, q=q, Kh=Kh, Vh=Vh, a=a, zh=zh, heads=heads, store=store)
    return S(z), cache


def agg_bwd(dz, cache, prm: Dict[str, np.ndarray]):
    """Adjoint of agg_fwd: dtok and every parameter gradient."""
    p = {k_: _f(v_) for k_, v_ in prm.items()}
    dz = _f(dz)
    c = cache
    X, a, Kh, Vh = c["X"], c["a"], c["Kh"], c["Vh"]
    B, L, V, d = X.shape
    H = c["heads"]
    A = p["w_q"].shape[1]
    dh = A // H
    T = B * L
    gr: Dict[str, np.ndarray] = {}
    gr["pos"] = dz.sum(axis=0)
    gr["b_o"] = dz.reshape(T, d).sum(0)
    gr["w_o"] = c["zh"].reshape(T, A).T @ dz.reshape(T, d)
    S = _keep(c.get("store"))
    dzh = S(dz @ p["w_o"].T).reshape(B, L, H, dh)
    da = np.einsum("blhc,blvhc->blhv", dzh, Vh)
    dVh = np.einsum("blhv,blhc->blvhc", a, dzh)
    ds = a * (da - (da * a).sum(axis=-1, keepdims=True)) / math.sqrt(dh)
    qh = c["q"].reshape(H, dh)
    dKh = np.einsum("blhv,hc->blvhc", ds, qh)
    dqh = np.einsum("blhv,blvhc->hc", ds, Kh)
    dK = dKh.reshape(B, L, V, A)
    dVv = dVh.reshape(B, L, V, A)
    XT = X.reshape(T * V, d)
    gr["w_k"] = XT.T @ dK.reshape(T * V, A)
    gr["b_k"] = dK.reshape(T * V, A).sum(0)
    gr["w_v"] = XT.T @ dVv.reshape(T * V, A)
    gr["b_v"] = dVv.reshape(T * V, A).sum(0)
    dq = dqh.reshape(A)
    gr["w_q"] = np.outer(p["q0"], dq)
    gr["b_q"] = dq
    gr["q0"] = p["w_q"] @ dq
    dtok = S(dK @ p["w_k"].T + dVv @ p["w_v"].T)
    return dtok, gr


# ---------------------------------------------------------------------------
# Prediction head (Sec. II: projection from feature space to image space) and loss
# ---------------------------------------------------------------------------

def head_fwd(x, prm: Dict[str, np.ndarray], final_ln: int = 1, eps: float = 1e-5, store=None):
    """pred[B, L, V*p*p] = LN_f(x) followed by the prediction head (Sec. II:
    projection from feature space back to image space).

    Reading: the head of the ClimaX architecture the paper builds on, i.e.
    `hidden` layers h <- GELU(h W_k + b_k) of width d (weights w_hid[k] [d, d],
    b_hid[k] [d]; none when prm has no w_hid or it has zero layers), then one
    linear map d -> V*p*p (w_h, b_h). LN_f is skipped when final_ln == 0. The
    output row of a token holds its V patches, pixel index v*p*p + i*p + j.
    """
    x = _f(x)
    p = {k_: (None if v_ is None else _f(v_)) for k_, v_ in prm.items()}
    S = _keep(store)
    if final_ln:
        hf, c_ln = layer_norm_fwd(x, p["lnf_g"], p["lnf_b"], eps)
        hf = S(hf)
    else:
        hf, c_ln = x, None
    W, bias = p.get("w_hid"), p.get("b_hid")
    nh = 0 if W is None else W.shape[0]
    acts, pres = [hf], []
    h = hf
    for k in range(nh):
        u = h @ W[k] + bias[k]
        pres.append(S(u))
        h = S(gelu(u))
        acts.append(h)
    return h @ p["w_h"] + p["b_h"], dict(hf=hf, c_ln=c_ln, final_ln=final_ln, store=store, acts=acts, pres=pres)


def head_bwd(dpred, cache, prm: Dict[str, np.ndarray]):
    p = {k_: (None if v_ is None else _f(v_)) for k_, v_ in prm.items()}
    dpred = _f(dpred)
    B, L, n = dpred.shape
    acts, pres = cache["acts"], cache["pres"]
    d = cache["hf"].shape[-1]
    T = B * L
    S = _keep(cache.get("store"))
    gr = {"b_h": dpred.reshape(T, n).sum(0)}
    dpred = S(dpred)
    gr["w_h"] = acts[-1].reshape(T, -1).T @ dpred.reshape(T, n)
    dh = S(dpred @ p["w_h"].T)
    nh = len(pres)
    if nh:
        gr["w_hid"] = np.empty_like(p["w_hid"])
        gr["b_hid"] = np.empty_like(p["b_hid"])
    for k in range(nh - 1, -1, -1):
        du = S(dh * gelu_grad(pres[k]))
        gr["w_hid"][k] = acts[k].reshape(T, d).T @ du.reshape(T, d)
        gr["b_hid"][k] = du.reshape(T, d).sum(0)
        dh = S(du @ p["w_hid"][k].T)
    if cache["final_ln"]:
        dx, gr["lnf_g"], gr["lnf_b"] = layer_norm_bwd(dh, cache["c_ln"], p["lnf_g"])
        dx = S(dx)
    else:
        dx = dh
        gr["lnf_g"] = np.zeros(d)
        gr["lnf_b"] = np.zeros(d)
    return dx, gr


def mse(pred, tgt, scale: float = 1.0):
    """Mean squared error over every element and its gradient (times scale).
    Reading: plain mean; the paper's latitude weighting (Sec. IV) is not applied."""
    r = _f(pred) - _f(tgt)
    n = r.size
    return float((r * r).sum() / n), 2.0 * r / n * scale


def lat_weights(H: int) -> np.ndarray:
    """Latitude weights of the rows of an H-row equiangular grid (Sec. IV: the
    training loss is the latitude-weighted MSE; grid cells shrink towards the
    poles, so a row is weighted by its cell area, proportional to cos(latitude)).

    Reading: rows are equally spaced in latitude with cell centres at
    -90 + (y + 1/2) * 180 / H degrees, and the weights are normalised to mean 1.
    """
    lat = np.deg2rad(-90.0 + (np.arange(H, dtype=F64) + 0.5) * 180.0 / H)
    c = np.cos(lat)
    return c / c.mean()


def unpatchify(t, Wp: int, p: int) -> np.ndarray:
    """Token layout [B, L, V*p*p] (patch l = ph*Wp + pw, pixel v*p*p + i*p + j)
    -> image layout [B, V, (L/Wp)*p, Wp*p]; the inverse of patchify."""
    t = _f(t)
    B, L, n = t.shape
    V = n // (p * p)
    Hp = L // Wp
    x = t.reshape(B, Hp, Wp, V, p, p)                # [B,ph,pw,v,i,j]
    x = x.transpose(0, 3, 1, 4, 2, 5)                # [B,v,ph,i,pw,j]
    return x.reshape(B, V, Hp * p, Wp * p)


def wmse(pred, tgt, Wp: int, p: int, scale: float = 1.0):
    """Latitude-weighted mean squared error (Sec. IV) of predictions and targets
    in token layout [B, L, V*p*p], and its gradient (times scale) in that layout:
    loss = mean over (b, v, y, x) of w[y] (pred - tgt)^2, w = lat_weights(H)."""
    r = unpatchify(pred, Wp, p) - unpatchify(tgt, Wp, p)     # [B,V,H,W]
    w = lat_weights(r.shape[2])[None, None, :, None]
    n = r.size
    g = 2.0 * w * r / n * scale                               # [B,V,H,W]
    B, V = g.shape[:2]
    g_tok = patchify(g, p).transpose(0, 2, 1, 3)              # [B,L,V,p*p]
    return float((w * r * r).sum() / n), g_tok.reshape(B, -1, V * p * p)


# ---------------------------------------------------------------------------
# Whole model (Sec. II, Fig. 1): embed -> aggregate -> blocks -> head -> loss
# ---------------------------------------------------------------------------

def model_fwd_bwd(img, tgt, emb, agg, blocks, head, *, p: int, agg_heads: int, heads: int,
                  qk_norm: int = 1, eps: float = 1e-5, final_ln: int = 1, store=None, loss: str = "mse"):
    """Forward and backward of the full ClimaX-style model for one batch.

    Returns (loss, pred, grads) with grads = {"embed": .., "agg": ..,
    "blocks": [..], "head": ..}. `store` as in block_fwd (None: exact).
    loss: "mse" (plain mean) or "wmse" (latitude-weighted, Sec. IV).
    """
    tok = patch_embed_fwd(img, emb["w_pe"], emb["b_pe"], emb.get("ve"), p, store)
    x, c_agg = agg_fwd(tok, agg, agg_heads, store)
    caches = []
    for prm in blocks:
        x, c = block_fwd(x, prm, heads, qk_norm, eps, store)
        caches.append(c)
    pred, c_head = head_fwd(x, head, final_ln, eps, store)
    if loss == "wmse":
        loss, dpred = wmse(pred, tgt, _f(img).shape[3] // p, p)
    else:
        loss, dpred = mse(pred, tgt)
    dx, g_head = head_bwd(dpred, c_head, head)
    g_blocks = [None] * len(blocks)
    for i in range(len(blocks) - 1, -1, -1):
        dx, g_blocks[i] = block_bwd(dx, caches[i], blocks[i])
    dtok, g_agg = agg_bwd(dx, c_agg, agg)
    g_emb = patch_embed_bwd(img, dtok, p)
    return loss, pred, {"embed": g_emb, "agg": g_agg, "blocks": g_blocks, "head": g_head}


# ---------------------------------------------------------------------------
# Eq. (2) / Eq. (3): column/row shards of one sub-layer
# ---------------------------------------------------------------------------

def shard_block_params(prm: Dict[str, np.ndarray], heads: int, F: int, K: int, k: int,
                       keep_bias: bool) -> Dict[str, np.ndarray]:
    """Shard k of K of a block under Eq. (2): W_qkv columns of whole heads and
    W_fc1 columns (column shards A_{*,k}); the matching W_proj / W_fc2 rows
    (row shards B_{k,*}). Row-shard biases b_proj, b_fc2 are kept on one shard
    only (keep_bias) so that the sum over shards counts them once."""
    A = prm["w_proj"].shape[0]
    dh = A // heads
    hk = heads // K
    cols = np.arange(k * hk * dh, (k + 1) * hk * dh)
    qkv_cols = np.concatenate([cols, A + cols, 2 * A + cols])
    fk = F // K
    fcols = np.arange(k * fk, (k + 1) * fk)
    out = dict(prm)
    out["w_qkv"] = prm["w_qkv"][:, qkv_cols]
    out["b_qkv"] = prm["b_qkv"][qkv_cols]
    out["w_proj"] = prm["w_proj"][cols, :]
    out["w_fc1"] = prm["w_fc1"][:, fcols]
    out["b_fc1"] = prm["b_fc1"][fcols]
    out["w_fc2"] = prm["w_fc2"][fcols, :]
    if not keep_bias:
        out["b_proj"] = np.zeros_like(prm["b_proj"])
        out["b_fc2"] = np.zeros_like(prm["b_fc2"])
    return out
