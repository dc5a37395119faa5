"""Pins of the fp64 oracle against facts the paper and mathematics fix.

Each test is independent of the HIP path. A plausible mistake in the oracle (a
dropped term, a wrong sign or index, a transposed operand) fails at least one:
finite differences catch any backward error, the closed forms / brute force /
golden fixtures catch forward errors, and the library cross-check in
test_oracle_torch.py catches semantic misreadings.
"""
import math
import os

import numpy as np
import pytest

import oracle as O

GOLD = os.path.join(os.path.dirname(__file__), "golden")
R = np.random.default_rng(12345)


def _rand(*shape, s=1.0):
    return R.standard_normal(shape) * s


def _block_prm(d, A, F, dh, s=0.3):
    p = {k: _rand(*shp, s=s) for k, shp in {
        "ln1_g": (d,), "ln1_b": (d,), "w_qkv": (d, 3 * A), "b_qkv": (3 * A,),
        "qn_g": (dh,), "qn_b": (dh,), "kn_g": (dh,), "kn_b": (dh,),
        "w_proj": (A, d), "b_proj": (d,), "ln2_g": (d,), "ln2_b": (d,),
        "w_fc1": (d, F), "b_fc1": (F,), "w_fc2": (F, d), "b_fc2": (d,)}.items()}
    for g in ("ln1_g", "ln2_g", "qn_g", "kn_g"):
        p[g] = p[g] + 1.0
    return p


def _agg_prm(d, A, L, s=0.4):
    return {"q0": _rand(d, s=s), "w_q": _rand(d, A, s=s), "b_q": _rand(A, s=s),
            "w_k": _rand(d, A, s=s), "b_k": _rand(A, s=s), "w_v": _rand(d, A, s=s),
            "b_v": _rand(A, s=s), "w_o": _rand(A, d, s=s), "b_o": _rand(d, s=s),
            "pos": _rand(L, d, s=s)}


def _head_prm(d, n, s=0.3):
    return {"lnf_g": 1 + _rand(d, s=s), "lnf_b": _rand(d, s=s), "w_h": _rand(d, n, s=s),
            "b_h": _rand(n, s=s)}


# ---------------------------------------------------------------------------
# P1: central finite differences for every backward
# ---------------------------------------------------------------------------

def _fd_check(f, tensors, grads, h=1e-6, tol=1e-6, full_max=48):
    """f(): scalar; tensors: dict name -> array (perturbed in place);
    grads: dict name -> analytic gradient. Checks every entry of small
    tensors and one random direction for each larger tensor."""
    for name, t in tensors.items():
        g = grads[name]
        assert g.shape == t.shape, name
        if t.size <= full_max:
            idx = list(np.ndindex(t.shape))
        else:
            idx = None
        if idx is not None:
            for ix in idx:
                old = t[ix]
                t[ix] = old + h
                fp = f()
                t[ix] = old - h
                fm = f()
                t[ix] = old
                num = (fp - fm) / (2 * h)
                assert abs(num - g[ix]) <= tol * max(1.0, abs(num)), (name, ix, num, g[ix])
        else:
            dirn = R.standard_normal(t.shape)
            old = t.copy()
            t[...] = old + h * dirn
            fp = f()
            t[...] = old - h * dirn
            fm = f()
            t[...] = old
            num = (fp - fm) / (2 * h)
            ana = float((g * dirn).sum())
            assert abs(num - ana) <= tol * max(1.0, abs(num)), (name, num, ana)


@pytest.mark.parametrize("qk_norm", [1, 0])
@pytest.mark.parametrize("shard", [False, True])
def test_fd_block(qk_norm, shard):
    B, L, d, H = 2, 5, 16, 2
    dh = 4 if shard else 8      # shard: A = H*dh = 8 != d (one GPU's column shard)
    A = H * dh
    F = 24
    x = _rand(B, L, d)
    prm = _block_prm(d, A, F, dh)
    Rw = _rand(B, L, d)

    def f():
        y, _ = O.block_fwd(x, prm, H, qk_norm)
        return float((y * Rw).sum())

    y, cache = O.block_fwd(x, prm, H, qk_norm)
    dx, gr = O.block_bwd(Rw, cache, prm)
    tensors = dict(prm)
    tensors["x"] = x
    grads = dict(gr)
    grads["x"] = dx
    _fd_check(f, tensors, grads)


def test_fd_agg():
    B, L, V, d, H = 2, 3, 4, 12, 3
    A = 12
    tok = _rand(B, L, V, d)
    prm = _agg_prm(d, A, L)
    Rw = _rand(B, L, d)

    def f():
        z, _ = O.agg_fwd(tok, prm, H)
        return float((z * Rw).sum())

    z, cache = O.agg_fwd(tok, prm, H)
    dtok, gr = O.agg_bwd(Rw, cache, prm)
    tensors = dict(prm)
    tensors["tok"] = tok
    grads = dict(gr)
    grads["tok"] = dtok
    _fd_check(f, tensors, grads)


def test_fd_agg_shard_width():
    """Aggregation with A != d (a column shard of the projections)."""
    B, L, V, d, H, A = 1, 2, 3, 16, 2, 8
    tok = _rand(B, L, V, d)
    prm = _agg_prm(d, A, L)
    Rw = _rand(B, L, d)

    def f():
        return float((O.agg_fwd(tok, prm, H)[0] * Rw).sum())

    z, cache = O.agg_fwd(tok, prm, H)
    dtok, gr = O.agg_bwd(Rw, cache, prm)
    t = dict(prm, tok=tok)
    g = dict(gr, tok=dtok)
    _fd_check(f, t, g)


@pytest.mark.parametrize("final_ln", [1, 0])
def test_fd_head(final_ln):
    B, L, d, n = 2, 3, 8, 12
    x = _rand(B, L, d)
    prm = _head_prm(d, n)
    Rw = _rand(B, L, n)

    def f():
        return float((O.head_fwd(x, prm, final_ln)[0] * Rw).sum())

    pred, cache = O.head_fwd(x, prm, final_ln)
    dx, gr = O.head_bwd(Rw, cache, prm)
    t = dict(x=x)
    g = dict(x=dx)
    for k in ("w_h", "b_h") + (("lnf_g", "lnf_b") if final_ln else ()):
        t[k] = prm[k]
        g[k] = gr[k]
    _fd_check(f, t, g)


def test_fd_patch_embed():
    B, V, Hg, Wg, p, d = 2, 3, 8, 12, 4, 5
    img = _rand(B, V, Hg, Wg)
    w = _rand(V, p * p, d)
    b = _rand(V, d)
    ve = _rand(V, d)
    L = (Hg // p) * (Wg // p)
    Rw = _rand(B, L, V, d)

    def f():
        return float((O.patch_embed_fwd(img, w, b, ve, p) * Rw).sum())

    gr = O.patch_embed_bwd(img, Rw, p)
    _fd_check(f, {"w_pe": w, "b_pe": b, "ve": ve}, gr)


def test_fd_mse():
    pred = _rand(3, 4, 5)
    tgt = _rand(3, 4, 5)
    loss, dpred = O.mse(pred, tgt)
    _fd_check(lambda: O.mse(pred, tgt)[0], {"pred": pred}, {"pred": dpred}, full_max=100)


def test_fd_whole_model():
    B, V, Hg, Wg, p, d, H, F, nb = 1, 2, 8, 8, 4, 8, 2, 16, 2
    L = (Hg // p) * (Wg // p)
    img = _rand(B, V, Hg, Wg)
    tgt = _rand(B, L, V * p * p)
    emb = {"w_pe": _rand(V, p * p, d, s=0.3), "b_pe": _rand(V, d, s=0.3), "ve": _rand(V, d, s=0.3)}
    agg = _agg_prm(d, d, L)
    blocks = [_block_prm(d, d, F, d // H) for _ in range(nb)]
    head = _head_prm(d, V * p * p)
    kw = dict(p=p, agg_heads=H, heads=H)

    def f():
        return O.model_fwd_bwd(img, tgt, emb, agg, blocks, head, **kw)[0]

    loss, pred, g = O.model_fwd_bwd(img, tgt, emb, agg, blocks, head, **kw)
    t, gg = {}, {}
    for k in emb:
        t["e." + k], gg["e." + k] = emb[k], g["embed"][k]
    for k in agg:
        t["a." + k], gg["a." + k] = agg[k], g["agg"][k]
    for i, bp in enumerate(blocks):
        for k in bp:
            t[f"b{i}.{k}"], gg[f"b{i}.{k}"] = bp[k], g["blocks"][i][k]
    for k in head:
        t["h." + k], gg["h." + k] = head[k], g["head"][k]
    _fd_check(f, t, gg, full_max=8)


# ---------------------------------------------------------------------------
# Golden fixtures (closed forms fixed by mathematics)
# ---------------------------------------------------------------------------

def _read(name):
    rows = []
    with open(os.path.join(GOLD, name)) as fh:
        for line in fh:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def test_golden_normal_cdf_gelu():
    for x, phi in _read("normal_cdf.txt"):
        x, phi = float(x), float(phi)
        assert abs(O.gelu(np.array([x]))[0] - x * phi) < 1e-14
        # derivative: Phi(x) + x phi(x) with phi the normal density
        dens = math.exp(-0.5 * x * x) / math.sqrt(2 * math.pi)
        assert abs(O.gelu_grad(np.array([x]))[0] - (phi + x * dens)) < 1e-14


def test_golden_attention():
    rows = _read("attention_closed_form.txt")
    get = lambda tag: np.array([[float(v) for v in r[1:]] for r in rows if r[0] == tag])
    q, k, v, out, w = get("q"), get("k"), get("v"), get("out"), get("weights")
    o, P = O.attention_fwd(q, k, v)
    assert np.allclose(o, out, atol=1e-14, rtol=0)
    assert np.allclose(P, w, atol=1e-15, rtol=0)


def test_golden_layernorm():
    rows = _read("layernorm_closed_form.txt")
    x = np.array([[float(v) for v in rows[0][1:]]])
    y = np.array([[float(v) for v in rows[1][1:]]])
    got, _ = O.layer_norm_fwd(x, np.ones(4), np.zeros(4), 0.0)
    assert np.allclose(got, y, atol=1e-15, rtol=0)


def test_golden_patchify():
    img = np.arange(64, dtype=np.float64).reshape(1, 1, 8, 8)
    P = O.patchify(img, 4)
    for r in _read("patchify_8x8.txt"):
        l = int(r[0])
        assert list(P[0, 0, l]) == [float(v) for v in r[1:]]


# ---------------------------------------------------------------------------
# P2/P3/P5/P6/P7/P8/P11/P12: invariants and special cases
# ---------------------------------------------------------------------------

def test_softmax_rows_sum_to_one():
    s = _rand(7, 11, s=30.0)
    P = O.softmax(s)
    assert np.all(P >= 0)
    assert np.allclose(P.sum(-1), 1.0, atol=1e-12, rtol=0)
    _, c = O.agg_fwd(_rand(2, 3, 5, 8), _agg_prm(8, 8, 3), 2)
    assert np.allclose(c["a"].sum(-1), 1.0, atol=1e-12, rtol=0)


def test_identical_keys_give_mean_of_values():
    q = _rand(4, 6)
    k = np.repeat(_rand(1, 6), 9, axis=0)
    v = _rand(9, 6)
    o, _ = O.attention_fwd(q, k, v)
    assert np.allclose(o, np.broadcast_to(v.mean(0), o.shape), atol=1e-13, rtol=0)


def test_agg_identical_tokens_closed_form():
    """All V tokens of a patch equal: attention weights are uniform, so
    z = (x W_v + b_v) W_o + b_o + pos."""
    B, L, V, d, H = 2, 3, 5, 8, 2
    x = _rand(B, L, 1, d)
    tok = np.repeat(x, V, axis=2)
    prm = _agg_prm(d, d, L)
    z, c = O.agg_fwd(tok, prm, H)
    assert np.allclose(c["a"], 1.0 / V, atol=1e-14)
    want = (x[:, :, 0] @ prm["w_v"] + prm["b_v"]) @ prm["w_o"] + prm["b_o"] + prm["pos"]
    assert np.allclose(z, want, atol=1e-12, rtol=0)


def test_agg_single_variable_is_two_linears():
    B, L, d, H = 2, 4, 8, 4
    tok = _rand(B, L, 1, d)
    prm = _agg_prm(d, d, L)
    z, _ = O.agg_fwd(tok, prm, H)
    want = (tok[:, :, 0] @ prm["w_v"] + prm["b_v"]) @ prm["w_o"] + prm["b_o"] + prm["pos"]
    assert np.allclose(z, want, atol=1e-12, rtol=0)


def test_attention_single_token_returns_value():
    q, k, v = _rand(1, 4), _rand(1, 4), _rand(1, 4)
    o, _ = O.attention_fwd(q, k, v)
    assert np.allclose(o, v, atol=1e-15, rtol=0)


def test_layernorm_moments_and_backward_orthogonality():
    x = _rand(6, 32, s=3.0) + 5.0
    eps = 1e-5
    y, (xhat, rstd) = O.layer_norm_fwd(x, np.ones(32), np.zeros(32), eps)
    var = x.var(axis=-1)
    assert np.allclose(y.mean(-1), 0.0, atol=1e-12)
    assert np.allclose((y ** 2).mean(-1), var / (var + eps), atol=1e-12, rtol=0)
    # backward: sum(dx) = 0 always; sum(dx * xhat) = 0 when eps = 0, because then
    # xhat has unit mean square exactly
    _, (xhat, rstd) = O.layer_norm_fwd(x, np.ones(32), np.zeros(32), 0.0)
    g = 1 + _rand(32, s=0.2)
    dx, _, _ = O.layer_norm_bwd(_rand(6, 32), (xhat, rstd), g)
    assert np.allclose(dx.sum(-1), 0.0, atol=1e-11)
    assert np.allclose((dx * xhat).sum(-1), 0.0, atol=1e-11)


def test_gelu_closed_forms():
    x = np.linspace(-6, 6, 101)
    assert np.allclose(O.gelu(x) - O.gelu(-x), x, atol=1e-14, rtol=0)
    assert O.gelu_grad(np.array([0.0]))[0] == 0.5
    assert abs(O.gelu(np.array([12.0]))[0] - 12.0) < 1e-12
    assert abs(O.gelu(np.array([-12.0]))[0]) < 1e-12


def test_key_bias_gradient_vanishes():
    """Adding a constant vector to every key of one query shifts all its scores
    equally, which softmax ignores: the key-bias gradient is exactly zero."""
    _, c = O.agg_fwd(_rand(2, 3, 4, 8), _agg_prm(8, 8, 3), 2)
    _, gr = O.agg_bwd(_rand(2, 3, 8), c, _agg_prm(8, 8, 3))
    assert np.abs(gr["b_k"]).max() < 1e-12
    prm = _block_prm(16, 16, 32, 8)
    y, cb = O.block_fwd(_rand(2, 5, 16), prm, 2, qk_norm=0)
    _, gb = O.block_bwd(_rand(2, 5, 16), cb, prm)
    A = 16
    assert np.abs(gb["b_qkv"][A:2 * A]).max() < 1e-12


def test_identity_block_when_branches_are_zero():
    d = 16
    prm = _block_prm(d, d, 32, 8)
    for k in ("w_proj", "b_proj", "w_fc2", "b_fc2"):
        prm[k] = np.zeros_like(prm[k])
    x = _rand(2, 5, d)
    y, c = O.block_fwd(x, prm, 2)
    assert np.array_equal(y, x)
    dy = _rand(2, 5, d)
    dx, _ = O.block_bwd(dy, c, prm)
    assert np.allclose(dx, dy, atol=1e-15, rtol=0)


def test_mse_closed_form():
    t = _rand(3, 4)
    loss, dp = O.mse(t, t)
    assert loss == 0.0 and np.all(dp == 0.0)
    pred = t + 2.0
    loss, dp = O.mse(pred, t, scale=3.0)
    assert abs(loss - 4.0) < 1e-14
    assert np.allclose(dp, 2 * 2.0 / t.size * 3.0)


def test_patch_embed_linearity():
    B, V, p, d = 2, 3, 4, 6
    img1, img2 = _rand(B, V, 8, 8), _rand(B, V, 8, 8)
    w, b, ve = _rand(V, p * p, d), _rand(V, d), _rand(V, d)
    f = lambda im: O.patch_embed_fwd(im, w, b, ve, p)
    off = f(np.zeros_like(img1))
    a, c = 1.7, -0.3
    lhs = f(a * img1 + c * img2) - off
    rhs = a * (f(img1) - off) + c * (f(img2) - off)
    assert np.allclose(lhs, rhs, atol=1e-12, rtol=0)


def test_head_linearity_without_final_ln():
    prm = _head_prm(8, 12)
    x1, x2 = _rand(2, 3, 8), _rand(2, 3, 8)
    f = lambda x: O.head_fwd(x, prm, 0)[0] - prm["b_h"]
    assert np.allclose(f(2 * x1 - x2), 2 * f(x1) - f(x2), atol=1e-12, rtol=0)


# ---------------------------------------------------------------------------
# P4: scalar-loop brute force on tiny shapes
# ---------------------------------------------------------------------------

def _bf_ln(row, g, b, eps):
    n = len(row)
    m = sum(row) / n
    var = sum((r - m) ** 2 for r in row) / n
    return [(row[i] - m) / math.sqrt(var + eps) * g[i] + b[i] for i in range(n)]


def _bf_attn(q, k, v):
    dh = len(q[0])
    out = []
    for qi in q:
        s = [sum(qi[c] * kj[c] for c in range(dh)) / math.sqrt(dh) for kj in k]
        m = max(s)
        e = [math.exp(x - m) for x in s]
        z = sum(e)
        out.append([sum(e[j] / z * v[j][c] for j in range(len(k))) for c in range(dh)])
    return out


def _mm(a, b):
    return [[sum(a[i][t] * b[t][j] for t in range(len(b))) for j in range(len(b[0]))]
            for i in range(len(a))]


def test_brute_force_block():
    B, L, d, H, F = 1, 3, 4, 2, 6
    dh = d // H
    x = _rand(B, L, d)
    prm = _block_prm(d, d, F, dh)
    y, _ = O.block_fwd(x, prm, H, 1, 1e-5)
    P = {k: v.tolist() for k, v in prm.items()}
    xs = x[0].tolist()
    h1 = [_bf_ln(r, P["ln1_g"], P["ln1_b"], 1e-5) for r in xs]
    qkv = [[v + b for v, b in zip(r, P["b_qkv"])] for r in _mm(h1, P["w_qkv"])]
    o = [[0.0] * d for _ in range(L)]
    for h in range(H):
        q = [_bf_ln(r[h * dh:(h + 1) * dh], P["qn_g"], P["qn_b"], 1e-5) for r in qkv]
        k = [_bf_ln(r[d + h * dh:d + (h + 1) * dh], P["kn_g"], P["kn_b"], 1e-5) for r in qkv]
        v = [r[2 * d + h * dh:2 * d + (h + 1) * dh] for r in qkv]
        oh = _bf_attn(q, k, v)
        for t in range(L):
            o[t][h * dh:(h + 1) * dh] = oh[t]
    x1 = [[xs[t][j] + sum(o[t][i] * P["w_proj"][i][j] for i in range(d)) + P["b_proj"][j]
           for j in range(d)] for t in range(L)]
    h2 = [_bf_ln(r, P["ln2_g"], P["ln2_b"], 1e-5) for r in x1]
    u = [[v + b for v, b in zip(r, P["b_fc1"])] for r in _mm(h2, P["w_fc1"])]
    g = [[0.5 * a * (1 + math.erf(a / math.sqrt(2))) for a in r] for r in u]
    yb = [[x1[t][j] + sum(g[t][i] * P["w_fc2"][i][j] for i in range(F)) + P["b_fc2"][j]
           for j in range(d)] for t in range(L)]
    assert np.allclose(y[0], np.array(yb), atol=1e-12, rtol=0)


def test_brute_force_agg():
    B, L, V, d, H = 1, 2, 3, 4, 2
    dh = d // H
    tok = _rand(B, L, V, d)
    prm = _agg_prm(d, d, L)
    z, _ = O.agg_fwd(tok, prm, H)
    P = {k: v.tolist() for k, v in prm.items()}
    q = [sum(P["q0"][i] * P["w_q"][i][j] for i in range(d)) + P["b_q"][j] for j in range(d)]
    for l in range(L):
        X = tok[0, l].tolist()
        K = [[sum(X[v][i] * P["w_k"][i][j] for i in range(d)) + P["b_k"][j] for j in range(d)]
             for v in range(V)]
        Vv = [[sum(X[v][i] * P["w_v"][i][j] for i in range(d)) + P["b_v"][j] for j in range(d)]
              for v in range(V)]
        zh = []
        for h in range(H):
            zh += _bf_attn([q[h * dh:(h + 1) * dh]], [r[h * dh:(h + 1) * dh] for r in K],
                           [r[h * dh:(h + 1) * dh] for r in Vv])[0]
        zz = [sum(zh[i] * P["w_o"][i][j] for i in range(d)) + P["b_o"][j] + P["pos"][l][j]
              for j in range(d)]
        assert np.allclose(z[0, l], zz, atol=1e-12, rtol=0)


def test_brute_force_patch_embed():
    B, V, p, d = 1, 2, 4, 3
    img = _rand(B, V, 8, 4)
    w, b, ve = _rand(V, p * p, d), _rand(V, d), _rand(V, d)
    tok = O.patch_embed_fwd(img, w, b, ve, p)
    for v in range(V):
        for ph in range(2):
            for pw in range(1):
                l = ph * 1 + pw
                for e in range(d):
                    s = b[v, e] + ve[v, e]
                    for i in range(p):
                        for j in range(p):
                            s += img[0, v, ph * p + i, pw * p + j] * w[v, i * p + j, e]
                    assert abs(tok[0, l, v, e] - s) < 1e-12


# ---------------------------------------------------------------------------
# P9: Eq. (2) and Eq. (3) — column/row shard sums of each sub-layer
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("K", [2, 4])
@pytest.mark.parametrize("branch", ["attn", "mlp"])
def test_hybrid_stop_shard_sum(K, branch):
    B, L, d, H, dh, F = 2, 6, 16, 4, 4, 32
    A = H * dh
    x = _rand(B, L, d)
    dy = _rand(B, L, d)
    prm = _block_prm(d, A, F, dh)
    zero = ("w_fc2", "b_fc2") if branch == "attn" else ("w_proj", "b_proj")
    for k in zero:
        prm[k] = np.zeros_like(prm[k])
    y, c = O.block_fwd(x, prm, H)
    dx, g = O.block_bwd(dy, c, prm)
    ysum = np.zeros_like(x)
    dxsum = np.zeros_like(x)
    for k in range(K):
        pk = O.shard_block_params(prm, H, F, K, k, keep_bias=(k == 0))
        yk, ck = O.block_fwd(x, pk, H // K)
        dxk, gk = O.block_bwd(dy, ck, pk)
        ysum += yk - x          # partial output x A_{*,k} B_{k,*} of Eq. (2)
        dxsum += dxk - dy       # partial input gradient of Eq. (3)
        # shard gradients are the matching slices of the full gradients
        hk = H // K
        cols = np.arange(k * hk * dh, (k + 1) * hk * dh)
        if branch == "attn":
            qkv_cols = np.concatenate([cols, A + cols, 2 * A + cols])
            assert np.allclose(gk["w_qkv"], g["w_qkv"][:, qkv_cols], atol=1e-12)
            assert np.allclose(gk["w_proj"], g["w_proj"][cols], atol=1e-12)
        else:
            fc = np.arange(k * F // K, (k + 1) * F // K)
            assert np.allclose(gk["w_fc1"], g["w_fc1"][:, fc], atol=1e-12)
            assert np.allclose(gk["w_fc2"], g["w_fc2"][fc], atol=1e-12)
    assert np.allclose(ysum, y - x, atol=1e-12, rtol=0)
    assert np.allclose(dxsum, dx - dy, atol=1e-12, rtol=0)


def test_store_hook_is_identity_when_exact():
    """The storage hook does not touch the arithmetic: identity storage gives
    bitwise the same results as none, and bf16 storage moves them slightly."""
    x = _rand(2, 5, 16)
    prm = _block_prm(16, 16, 32, 8)
    dy = _rand(2, 5, 16)
    y0, c0 = O.block_fwd(x, prm, 2)
    y1, c1 = O.block_fwd(x, prm, 2, store=lambda a: a)
    assert np.array_equal(y0, y1)
    assert np.array_equal(O.block_bwd(dy, c0, prm)[0], O.block_bwd(dy, c1, prm)[0])
    import synth
    r = lambda a: synth.bf16_round(np.asarray(a, np.float32)).astype(np.float64)
    y2, _ = O.block_fwd(x, prm, 2, store=r)
    e = np.abs(y2 - y0).max() / np.abs(y0).max()
    assert 0 < e < 2e-2


# ---------------------------------------------------------------------------
# latitude-weighted MSE (Sec. IV) and the multi-layer prediction head (Sec. II)
# ---------------------------------------------------------------------------
def test_lat_weights_closed_forms():
    # 2 rows at +-45 degrees: equal weights; 4 rows at +-22.5 / +-67.5 degrees:
    # cos(67.5) / cos(22.5) = tan(22.5) = sqrt(2) - 1 and a mean of 1 give
    # weights 2 - sqrt(2) and sqrt(2)
    assert np.allclose(O.lat_weights(2), [1.0, 1.0], atol=1e-15)
    r2 = np.sqrt(2.0)
    assert np.allclose(O.lat_weights(4), [2 - r2, r2, r2, 2 - r2], atol=1e-14)
    w = O.lat_weights(128)
    assert abs(w.mean() - 1.0) < 1e-14 and np.allclose(w, w[::-1], atol=1e-14)
    # sum of cos over equiangular cell centres = 1 / sin(pi / (2H)), so w[y] = cos(lat_y) H sin(pi / (2H))
    H = 128
    lat = np.deg2rad(-90 + (np.arange(H) + 0.5) * 180 / H)
    assert np.allclose(w, np.cos(lat) * H * np.sin(np.pi / (2 * H)), atol=1e-13)


def _tok_layout(img, p):
    B, V = img.shape[:2]
    return O.patchify(img, p).transpose(0, 2, 1, 3).reshape(B, -1, V * p * p)


def test_wmse_layout_roundtrip_and_special_cases():
    r = np.random.default_rng(7)
    img = r.standard_normal((2, 3, 8, 12))
    tok = _tok_layout(img, 4)
    assert np.array_equal(O.unpatchify(tok, 3, 4), img)
    tgt = _tok_layout(r.standard_normal((2, 3, 8, 12)), 4)
    # pred = tgt: zero loss and gradient
    l0, g0 = O.wmse(tgt, tgt, 3, 4)
    assert l0 == 0.0 and not g0.any()
    # a residual constant over the grid: the weights average to 1, so the loss
    # is the plain MSE (the square of the constant)
    l1, _ = O.wmse(tgt + 0.5, tgt, 3, 4)
    assert abs(l1 - 0.25) < 1e-14
    # a residual on the two equatorial rows only weighs more than one on the
    # two polar rows (cells shrink towards the poles)
    eq, po = np.zeros((2, 3, 8, 12)), np.zeros((2, 3, 8, 12))
    eq[:, :, 3:5] = 1.0
    po[:, :, [0, 7]] = 1.0
    le = O.wmse(_tok_layout(eq, 4), 0 * tgt, 3, 4)[0]
    lp = O.wmse(_tok_layout(po, 4), 0 * tgt, 3, 4)[0]
    assert le > 4.5 * lp


def test_wmse_brute_force():
    """Scalar loop over the token layout: the row of element (b, l, v*16 + i*4 + j)
    is (l // Wp) * 4 + i; its weight is cos(latitude) over the mean of cos."""
    r = np.random.default_rng(8)
    B, L, V, Wp, p = 1, 6, 2, 3, 4
    pred = r.standard_normal((B, L, V * p * p))
    tgt = r.standard_normal((B, L, V * p * p))
    H = (L // Wp) * p
    lat = [math.radians(-90 + (y + 0.5) * 180 / H) for y in range(H)]
    cm = sum(math.cos(a) for a in lat) / H
    tot, n, g = 0.0, pred.size, np.zeros_like(pred)
    for l in range(L):
        for c in range(V * p * p):
            y = (l // Wp) * p + (c % (p * p)) // p
            w = math.cos(lat[y]) / cm
            e = pred[0, l, c] - tgt[0, l, c]
            tot += w * e * e
            g[0, l, c] = 2 * w * e / n * 1.5
    loss, dpred = O.wmse(pred, tgt, Wp, p, scale=1.5)
    assert abs(loss - tot / n) < 1e-12 and np.allclose(dpred, g, atol=1e-15)


def test_fd_wmse():
    r = np.random.default_rng(9)
    pred = r.standard_normal((2, 6, 32))
    tgt = r.standard_normal((2, 6, 32))
    loss, dpred = O.wmse(pred, tgt, 3, 4)
    _fd_check(lambda: O.wmse(pred, tgt, 3, 4)[0], {"pred": pred}, {"pred": dpred}, full_max=400)


@pytest.mark.parametrize("final_ln", [0, 1])
def test_fd_decoder_head(final_ln):
    """The head with two hidden GELU layers (the ClimaX decoder) against finite differences."""
    r = np.random.default_rng(10)
    d, n, nh = 8, 12, 2
    x = r.standard_normal((2, 3, d))
    prm = _head_prm(d, n)
    prm["w_hid"] = r.standard_normal((nh, d, d)) * 0.5
    prm["b_hid"] = r.standard_normal((nh, d)) * 0.3
    Rw = r.standard_normal((2, 3, n))

    def f():
        return float((O.head_fwd(x, prm, final_ln)[0] * Rw).sum())

    pred, cache = O.head_fwd(x, prm, final_ln)
    dx, gr = O.head_bwd(Rw, cache, prm)
    tensors = {"x": x, **{k: v for k, v in prm.items() if final_ln or not k.startswith("lnf")}}
    grads = {"x": dx, **{k: gr[k] for k in tensors if k != "x"}}
    _fd_check(f, tensors, grads, full_max=400)


def test_decoder_head_without_hidden_layers_is_the_linear_head():
    r = np.random.default_rng(11)
    d, n = 8, 12
    x = r.standard_normal((2, 3, d))
    prm = _head_prm(d, n)
    p0 = dict(prm, w_hid=np.zeros((0, d, d)), b_hid=np.zeros((0, d)))
    a, ca = O.head_fwd(x, prm, 1)
    b, cb = O.head_fwd(x, p0, 1)
    assert np.array_equal(a, b)
    Rw = r.standard_normal((2, 3, n))
    ga, gb = O.head_bwd(Rw, ca, prm)[1], O.head_bwd(Rw, cb, p0)[1]
    for k in ga:
        assert np.array_equal(ga[k], gb[k]), k
