"""P10: the oracle against independent library code (PyTorch CPU, float64 autograd).

PyTorch's Conv2d, LayerNorm, GELU, scaled_dot_product_attention and
MultiheadAttention are independent implementations of the definitions the
oracle writes out; autograd supplies independent gradients. Used in tests
only, never in the product.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

import oracle as O

R = np.random.default_rng(777)
T64 = torch.float64


def _t(a, grad=True):
    return torch.tensor(np.asarray(a), dtype=T64, requires_grad=grad)


def _rand(*shape, s=1.0):
    return R.standard_normal(shape) * s


def _torch_block(x, p, H, qk_norm, eps):
    d = x.shape[-1]
    A = p["w_proj"].shape[0]
    dh = A // H
    B, L, _ = x.shape
    h1 = Fn.layer_norm(x, (d,), p["ln1_g"], p["ln1_b"], eps)
    qkv = h1 @ p["w_qkv"] + p["b_qkv"]
    q, k, v = qkv[..., :A], qkv[..., A:2 * A], qkv[..., 2 * A:]
    sh = lambda t: t.reshape(B, L, H, dh).transpose(1, 2)
    q, k, v = sh(q), sh(k), sh(v)
    if qk_norm:
        q = Fn.layer_norm(q, (dh,), p["qn_g"], p["qn_b"], eps)
        k = Fn.layer_norm(k, (dh,), p["kn_g"], p["kn_b"], eps)
    o = Fn.scaled_dot_product_attention(q, k, v)
    o = o.transpose(1, 2).reshape(B, L, A)
    x1 = x + o @ p["w_proj"] + p["b_proj"]
    h2 = Fn.layer_norm(x1, (d,), p["ln2_g"], p["ln2_b"], eps)
    u = h2 @ p["w_fc1"] + p["b_fc1"]
    return x1 + Fn.gelu(u, approximate="none") @ p["w_fc2"] + p["b_fc2"]


def _block_prm(d, A, F, dh, s=0.3):
    shapes = {"ln1_g": (d,), "ln1_b": (d,), "w_qkv": (d, 3 * A), "b_qkv": (3 * A,),
              "qn_g": (dh,), "qn_b": (dh,), "kn_g": (dh,), "kn_b": (dh,),
              "w_proj": (A, d), "b_proj": (d,), "ln2_g": (d,), "ln2_b": (d,),
              "w_fc1": (d, F), "b_fc1": (F,), "w_fc2": (F, d), "b_fc2": (d,)}
    p = {k: _rand(*v, s=s) for k, v in shapes.items()}
    for g in ("ln1_g", "ln2_g", "qn_g", "kn_g"):
        p[g] += 1.0
    return p


@pytest.mark.parametrize("qk_norm", [1, 0])
@pytest.mark.parametrize("A", [32, 16])
def test_block_vs_torch(qk_norm, A):
    B, L, d, H, F = 2, 7, 32, 4 if A == 32 else 2, 64
    dh = A // H
    x = _rand(B, L, d)
    prm = _block_prm(d, A, F, dh)
    dy = _rand(B, L, d)
    y, c = O.block_fwd(x, prm, H, qk_norm, 1e-5)
    dx, g = O.block_bwd(dy, c, prm)

    xt = _t(x)
    pt = {k: _t(v) for k, v in prm.items()}
    yt = _torch_block(xt, pt, H, qk_norm, 1e-5)
    yt.backward(torch.tensor(dy, dtype=T64))
    assert np.allclose(y, yt.detach().numpy(), atol=1e-12, rtol=0)
    assert np.allclose(dx, xt.grad.numpy(), atol=1e-11, rtol=0)
    for k in prm:
        tg = pt[k].grad
        tg = np.zeros_like(prm[k]) if tg is None else tg.numpy()
        assert np.allclose(g[k], tg, atol=1e-11, rtol=0), k


def _torch_patch_embed(img, w_pe, b_pe, ve, p):
    """Per-variable stride-p convolution (groups = V)."""
    V, pp, d = w_pe.shape
    B = img.shape[0]
    wt = w_pe.permute(0, 2, 1).reshape(V * d, 1, p, p)
    e = Fn.conv2d(img, wt, (b_pe + ve).reshape(V * d), stride=p, groups=V)  # [B, V*d, nh, nw]
    nh, nw = e.shape[2], e.shape[3]
    return e.reshape(B, V, d, nh * nw).permute(0, 3, 1, 2)      # [B, L, V, d]


def _torch_agg(tok, p, H):
    """Single learned query over the V tokens of each patch with nn.MultiheadAttention."""
    B, L, V, d = tok.shape
    mha = torch.nn.MultiheadAttention(d, H, bias=True, batch_first=True, dtype=T64)
    with torch.no_grad():
        mha.in_proj_weight.copy_(torch.cat([p["w_q"].T, p["w_k"].T, p["w_v"].T], 0))
        mha.in_proj_bias.copy_(torch.cat([p["b_q"], p["b_k"], p["b_v"]]))
        mha.out_proj.weight.copy_(p["w_o"].T)
        mha.out_proj.bias.copy_(p["b_o"])
    X = tok.reshape(B * L, V, d)
    q = p["q0"].reshape(1, 1, d).expand(B * L, 1, d)
    out, _ = mha(q, X, X, need_weights=False)
    return out.reshape(B, L, d) + p["pos"], mha


def test_patch_embed_vs_conv():
    B, V, Hg, Wg, p, d = 2, 3, 8, 12, 4, 6
    img = _rand(B, V, Hg, Wg)
    w, b, ve = _rand(V, p * p, d), _rand(V, d), _rand(V, d)
    tok = O.patch_embed_fwd(img, w, b, ve, p)
    wt, bt, vt = _t(w), _t(b), _t(ve)
    tt = _torch_patch_embed(_t(img, False), wt, bt, vt, p)
    assert np.allclose(tok, tt.detach().numpy(), atol=1e-12, rtol=0)
    dt = _rand(*tok.shape)
    tt.backward(torch.tensor(dt, dtype=T64))
    g = O.patch_embed_bwd(img, dt, p)
    assert np.allclose(g["w_pe"], wt.grad.numpy(), atol=1e-11)
    assert np.allclose(g["b_pe"], bt.grad.numpy(), atol=1e-11)
    assert np.allclose(g["ve"], vt.grad.numpy(), atol=1e-11)


def test_agg_vs_multihead_attention():
    B, L, V, d, H = 2, 3, 5, 16, 4
    tok = _rand(B, L, V, d)
    prm = {"q0": _rand(d, s=.5), "w_q": _rand(d, d, s=.5), "b_q": _rand(d, s=.5),
           "w_k": _rand(d, d, s=.5), "b_k": _rand(d, s=.5), "w_v": _rand(d, d, s=.5),
           "b_v": _rand(d, s=.5), "w_o": _rand(d, d, s=.5), "b_o": _rand(d, s=.5),
           "pos": _rand(L, d, s=.5)}
    z, c = O.agg_fwd(tok, prm, H)
    dz = _rand(B, L, d)
    dtok, g = O.agg_bwd(dz, c, prm)
    tt = _t(tok)
    pt = {k: _t(v) for k, v in prm.items()}
    zt, mha = _torch_agg(tt, pt, H)
    assert np.allclose(z, zt.detach().numpy(), atol=1e-12, rtol=0)
    zt.backward(torch.tensor(dz, dtype=T64))
    assert np.allclose(dtok, tt.grad.numpy(), atol=1e-11)
    assert np.allclose(g["q0"], pt["q0"].grad.numpy(), atol=1e-11)
    assert np.allclose(g["pos"], pt["pos"].grad.numpy(), atol=1e-11)
    wg = mha.in_proj_weight.grad.numpy()
    bg = mha.in_proj_bias.grad.numpy()
    assert np.allclose(g["w_q"], wg[:d].T, atol=1e-11)
    assert np.allclose(g["w_k"], wg[d:2 * d].T, atol=1e-11)
    assert np.allclose(g["w_v"], wg[2 * d:].T, atol=1e-11)
    assert np.allclose(g["b_q"], bg[:d], atol=1e-11)
    assert np.allclose(g["b_k"], bg[d:2 * d], atol=1e-11)
    assert np.allclose(g["b_v"], bg[2 * d:], atol=1e-11)
    assert np.allclose(g["w_o"], mha.out_proj.weight.grad.numpy().T, atol=1e-11)
    assert np.allclose(g["b_o"], mha.out_proj.bias.grad.numpy(), atol=1e-11)


def test_whole_model_vs_torch():
    B, V, Hg, Wg, p, d, H, F, nb = 2, 3, 8, 16, 4, 16, 2, 32, 2
    L = (Hg // p) * (Wg // p)
    img = _rand(B, V, Hg, Wg)
    tgt = _rand(B, L, V * p * p)
    emb = {"w_pe": _rand(V, p * p, d, s=.3), "b_pe": _rand(V, d, s=.3), "ve": _rand(V, d, s=.3)}
    agg = {"q0": _rand(d, s=.3), "w_q": _rand(d, d, s=.3), "b_q": _rand(d, s=.3),
           "w_k": _rand(d, d, s=.3), "b_k": _rand(d, s=.3), "w_v": _rand(d, d, s=.3),
           "b_v": _rand(d, s=.3), "w_o": _rand(d, d, s=.3), "b_o": _rand(d, s=.3),
           "pos": _rand(L, d, s=.3)}
    blocks = [_block_prm(d, d, F, d // H) for _ in range(nb)]
    head = {"lnf_g": 1 + _rand(d, s=.3), "lnf_b": _rand(d, s=.3),
            "w_h": _rand(d, V * p * p, s=.3), "b_h": _rand(V * p * p, s=.3)}
    loss, pred, g = O.model_fwd_bwd(img, tgt, emb, agg, blocks, head, p=p, agg_heads=H, heads=H)

    et = {k: _t(v) for k, v in emb.items()}
    at = {k: _t(v) for k, v in agg.items()}
    bt = [{k: _t(v) for k, v in bp.items()} for bp in blocks]
    ht = {k: _t(v) for k, v in head.items()}
    tok = _torch_patch_embed(_t(img, False), et["w_pe"], et["b_pe"], et["ve"], p)
    x, mha = _torch_agg(tok, at, H)
    for bp in bt:
        x = _torch_block(x, bp, H, 1, 1e-5)
    xf = Fn.layer_norm(x, (d,), ht["lnf_g"], ht["lnf_b"], 1e-5)
    pr = xf @ ht["w_h"] + ht["b_h"]
    lt = Fn.mse_loss(pr, torch.tensor(tgt, dtype=T64))
    lt.backward()
    assert abs(loss - lt.item()) < 1e-12
    assert np.allclose(pred, pr.detach().numpy(), atol=1e-12)
    for k in emb:
        assert np.allclose(g["embed"][k], et[k].grad.numpy(), atol=1e-12), k
    for i in range(nb):
        for k in blocks[i]:
            assert np.allclose(g["blocks"][i][k], bt[i][k].grad.numpy(), atol=1e-12), (i, k)
    for k in head:
        assert np.allclose(g["head"][k], ht[k].grad.numpy(), atol=1e-12), k
    assert np.allclose(g["agg"]["q0"], at["q0"].grad.numpy(), atol=1e-12)
    assert np.allclose(g["agg"]["pos"], at["pos"].grad.numpy(), atol=1e-12)
    assert np.allclose(g["agg"]["w_o"], mha.out_proj.weight.grad.numpy().T, atol=1e-12)


def test_decoder_head_and_wmse_vs_torch():
    """The multi-layer prediction head (LayerNorm, two Linear + exact GELU
    layers, a final Linear; torch.nn modules) and the latitude-weighted MSE
    (torch's own fold back to the image layout and its cos), with autograd."""
    B, V, Hg, Wg, p, d, nh = 2, 3, 8, 12, 4, 16, 2
    Wp = Wg // p
    L = (Hg // p) * Wp
    n = V * p * p
    x = _rand(B, L, d)
    tgt = _rand(B, L, n)
    head = {"lnf_g": 1 + _rand(d, s=.3), "lnf_b": _rand(d, s=.3), "w_hid": _rand(nh, d, d, s=.4),
            "b_hid": _rand(nh, d, s=.3), "w_h": _rand(d, n, s=.3), "b_h": _rand(n, s=.3)}
    pred, cache = O.head_fwd(x, head, 1)
    loss, dpred = O.wmse(pred, tgt, Wp, p)
    dx, g = O.head_bwd(dpred, cache, head)

    xt = _t(x)
    ln = torch.nn.LayerNorm(d, eps=1e-5, dtype=T64)
    lins = [torch.nn.Linear(d, d, dtype=T64) for _ in range(nh)]
    out = torch.nn.Linear(d, n, dtype=T64)
    with torch.no_grad():
        ln.weight.copy_(torch.tensor(head["lnf_g"]))
        ln.bias.copy_(torch.tensor(head["lnf_b"]))
        for k, lin in enumerate(lins):
            lin.weight.copy_(torch.tensor(head["w_hid"][k].T))
            lin.bias.copy_(torch.tensor(head["b_hid"][k]))
        out.weight.copy_(torch.tensor(head["w_h"].T))
        out.bias.copy_(torch.tensor(head["b_h"]))
    h = ln(xt)
    for lin in lins:
        h = Fn.gelu(lin(h), approximate="none")
    pr = out(h)
    # token layout [B, L, V*p*p] -> image [B, V, H, W] with torch's fold
    cols = pr.reshape(B, L, V, p * p).permute(0, 2, 3, 1).reshape(B, V * p * p, L)
    img = Fn.fold(cols, (Hg, Wg), kernel_size=p, stride=p).reshape(B, V, Hg, Wg)
    tcols = torch.tensor(tgt).reshape(B, L, V, p * p).permute(0, 2, 3, 1).reshape(B, V * p * p, L)
    timg = Fn.fold(tcols, (Hg, Wg), kernel_size=p, stride=p).reshape(B, V, Hg, Wg)
    lat = torch.deg2rad(torch.linspace(-90 + 90 / Hg, 90 - 90 / Hg, Hg, dtype=T64))
    w = torch.cos(lat) / torch.cos(lat).mean()
    lt = (w[None, None, :, None] * (img - timg) ** 2).mean()
    lt.backward()
    assert abs(loss - lt.item()) < 1e-12
    assert np.allclose(pred, pr.detach().numpy(), atol=1e-12)
    assert np.allclose(dx, xt.grad.numpy(), atol=1e-12)
    assert np.allclose(g["lnf_g"], ln.weight.grad.numpy(), atol=1e-12)
    assert np.allclose(g["lnf_b"], ln.bias.grad.numpy(), atol=1e-12)
    for k, lin in enumerate(lins):
        assert np.allclose(g["w_hid"][k], lin.weight.grad.numpy().T, atol=1e-12), k
        assert np.allclose(g["b_hid"][k], lin.bias.grad.numpy(), atol=1e-12), k
    assert np.allclose(g["w_h"], out.weight.grad.numpy().T, atol=1e-12)
    assert np.allclose(g["b_h"], out.bias.grad.numpy(), atol=1e-12)
