"""Parity of every configuration at its full depth: the blocks chained as the
paper's model chains them (Sec. II), forward and backward, against the fp64
oracle run the same way.

* 115M-scale model: patch embedding, aggregation over 48 variables, 8 blocks,
  head and loss, on one sample of the full 128x256 grid (2048 patches).
* 1B-scale model: 91 variables with per-variable scales, 16 blocks of width
  2048, on one sample of the full 128x256 grid (2048 patches).
* 10B-scale shard: 4 chained shard blocks on the full batch of 2 x 2048
  tokens, the upstream gradient nonzero on the first sample only (samples are
  independent, so the oracle runs that sample and the other's input gradient
  must be exactly zero).
* 113B-scale shard: aggregation over 91 variables at width 16384 followed by 2
  shard blocks, on 512 of the 2048 patches (the oracle's unfolded key/value
  projections cost 2 x 512 x 91 x 16384 x 1024 flops each at this size, and
  its float64 copy of the token tensor takes 5.6 GB).

Every tensor is held to the bf16 bound 2e-2, except the query/key LayerNorm
parameter gradients of the blocks after the first, whose bf16 storage floor is
at or above that bound on these models (tests/test_bf16_floor.py); they are
compared in the *_qkln expected-failure tests with their errors reported.
"""
import time

import numpy as np
import pytest

import oracle as O
import synth
from helpers import TOL, check, dev, host, record
from test_gpu_parity import QKLN_PARAMS, _dims, _dev_params, check_pass, check_qkln_depth

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

_CACHE = {}


def _log(msg):
    print(msg, flush=True)


def _oracle_chain(x, prms, c, dy, tok=None, agg=None):
    ca = None
    if tok is not None:
        x, ca = O.agg_fwd(tok, agg, c.agg_heads)
    caches = []
    for p in prms:
        x, cc = O.block_fwd(x, p, c.heads, c.qk_norm, c.eps)
        caches.append(cc)
    y, g, grads = x, dy, [None] * len(prms)
    for i in range(len(prms) - 1, -1, -1):
        g, grads[i] = O.block_bwd(g, caches[i], prms[i])
        caches[i] = None
    ag = None
    if ca is not None:
        g, ag = O.agg_bwd(g, ca, agg)
    return y, g, grads, ag


def _check_blocks(G, rg, deferred):
    for i, gb in enumerate(rg):
        for k, v in gb.items():
            if i > 0 and k in QKLN_PARAMS:
                deferred.append((f"block{i}.d{k}", host(G[i][k]), v, gb["ln1_b"]))
                continue
            check(f"block{i}.d{k}", host(G[i][k]), v, TOL["bf16"], floor_ref=gb["ln1_b"])


def _full_model(lib, key, c):
    if key in _CACHE:
        return _CACHE[key]
    import torch
    from paper_2404_14712_amd.model import ViTPass
    try:
        img, tgt = synth.image(c), synth.target(c)
        emb, agg, head = synth.embed_params(c), synth.agg_params(c), synth.head_params(c)
        blocks = [synth.block_params(c, i) for i in range(c.blocks)]
        params = {"embed": _dev_params(emb, c.dtype), "agg": _dev_params(agg, c.dtype),
                  "blocks": [_dev_params(b, c.dtype) for b in blocks], "head": _dev_params(head, c.dtype)}
        _log(f"{key}: GPU pass B={c.B} L={c.L} V={c.V} d={c.d} blocks={c.blocks}")
        vp = ViTPass(lib, _dims(c, "full"), params)
        loss = vp.forward_backward({"img": dev(img, "f32"), "tgt": dev(tgt, "f32")})
        torch.cuda.synchronize()
        t = time.time()
        kw = dict(p=4, agg_heads=c.agg_heads, heads=c.heads, qk_norm=c.qk_norm, eps=c.eps)
        rl, pred, rg = O.model_fwd_bwd(img, tgt, emb, agg, blocks, head, **kw)
        _log(f"{key}: oracle {time.time() - t:.1f} s")
        _CACHE[key] = (None, check_pass(vp, loss, rl, pred, rg, c, TOL["bf16"]))
    except AssertionError as e:
        _CACHE[key] = (e, None)
    return _CACHE[key]


def _shard_chain(lib, key, c, keep=(0,)):
    if key in _CACHE:
        return _CACHE[key]
    import torch
    from paper_2404_14712_amd.model import ViTPass
    try:
        blocks = [synth.block_params(c, i) for i in range(c.blocks)]
        dy = synth.normal(c.seed, "dy", (c.B, c.L, c.d), dtype=c.dtype)
        drop = [b for b in range(c.B) if b not in keep]
        dy[drop] = 0.0
        keep = list(keep)
        params = {"blocks": [_dev_params(b, c.dtype) for b in blocks]}
        tok = agg = x = None
        if c.agg_only_prefix:
            tok = synth.normal(c.seed, "tok", (c.B, c.L, c.V, c.d), dtype=c.dtype)
            agg = synth.agg_params(c)
            params["agg"] = _dev_params(agg, c.dtype)
            mode, inputs = "agg_blocks", {"tok": dev(tok, c.dtype), "dy": dev(dy, c.dtype)}
        else:
            x = synth.activations(c, "x")
            mode, inputs = "blocks", {"x": dev(x, c.dtype), "dy": dev(dy, c.dtype)}
        _log(f"{key}: GPU pass mode={mode} B={c.B} L={c.L} d={c.d} blocks={c.blocks}")
        vp = ViTPass(lib, _dims(c, mode), params)
        dx = vp.forward_backward(inputs)
        torch.cuda.synchronize()
        y = vp.xs[-1]
        t = time.time()
        ry, rdx, rg, rag = _oracle_chain(None if x is None else x[keep], blocks, c, dy[keep],
                                         None if tok is None else tok[keep], agg)
        _log(f"{key}: oracle {time.time() - t:.1f} s")
        tol = TOL["bf16"]
        check("y", host(y[keep]), ry, tol)
        if mode == "blocks":
            check("dx", host(dx[keep]), rdx, tol)
            if drop:
                assert int(torch.count_nonzero(dx[drop])) == 0, "dx leaks into samples whose dy is zero"
        else:
            check("dtok", host(vp.dtok[keep]), rdx, tol)
            if drop:
                assert int(torch.count_nonzero(vp.dtok[drop])) == 0, "dtok leaks into samples whose dy is zero"
            for k, v in rag.items():
                check(f"agg.d{k}", host(vp.grads["agg"][k]), v, tol, floor_ref=rag["b_q"])
        deferred = []
        _check_blocks(vp.grads["blocks"], rg, deferred)
        _CACHE[key] = (None, deferred)
    except AssertionError as e:
        _CACHE[key] = (e, None)
    return _CACHE[key]


CHAINS = {
    "115m": lambda lib: _full_model(lib, "115m", synth.small_config("115m", B=1)),
    "1b": lambda lib: _full_model(lib, "1b", synth.small_config("1b", B=1)),
    "10b-shard": lambda lib: _shard_chain(lib, "10b-shard", synth.CONFIGS["10b-shard"]),
    "113b-shard": lambda lib: _shard_chain(lib, "113b-shard", synth.small_config("113b-shard", L=512)),
}


@pytest.mark.parametrize("key", list(CHAINS))
def test_chain(lib, key):
    err, _ = CHAINS[key](lib)
    if err is not None:
        raise err


@pytest.mark.xfail(strict=False, reason="bf16 storage floor of the QK-LayerNorm parameter gradients past the "
                                        "first block is at or above 2e-2 (tests/test_bf16_floor.py)")
@pytest.mark.parametrize("key", list(CHAINS))
def test_chain_qkln(lib, key):
    err, deferred = CHAINS[key](lib)
    if err is not None:
        raise err
    check_qkln_depth(deferred, TOL["bf16"])


# ---------------------------------------------------------------------------
# Eq. (2) / (3) on one GPU: K shards of a 10B-width block run one after
# another; their partial outputs and input gradients sum to the unsharded ones
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("K", [2, 4])
@pytest.mark.parametrize("branch", ["attention", "mlp"])
def test_shard_sum_gpu(lib, K, branch):
    import torch
    from paper_2404_14712_amd._lib import BlockDesc
    c = synth.small_config("10b-shard", B=1, L=512)
    H, F, d, dh = c.heads, c.mlp, c.d, c.head_dim
    x = synth.activations(c, "x")
    dy = synth.normal(c.seed, "dy", x.shape, dtype=c.dtype)
    prm = synth.block_params(c, 0)
    # one sub-layer at a time: the other branch's output weights and bias are zero
    zero = ("w_fc2", "b_fc2") if branch == "attention" else ("w_proj", "b_proj")
    for k in zero:
        prm[k] = np.zeros_like(prm[k])
    xd, dyd = dev(x, c.dtype), dev(dy, c.dtype)

    def run(p, heads, mlp):
        desc = BlockDesc(c.B, c.L, d, heads, dh, mlp, c.qk_norm, c.eps, 1)
        saved = torch.empty(lib.orbit_vit_block_saved_bytes(desc), dtype=torch.uint8, device="cuda")
        ws = torch.empty(lib.orbit_vit_block_workspace_bytes(desc), dtype=torch.uint8, device="cuda")
        pd = _dev_params(p, c.dtype)
        y = torch.empty_like(xd)
        dx = torch.empty_like(xd)
        g = {k: torch.empty(v.shape, dtype=torch.float32, device="cuda") for k, v in p.items()}
        lib.orbit_vit_block_fwd(desc, pd, xd, y, saved, ws)
        lib.orbit_vit_block_bwd(desc, pd, xd, saved, dyd, dx, g, 0, ws)
        torch.cuda.synchronize()
        return host(y), host(dx), {k: host(v) for k, v in g.items()}

    y_full, dx_full, g_full = run(prm, H, F)
    ysum = x.astype(np.float64).copy()
    dxsum = dy.astype(np.float64).copy()
    for k in range(K):
        pk = O.shard_block_params(prm, H, F, K, k, keep_bias=(k == 0))
        yk, dxk, gk = run(pk, H // K, F // K)
        ysum += yk - x
        dxsum += dxk - dy
    ref, cache = O.block_fwd(x, prm, H, c.qk_norm, c.eps)
    rdx, _ = O.block_bwd(dy, cache, prm)
    tol = TOL["bf16"]
    check(f"sum of {K} shard outputs vs oracle", ysum, ref, tol)
    check(f"sum of {K} shard input gradients vs oracle", dxsum, rdx, tol)
    check(f"sum of {K} shard outputs vs unsharded call", ysum, y_full, tol)
    check(f"sum of {K} shard input gradients vs unsharded call", dxsum, dx_full, tol)
