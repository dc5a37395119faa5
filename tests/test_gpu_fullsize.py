"""Parity at the full workload sizes, with the descriptors the benchmark
launches (the 115M- and 1B-scale models, the 10B-scale shard block and the
113B-scale shard aggregation + block).

Every compared value is computed by the fp64 oracle. Where the oracle cannot
afford every output, the upstream gradient is nonzero only on a sample (whole
batch elements for a block, single patches for the aggregation and the patch
embedding). The parameter gradients then reduce exactly to that sample, so
they are compared in full; the input gradient is compared on the sample and
must be exactly zero everywhere else (samples and patches are independent).
The bound is the per-tensor max relative error of bf16 mode, 2e-2.
"""
import numpy as np
import pytest

import oracle as O
import synth
from helpers import TOL, check, dev, host

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _dev_params(p: dict, dtype: str):
    return {k: (None if v is None else dev(v, dtype)) for k, v in p.items()}


def _sample_patches(c: synth.Config, per_batch: int):
    """(batch, patch) pairs: the first and last patch of every sample plus seeded others."""
    r = synth.rng(c.seed, "fullsize.patches")
    bs, ls = [], []
    for b in range(c.B):
        pick = {0, c.L - 1} | set(r.choice(c.L, size=per_batch - 2, replace=False).tolist())
        for l in sorted(pick):
            bs.append(b)
            ls.append(l)
    return np.array(bs), np.array(ls)


# ---------------------------------------------------------------------------
# transformer block: 115M (B=4, d=1024), 1B (B=2, d=2048), 10B shard
# (d=8192, 8 of 64 heads, MLP 4096 of 32768), 113B shard (d=16384)
# ---------------------------------------------------------------------------
BLOCK_FULL = [("115m", (0, 3)), ("1b", (1,)), ("10b-shard", (0,)), ("113b-shard", (0,))]


@pytest.mark.parametrize("workload,keep", BLOCK_FULL, ids=[w for w, _ in BLOCK_FULL])
def test_block_full_size(lib, workload, keep):
    import torch
    from paper_2404_14712_amd._lib import BlockDesc
    c = synth.CONFIGS[workload]
    x = synth.activations(c, "x")
    dy = synth.normal(c.seed, "dy", x.shape, dtype=c.dtype)
    drop = [b for b in range(c.B) if b not in keep]
    dy[drop] = 0.0
    prm = synth.block_params(c, 0)
    desc = BlockDesc(c.B, c.L, c.d, c.heads, c.head_dim, c.mlp, c.qk_norm, c.eps, 1)
    saved = torch.empty(lib.orbit_vit_block_saved_bytes(desc), dtype=torch.uint8, device="cuda")
    ws = torch.empty(lib.orbit_vit_block_workspace_bytes(desc), dtype=torch.uint8, device="cuda")
    pd = _dev_params(prm, c.dtype)
    xd = dev(x, c.dtype)
    y = torch.empty_like(xd)
    dx = torch.full_like(xd, 3.0)
    g = {k: torch.full(v.shape, 5.0, dtype=torch.float32, device="cuda") for k, v in prm.items()}
    lib.orbit_vit_block_fwd(desc, pd, xd, y, saved, ws)
    lib.orbit_vit_block_bwd(desc, pd, xd, saved, dev(dy, c.dtype), dx, g, 0, ws)
    torch.cuda.synchronize()
    keep = list(keep)
    ref, cache = O.block_fwd(x[keep], prm, c.heads, c.qk_norm, c.eps)
    rdx, rg = O.block_bwd(dy[keep], cache, prm)
    del cache
    tol = TOL[c.dtype]
    check("y", host(y[keep]), ref, tol)
    check("dx", host(dx[keep]), rdx, tol)
    if drop:
        assert int(torch.count_nonzero(dx[drop])) == 0, "dx leaks into samples whose dy is zero"
    for k in rg:
        check(f"d{k}", host(g[k]), rg[k], tol, floor_ref=rg["ln1_b"])


# ---------------------------------------------------------------------------
# the paper's own model shapes (Sec. IV): the 1B model (3072 wide, 16 heads of
# 192, unsharded), the 10B model's tensor-parallel shard over 8 GPUs (8192
# wide, 4 of 32 heads of 256, MLP 4096 of 32768) and the 113B model's (12288
# wide, 8 of 64 heads of 192, MLP 6144 of 49152): one block of 2048 tokens
# ---------------------------------------------------------------------------
PAPER_SHAPES = {
    "1b-paper": dict(d=3072, heads=16, head_dim=192, mlp=12288, sigma=0.02),
    "10b-paper-tp8": dict(d=8192, heads=4, head_dim=256, mlp=4096, sigma=0.01),
    "113b-paper-tp8": dict(d=12288, heads=8, head_dim=192, mlp=6144, sigma=0.005),
}


@pytest.mark.parametrize("name", list(PAPER_SHAPES))
def test_block_paper_shapes(lib, name):
    import torch
    from paper_2404_14712_amd._lib import BlockDesc
    c = synth.small_config("10b-shard", B=1, L=2048, **PAPER_SHAPES[name])
    x = synth.activations(c, "x")
    dy = synth.normal(c.seed, "dy", x.shape, dtype=c.dtype)
    prm = synth.block_params(c, 0)
    desc = BlockDesc(c.B, c.L, c.d, c.heads, c.head_dim, c.mlp, c.qk_norm, c.eps, 1)
    saved = torch.empty(lib.orbit_vit_block_saved_bytes(desc), dtype=torch.uint8, device="cuda")
    ws = torch.empty(lib.orbit_vit_block_workspace_bytes(desc), dtype=torch.uint8, device="cuda")
    pd = _dev_params(prm, c.dtype)
    xd = dev(x, c.dtype)
    y = torch.empty_like(xd)
    dx = torch.empty_like(xd)
    g = {k: torch.full(v.shape, 5.0, dtype=torch.float32, device="cuda") for k, v in prm.items()}
    print(f"{name}: block d={c.d} heads={c.heads}x{c.head_dim} mlp={c.mlp} L={c.L}", flush=True)
    lib.orbit_vit_block_fwd(desc, pd, xd, y, saved, ws)
    lib.orbit_vit_block_bwd(desc, pd, xd, saved, dev(dy, c.dtype), dx, g, 0, ws)
    torch.cuda.synchronize()
    ref, cache = O.block_fwd(x, prm, c.heads, c.qk_norm, c.eps)
    rdx, rg = O.block_bwd(dy, cache, prm)
    del cache
    tol = TOL[c.dtype]
    check("y", host(y), ref, tol)
    check("dx", host(dx), rdx, tol)
    for k in rg:
        check(f"d{k}", host(g[k]), rg[k], tol, floor_ref=rg["ln1_b"])


# ---------------------------------------------------------------------------
# aggregation: 115M (V=48), 1B (V=91), 113B shard (V=91, d=16384, 8 of 128 heads)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("workload,per_batch", [("115m", 8), ("1b", 8), ("113b-shard", 12)],
                         ids=["115m", "1b", "113b-shard"])
def test_var_aggregate_full_size(lib, workload, per_batch):
    import torch
    from paper_2404_14712_amd._lib import AggDesc
    c = synth.CONFIGS[workload]
    B, L, V, d, H = c.B, c.L, c.V, c.d, c.agg_heads
    tok = synth.device_normal(c.seed, "tok", (B * L, V, d), c.dtype, "cuda", chunk_rows=256).view(B, L, V, d)
    prm = synth.agg_params(c)
    bs, ls = _sample_patches(c, per_batch)
    dz_s = synth.normal(c.seed, "fullsize.dz", (len(bs), d), dtype=c.dtype)
    dz = torch.zeros(B, L, d, dtype=torch.bfloat16, device="cuda")
    dz[torch.from_numpy(bs), torch.from_numpy(ls)] = dev(dz_s, c.dtype)
    desc = AggDesc(B, L, V, d, H, c.agg_head_dim, 1)
    saved = torch.empty(lib.orbit_var_aggregate_saved_bytes(desc), dtype=torch.uint8, device="cuda")
    ws = torch.empty(lib.orbit_var_aggregate_workspace_bytes(desc), dtype=torch.uint8, device="cuda")
    pd = _dev_params(prm, c.dtype)
    z = torch.empty(B, L, d, dtype=torch.bfloat16, device="cuda")
    dtok = torch.empty_like(tok)
    g = {k: torch.full(v.shape, 5.0, dtype=torch.float32, device="cuda") for k, v in prm.items() if v is not None}
    lib.orbit_var_aggregate(desc, tok, pd, z, saved, ws)
    lib.orbit_var_aggregate_bwd(desc, tok, pd, saved, dz, dtok, g, 0, ws)
    torch.cuda.synchronize()
    bi, li = torch.from_numpy(bs).cuda(), torch.from_numpy(ls).cuda()
    tok_s = host(tok[bi, li])
    z_s = host(z[bi, li])
    dtok_s = host(dtok[bi, li])
    dtok[bi, li] = 0
    assert int(torch.count_nonzero(dtok)) == 0, "dtok leaks into patches whose dz is zero"
    del tok, dtok
    # the oracle on the sampled patches only, as one batch of len(bs) patches
    prm_s = dict(prm)
    if prm.get("pos") is not None:
        prm_s["pos"] = prm["pos"][ls]
    ref, cache = O.agg_fwd(tok_s[None], prm_s, H)
    rdtok, rg = O.agg_bwd(dz_s[None].astype(np.float64), cache, prm_s)
    if prm.get("pos") is not None:
        full = np.zeros((L, d))
        np.add.at(full, ls, rg["pos"])
        rg["pos"] = full
    tol = TOL[c.dtype]
    check("z", z_s, ref[0], tol)
    check("dtok", dtok_s, rdtok[0], tol)
    for k in rg:
        if k in g:
            check(f"d{k}", host(g[k]), rg[k], tol, floor_ref=rg["b_q"])


# ---------------------------------------------------------------------------
# patch embedding: 115M (4 x 48 variables), 1B (2 x 91 variables, scaled fields)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("workload", ["115m", "1b"])
def test_patch_embed_full_size(lib, workload):
    import torch
    from paper_2404_14712_amd._lib import EmbedDesc
    c = synth.CONFIGS[workload]
    B, L, V, d = c.B, c.L, c.V, c.d
    Hg, Wg = c.grid
    img = synth.image(c)
    e = synth.embed_params(c)
    bs, ls = _sample_patches(c, 8)
    dtok_s = synth.normal(c.seed, "fullsize.dtok", (len(bs), V, d), dtype=c.dtype)
    desc = EmbedDesc(B, V, Hg, Wg, 4, d, 1)
    tok = torch.empty(B, L, V, d, dtype=torch.bfloat16, device="cuda")
    dtok = torch.zeros_like(tok)
    bi, li = torch.from_numpy(bs).cuda(), torch.from_numpy(ls).cuda()
    dtok[bi, li] = dev(dtok_s, c.dtype)
    ed = _dev_params(e, c.dtype)
    imgd = dev(img, "f32")
    g = {k: torch.full(v.shape, 5.0, dtype=torch.float32, device="cuda") for k, v in e.items()}
    ws = torch.empty(lib.orbit_patch_embed_workspace_bytes(desc), dtype=torch.uint8, device="cuda")
    lib.orbit_patch_embed(desc, imgd, ed["w_pe"], ed["b_pe"], ed["ve"], tok)
    lib.orbit_patch_embed_bwd(desc, imgd, dtok, g["w_pe"], g["b_pe"], g["ve"], 0, ws)
    torch.cuda.synchronize()
    tok_s = host(tok[bi, li])
    del tok, dtok
    # a patch's tokens depend only on its own 4x4 pixels: the oracle runs per patch
    W4 = Wg // 4
    ref = np.empty((len(bs), V, d))
    rg = {k: 0.0 for k in e}
    for i, (b, l) in enumerate(zip(bs, ls)):
        ph, pw = divmod(int(l), W4)
        crop = img[b:b + 1, :, 4 * ph:4 * ph + 4, 4 * pw:4 * pw + 4]
        ref[i] = O.patch_embed_fwd(crop, e["w_pe"], e["b_pe"], e["ve"], 4)[0, 0]
        gi = O.patch_embed_bwd(crop, dtok_s[i][None, None], 4)
        for k in rg:
            rg[k] = rg[k] + gi[k]
    tol = TOL[c.dtype]
    check("tok", tok_s, ref, tol)
    for k in rg:
        check(f"d{k}", host(g[k]), rg[k], tol)


# ---------------------------------------------------------------------------
# head: 115M (out 768), 1B (out 1456); the oracle covers every output
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("workload", ["115m", "1b"])
def test_head_full_size(lib, workload):
    import torch
    from paper_2404_14712_amd._lib import HeadDesc
    c = synth.CONFIGS[workload]
    B, L, d, out = c.B, c.L, c.d, c.out_dim
    x = synth.activations(c, "x")
    prm = synth.head_params(c)
    desc = HeadDesc(B, L, d, out, 1, c.eps, 1)
    saved = torch.empty(lib.orbit_head_saved_bytes(desc), dtype=torch.uint8, device="cuda")
    ws = torch.empty(lib.orbit_head_workspace_bytes(desc), dtype=torch.uint8, device="cuda")
    pred = torch.empty(B, L, out, dtype=torch.float32, device="cuda")
    pd = _dev_params(prm, c.dtype)
    xd = dev(x, c.dtype)
    lib.orbit_head_fwd(desc, xd, pd, pred, saved, ws)
    dpred = synth.normal(c.seed, "dpred", (B, L, out))
    dx = torch.empty_like(xd)
    g = {k: torch.full(v.shape, 5.0, dtype=torch.float32, device="cuda") for k, v in prm.items()}
    lib.orbit_head_bwd(desc, xd, pd, saved, dev(dpred, "f32"), dx, g, 0, ws)
    torch.cuda.synchronize()
    ref, cache = O.head_fwd(x, prm, 1, c.eps)
    # the backward products take dpred in the compute dtype; the bias gradient sums it in float32
    rdx, rg = O.head_bwd(synth.bf16_round(dpred), cache, prm)
    rg["b_h"] = O.head_bwd(dpred, cache, prm)[1]["b_h"]
    tol = TOL[c.dtype]
    check("pred", host(pred), ref, tol)
    check("dx", host(dx), rdx, tol)
    for k in rg:
        check(f"d{k}", host(g[k]), rg[k], tol, floor_ref=rg["b_h"])
