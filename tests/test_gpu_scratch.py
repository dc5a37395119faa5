"""The caller-provided scratch buffers (`ws` and `saved`) are opaque to the
caller: every kernel writes what it later reads. Each component runs its
forward and backward twice, once on scratch filled with 0xFF bytes (a NaN
pattern in both float32 and bf16) and once on zeroed scratch; every output
must be bitwise equal. A kernel that read scratch it had not written (an
accumulation into partials assumed zero, a stale split-K or attention
partial, an unwritten saved tensor) would show NaN on one side only."""
import numpy as np
import pytest

import synth
from helpers import dev

pytestmark = pytest.mark.gpu


def _dev_params(p: dict, dtype: str):
    return {k: (None if v is None else dev(v, dtype)) for k, v in p.items()}


def _scratch(nbytes: int, fill: int):
    import torch
    t = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device="cuda")
    t.fill_(fill)
    return t


def _same(run):
    import torch
    a = run(0xFF)
    b = run(0x00)
    torch.cuda.synchronize()
    assert len(a) == len(b)
    for i, (x, y) in enumerate(zip(a, b)):
        assert not torch.isnan(y.float()).any(), f"output {i}: NaN with zeroed scratch"
        assert torch.equal(x, y), f"output {i} depends on the scratch contents"


# block: qk_norm on and off, a grid that splits the attention sweep (600
# positions, 2 heads of 128) and ragged token counts
BLOCKS = [("bf16", 2, 37, 256, 4, 64, 1024, 1), ("bf16", 1, 600, 256, 2, 128, 512, 1),
          ("bf16", 2, 45, 512, 8, 64, 1024, 0), ("f32", 2, 37, 128, 4, 32, 512, 1)]


@pytest.mark.parametrize("case", BLOCKS)
def test_block_scratch(lib, case):
    import torch
    from paper_2404_14712_amd._lib import BlockDesc
    dtype, B, L, d, H, dh, F, qk = case
    c = synth.small_config("10b-shard", dtype=dtype, B=B, L=L, d=d, heads=H, head_dim=dh, mlp=F, qk_norm=qk,
                           sigma=0.05)
    x = dev(synth.activations(c, "x"), dtype)
    dy = dev(synth.normal(c.seed, "dy", (B, L, d), dtype=dtype), dtype)
    pd = _dev_params(synth.block_params(c, 0), dtype)
    desc = BlockDesc(B, L, d, H, dh, F, qk, 1e-5, 1 if dtype == "bf16" else 0)
    tdt = x.dtype

    def run(fill):
        saved = _scratch(lib.orbit_vit_block_saved_bytes(desc), fill)
        ws = _scratch(lib.orbit_vit_block_workspace_bytes(desc), fill)
        y = torch.zeros(B, L, d, dtype=tdt, device="cuda")
        lib.orbit_vit_block_fwd(desc, pd, x, y, saved, ws)
        dx = torch.zeros(B, L, d, dtype=tdt, device="cuda")
        g = {k: torch.zeros(v.shape, dtype=torch.float32, device="cuda") for k, v in pd.items()}
        lib.orbit_vit_block_bwd(desc, pd, x, saved, dy, dx, g, 0, ws)
        # the activation-checkpoint backward (saved = NULL) on the same scratch
        dx2 = torch.zeros(B, L, d, dtype=tdt, device="cuda")
        g2 = {k: torch.zeros(v.shape, dtype=torch.float32, device="cuda") for k, v in pd.items()}
        lib.orbit_vit_block_bwd(desc, pd, x, None, dy, dx2, g2, 0, ws)
        return [y, dx, dx2] + [g[k] for k in sorted(g)] + [g2[k] for k in sorted(g2)]

    _same(run)


@pytest.mark.parametrize("case", [("bf16", 1, 70, 91, 512, 8, 64), ("bf16", 2, 37, 20, 512, 8, 128),
                                  ("f32", 2, 37, 4, 128, 4, 32)])
def test_var_aggregate_scratch(lib, case):
    import torch
    from paper_2404_14712_amd._lib import AggDesc
    dtype, B, L, V, d, H, dh = case
    c = synth.small_config("115m", dtype=dtype, B=B, L=L, V=V, d=d, agg_heads=H, agg_head_dim=dh, sigma=0.2)
    tok = dev(synth.normal(c.seed, "tok", (B, L, V, d), dtype=dtype), dtype)
    pd = _dev_params(synth.make_params(c.seed, "agg", synth.agg_param_shapes(d, H * dh, L), 0.2, dtype), dtype)
    dz = dev(synth.normal(c.seed, "dz", (B, L, d), dtype=dtype), dtype)
    desc = AggDesc(B, L, V, d, H, dh, 1 if dtype == "bf16" else 0)

    def run(fill):
        saved = _scratch(lib.orbit_var_aggregate_saved_bytes(desc), fill)
        ws = _scratch(lib.orbit_var_aggregate_workspace_bytes(desc), fill)
        z = torch.zeros(B, L, d, dtype=tok.dtype, device="cuda")
        lib.orbit_var_aggregate(desc, tok, pd, z, saved, ws)
        dtok = torch.zeros(B, L, V, d, dtype=tok.dtype, device="cuda")
        g = {k: torch.zeros(v.shape, dtype=torch.float32, device="cuda") for k, v in pd.items()}
        lib.orbit_var_aggregate_bwd(desc, tok, pd, saved, dz, dtok, g, 0, ws)
        return [z, dtok] + [g[k] for k in sorted(g)]

    _same(run)


@pytest.mark.parametrize("dtype,hidden", [("bf16", 1), ("bf16", 0), ("f32", 1)])
def test_head_scratch(lib, dtype, hidden):
    import torch
    from paper_2404_14712_amd._lib import HeadDesc
    B, L, d, out = 2, 37, 256, 64
    c = synth.small_config("tiny", dtype=dtype, B=B, L=L, d=d, V=out // 16, sigma=0.05)
    x = dev(synth.activations(c, "x"), dtype)
    prm = synth.head_params(c, hidden)
    if hidden:
        prm["w_hid"] = synth.normal(c.seed, "head.w_hid.unit", prm["w_hid"].shape, std=1.0 / np.sqrt(d), dtype=dtype)
    pd = _dev_params(prm, dtype)
    dpred = dev(synth.normal(c.seed, "dpred", (B, L, out)), "f32")
    desc = HeadDesc(B, L, d, out, 1, 1e-5, 1 if dtype == "bf16" else 0, hidden)

    def run(fill):
        saved = _scratch(lib.orbit_head_saved_bytes(desc), fill)
        ws = _scratch(lib.orbit_head_workspace_bytes(desc), fill)
        pred = torch.zeros(B, L, out, dtype=torch.float32, device="cuda")
        lib.orbit_head_fwd(desc, x, pd, pred, saved, ws)
        dx = torch.zeros_like(x)
        g = {k: torch.zeros(v.shape, dtype=torch.float32, device="cuda") for k, v in pd.items()}
        lib.orbit_head_bwd(desc, x, pd, saved, dpred, dx, g, 0, ws)
        return [pred, dx] + [g[k] for k in sorted(g)]

    _same(run)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_patch_embed_scratch(lib, dtype):
    import torch
    from paper_2404_14712_amd._lib import EmbedDesc
    B, V, Hg, Wg, d = 2, 5, 16, 16, 1032
    c = synth.small_config("tiny", dtype=dtype, B=B, V=V, grid=(Hg, Wg), d=d, L=(Hg // 4) * (Wg // 4))
    img = dev(synth.image(c), "f32")
    pd = _dev_params(synth.embed_params(c), dtype)
    dtok = dev(synth.normal(c.seed, "dtok", (B, c.L, V, d), dtype=dtype), dtype)
    desc = EmbedDesc(B, V, Hg, Wg, 4, d, 1 if dtype == "bf16" else 0)

    def run(fill):
        ws = _scratch(lib.orbit_patch_embed_workspace_bytes(desc), fill)
        tok = torch.zeros(B, c.L, V, d, dtype=dtok.dtype, device="cuda")
        lib.orbit_patch_embed(desc, img, pd["w_pe"], pd["b_pe"], pd["ve"], tok)
        g = {k: torch.zeros(v.shape, dtype=torch.float32, device="cuda") for k, v in pd.items()}
        lib.orbit_patch_embed_bwd(desc, img, dtok, g["w_pe"], g["b_pe"], g["ve"], 0, ws)
        return [tok] + [g[k] for k in sorted(g)]

    _same(run)
