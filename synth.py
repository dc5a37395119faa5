"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the bench.

This module holds shapes and random numbers only: it performs none of the
model's arithmetic. Both the fp64 oracle and the HIP path receive exactly the
arrays produced here (in bf16 mode: values already rounded to bf16 with
round-to-nearest-even, carried as float32 on the host).

The workloads stand in for the paper's CMIP6 / ERA5 observations (Sec. IV:
128x256 grid per variable, 48 or 91 variables), which are not available:
i.i.d. normal fields per variable reproduce the shapes and the unit dynamic
range of normalised climate variables.

Seeding: every tensor has a name; its generator is
``numpy.random.Generator(PCG64(SeedSequence([240414712, seed, crc32(name)])))``,
so any tensor can be regenerated alone, in any order.
"""
from __future__ import annotations

import dataclasses
import zlib
from typing import Dict

import numpy as np

BASE_SEED = 240414712
PATCH = 4


@dataclasses.dataclass(frozen=True)
class Config:
    """One workload. ``heads``/``mlp``/``attn_dim`` are the LOCAL (per-GPU) sizes."""
    seed: int             # seed stream of the workload's tensors
    name: str
    dtype: str            # "f32" or "bf16"
    B: int
    L: int                # tokens per sample
    d: int                # embedding width
    blocks: int
    heads: int            # local self-attention heads
    head_dim: int
    mlp: int              # local MLP width F
    sigma: float
    V: int = 0            # variables (0: no patch embed / aggregation)
    grid: tuple = (0, 0)  # (Hg, Wg); (0, 0): no patch embed
    agg_heads: int = 0
    agg_head_dim: int = 0
    full_model: bool = False   # patch embed + aggregation + blocks + head + MSE
    agg_only_prefix: bool = False  # aggregation from a given token tensor, then blocks
    var_scale: bool = False    # per-variable input scale U(0.5, 2)
    qk_norm: int = 1
    eps: float = 1e-5

    @property
    def T(self) -> int:
        return self.B * self.L

    @property
    def A(self) -> int:
        return self.heads * self.head_dim

    @property
    def agg_A(self) -> int:
        return self.agg_heads * self.agg_head_dim

    @property
    def out_dim(self) -> int:
        return self.V * PATCH * PATCH


CONFIGS: Dict[str, Config] = {
    "tiny": Config(1, "tiny ClimaX-style ViT, fp32", "f32", B=2, L=128, d=128, blocks=2,
              heads=4, head_dim=32, mlp=512, sigma=0.02, V=4, grid=(32, 64),
              agg_heads=4, agg_head_dim=32, full_model=True),
    "115m": Config(2, "115M-scale ViT (d=1024, 8 blocks, V=48)", "bf16", B=4, L=2048, d=1024,
              blocks=8, heads=16, head_dim=64, mlp=4096, sigma=0.02, V=48,
              grid=(128, 256), agg_heads=16, agg_head_dim=64, full_model=True),
    "1b": Config(3, "1B-scale ViT (d=2048, 16 blocks, V=91)", "bf16", B=2, L=2048, d=2048,
              blocks=16, heads=16, head_dim=128, mlp=8192, sigma=0.02, V=91,
              grid=(128, 256), agg_heads=16, agg_head_dim=128, full_model=True,
              var_scale=True),
    "10b-shard": Config(4, "10B-scale tensor-parallel shard (d=8192, TP 8), 4 blocks", "bf16", B=2,
              L=2048, d=8192, blocks=4, heads=8, head_dim=128, mlp=4096, sigma=0.01),
    "113b-shard": Config(5, "113B-scale tensor-parallel shard (d=16384, TP 16), aggregation + 2 blocks",
              "bf16", B=1, L=2048, d=16384, blocks=2, heads=8, head_dim=128, mlp=4096,
              sigma=0.005, V=91, agg_heads=8, agg_head_dim=128, agg_only_prefix=True),
    # the paper's own widths (Sec. IV) under tensor parallelism over the 8 GPUs
    # of a node (the paper's best 113B layout, Sec. V-C, is FSDP x TP 8)
    "10b-paper-tp8": Config(6, "10B model's tensor-parallel shard at the paper's widths (d=8192, 4 of 32 heads of 256, TP 8), "
                 "4 blocks", "bf16", B=2, L=2048, d=8192, blocks=4, heads=4, head_dim=256, mlp=4096, sigma=0.01),
    "113b-paper-tp8": Config(7, "113B model's tensor-parallel shard at the paper's widths (d=12288, 8 of 64 heads of 192, TP 8), "
                 "2 blocks", "bf16", B=1, L=2048, d=12288, blocks=2, heads=8, head_dim=192, mlp=6144,
              sigma=0.005),
}


def rng(seed: int, name: str) -> np.random.Generator:
    ss = np.random.SeedSequence([BASE_SEED, int(seed), zlib.crc32(name.encode())])
    return np.random.Generator(np.random.PCG64(ss))


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); returns float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return (u.astype(np.uint32) << 16).view(np.float32)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) of float32 values that are already bf16-exact."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    return (a.view(np.uint32) >> 16).astype(np.uint16)


def _cast(a: np.ndarray, dtype: str) -> np.ndarray:
    a = a.astype(np.float32)
    return bf16_round(a) if dtype == "bf16" else a


def normal(seed: int, name: str, shape, std: float = 1.0, mean: float = 0.0,
           dtype: str = "f32") -> np.ndarray:
    g = rng(seed, name)
    a = g.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    if mean != 0.0:
        a += np.float32(mean)
    return _cast(a, dtype)


# ---------------------------------------------------------------------------
# parameter sets (names match the C-ABI parameter structs)
# ---------------------------------------------------------------------------

BLOCK_PARAM_NAMES = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "qn_g", "qn_b", "kn_g", "kn_b",
                     "w_proj", "b_proj", "ln2_g", "ln2_b", "w_fc1", "b_fc1", "w_fc2", "b_fc2")
AGG_PARAM_NAMES = ("q0", "w_q", "b_q", "w_k", "b_k", "w_v", "b_v", "w_o", "b_o", "pos")
EMBED_PARAM_NAMES = ("w_pe", "b_pe", "ve")
HEAD_PARAM_NAMES = ("lnf_g", "lnf_b", "w_h", "b_h")


def block_param_shapes(d: int, A: int, F: int, dh: int) -> Dict[str, tuple]:
    return {
        "ln1_g": (d,), "ln1_b": (d,),
        "w_qkv": (d, 3 * A), "b_qkv": (3 * A,),
        "qn_g": (dh,), "qn_b": (dh,), "kn_g": (dh,), "kn_b": (dh,),
        "w_proj": (A, d), "b_proj": (d,),
        "ln2_g": (d,), "ln2_b": (d,),
        "w_fc1": (d, F), "b_fc1": (F,),
        "w_fc2": (F, d), "b_fc2": (d,),
    }


def agg_param_shapes(d: int, A: int, L: int) -> Dict[str, tuple]:
    return {"q0": (d,), "w_q": (d, A), "b_q": (A,), "w_k": (d, A), "b_k": (A,),
            "w_v": (d, A), "b_v": (A,), "w_o": (A, d), "b_o": (d,), "pos": (L, d)}


def embed_param_shapes(V: int, d: int, p: int = PATCH) -> Dict[str, tuple]:
    return {"w_pe": (V, p * p, d), "b_pe": (V, d), "ve": (V, d)}


def head_param_shapes(d: int, out: int, hidden: int = 0) -> Dict[str, tuple]:
    s = {"lnf_g": (d,), "lnf_b": (d,), "w_h": (d, out), "b_h": (out,)}
    if hidden:
        s.update({"w_hid": (hidden, d, d), "b_hid": (hidden, d)})
    return s


def _is_ln_gain(name: str) -> bool:
    return name.endswith("_g")


def make_params(seed: int, prefix: str, shapes: Dict[str, tuple], sigma: float,
                dtype: str) -> Dict[str, np.ndarray]:
    """Every matrix, bias, embedding and the query ~ N(0, sigma);
    LayerNorm gains ~ 1 + N(0, sigma) and shifts ~ N(0, sigma)."""
    out = {}
    for name, shape in shapes.items():
        full = f"{prefix}.{name}"
        if _is_ln_gain(name):
            out[name] = normal(seed, full, shape, std=sigma, mean=1.0, dtype=dtype)
        else:
            out[name] = normal(seed, full, shape, std=sigma, dtype=dtype)
    return out


def block_params(c: Config, i: int, d=None, A=None, F=None, dh=None) -> Dict[str, np.ndarray]:
    d = c.d if d is None else d
    A = c.A if A is None else A
    F = c.mlp if F is None else F
    dh = c.head_dim if dh is None else dh
    return make_params(c.seed, f"block{i}", block_param_shapes(d, A, F, dh), c.sigma, c.dtype)


def agg_params(c: Config) -> Dict[str, np.ndarray]:
    return make_params(c.seed, "agg", agg_param_shapes(c.d, c.agg_A, c.L), c.sigma, c.dtype)


def embed_params(c: Config) -> Dict[str, np.ndarray]:
    return make_params(c.seed, "embed", embed_param_shapes(c.V, c.d), c.sigma, c.dtype)


def head_params(c: Config, hidden: int = 0) -> Dict[str, np.ndarray]:
    return make_params(c.seed, "head", head_param_shapes(c.d, c.out_dim, hidden), c.sigma, c.dtype)


def image(c: Config) -> np.ndarray:
    """img[B, V, Hg, Wg] float32; with var_scale, a per-variable scale s_v ~ U(0.5, 2)."""
    Hg, Wg = c.grid
    img = normal(c.seed, "img", (c.B, c.V, Hg, Wg))
    if c.var_scale:
        s = rng(c.seed, "img.var_scale").uniform(0.5, 2.0, size=c.V).astype(np.float32)
        img *= s[None, :, None, None]
    return img


def target(c: Config) -> np.ndarray:
    """tgt[B, L, V*p*p] float32, token layout."""
    return normal(c.seed, "tgt", (c.B, c.L, c.out_dim))


def activations(c: Config, name: str = "x") -> np.ndarray:
    """x[B, L, d] ~ N(0, 1) in the config's dtype."""
    return normal(c.seed, name, (c.B, c.L, c.d), dtype=c.dtype)


def tokens_chunk(c: Config, b: int, l0: int, l1: int) -> np.ndarray:
    """tok[b, l0:l1, V, d] ~ N(0,1) for the aggregation-prefixed shard workload.

    Generated per 64-patch chunk so any patch range can be regenerated alone."""
    CH = 64
    out = np.empty((l1 - l0, c.V, c.d), np.float32)
    for ch in range(l0 // CH, (l1 + CH - 1) // CH):
        a, bnd = ch * CH, min((ch + 1) * CH, c.L)
        blk = normal(c.seed, f"tok.b{b}.c{ch}", (bnd - a, c.V, c.d), dtype=c.dtype)
        s0, s1 = max(a, l0), min(bnd, l1)
        out[s0 - l0:s1 - l0] = blk[s0 - a:s1 - a]
    return out


def small_config(workload: str, **over) -> Config:
    """A copy of a config with some sizes replaced (parity cases that the oracle
    finishes in seconds)."""
    return dataclasses.replace(CONFIGS[workload], **over)


def device_normal(seed: int, name: str, shape, dtype: str, device, chunk_rows: int = 0):
    """N(0, 1) tensor drawn on the device by torch's seeded generator, for
    inputs too large to draw on the host (full-size token and activation
    tensors). Drawn in float32 and rounded to the dtype. With ``chunk_rows``,
    the leading axis is drawn in slabs of that many rows (bounds the float32
    temporary). Deterministic for a given device type and torch version."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed((BASE_SEED * 1000 + int(seed) * 7919 + zlib.crc32(name.encode())) % (2 ** 63))
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    out = torch.empty(*shape, dtype=tdt, device=device)
    n0 = shape[0]
    step = chunk_rows if chunk_rows > 0 else n0
    for a in range(0, n0, step):
        b = min(n0, a + step)
        out[a:b] = torch.randn(b - a, *shape[1:], generator=gen, device=device, dtype=torch.float32).to(tdt)
    return out
