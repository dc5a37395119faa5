"""The bf16 storage floor of the synthetic models' gradients (CPU, oracle only).

The oracle's `store` hook rounds every intermediate that a bf16 implementation
keeps between two steps (the operands of the matrix products among them) to
bf16, the paper's training precision (Sec. III-B), and leaves the arithmetic in
float64. How far that moves each result from the exact oracle bounds what any
bf16 implementation can reach. On the reduced 115M-structure model these
checks hold:

* every output and gradient moves by less than half the 2e-2 bf16 tolerance,
  except
* the query/key LayerNorm gain and shift gradients of the second block, which
  move by more than 2e-2: the tokens entering that block differ by a few
  percent of their common part (weights at initialisation), so the attention
  pattern is nearly flat and the loss's sensitivity to it, which these
  gradients measure, is small against the perturbation that rounding the
  forward activations causes.

The GPU parity tests compare those gradients at the same bound but as an
expected failure (tests/test_gpu_parity.py, tests/test_gpu_chain.py).
"""
import numpy as np

import oracle as O
import synth

TOL = 2e-2
QKLN = ("qn_g", "qn_b", "kn_g", "kn_b")


def _b16(a):
    return synth.bf16_round(np.asarray(a, np.float32)).astype(np.float64)


def _rel(got, ref, sib):
    ref = np.asarray(ref, np.float64)
    den = np.abs(ref).max()
    if den <= 1e-9 * np.abs(sib).max():
        den = np.abs(sib).max()
    return float(np.abs(np.asarray(got) - ref).max() / den)


def test_bf16_floor_reduced_model():
    c = synth.small_config("115m", B=2, L=128, grid=(32, 64), V=12, d=256, blocks=2, heads=4, head_dim=64, mlp=1024,
                           agg_heads=8, agg_head_dim=32, sigma=0.05)
    args = (synth.image(c), synth.target(c), synth.embed_params(c), synth.agg_params(c),
            [synth.block_params(c, i) for i in range(c.blocks)], synth.head_params(c))
    kw = dict(p=4, agg_heads=c.agg_heads, heads=c.heads, qk_norm=c.qk_norm, eps=c.eps)
    _, pred, ex = O.model_fwd_bwd(*args, **kw)
    _, pred_s, st = O.model_fwd_bwd(*args, store=_b16, **kw)
    floors = {"pred": _rel(pred_s, pred, pred)}
    for grp in ("embed", "agg", "head"):
        sib = ex[grp]["b_q"] if grp == "agg" else None
        for k, v in ex[grp].items():
            floors[f"{grp}.{k}"] = _rel(st[grp][k], v, sib if sib is not None else v)
    for i, gb in enumerate(ex["blocks"]):
        for k, v in gb.items():
            floors[f"block{i}.{k}"] = _rel(st["blocks"][i][k], v, gb["ln1_b"])
    limited = {k: e for k, e in floors.items() if k.startswith("block1.") and k.split(".")[1] in QKLN}
    others = {k: e for k, e in floors.items() if k not in limited}
    worst = max(others, key=others.get)
    assert others[worst] < TOL / 2, (worst, others[worst])
    # the analytically vanishing key-LayerNorm shift gradient aside, the second
    # block's QK-LayerNorm gradients are floor-limited beyond the tolerance
    assert max(limited.values()) > TOL, limited
    print("bf16 storage floor:", {k: f"{e:.2e}" for k, e in sorted(limited.items())},
          f"worst other {worst} {others[worst]:.2e}")
