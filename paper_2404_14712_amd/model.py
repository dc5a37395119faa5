"""One forward+backward pass of the ViT path through the C ABI.

`ViTPass` owns the device buffers (activations, saved tensors, one shared
workspace, float32 gradients) that a pass needs, allocated with torch, and
enqueues the entry points in order on the current stream:

    full model : orbit_patch_embed -> orbit_var_aggregate -> orbit_vit_block_fwd x n
                 -> orbit_head_fwd -> orbit_mse_loss -> orbit_head_bwd
                 -> orbit_vit_block_bwd x n -> orbit_var_aggregate_bwd -> orbit_patch_embed_bwd
    block stack: orbit_vit_block_fwd x n -> orbit_vit_block_bwd x n (upstream gradient given)
    agg + stack: orbit_var_aggregate -> blocks -> blocks backward -> orbit_var_aggregate_bwd

Only marshalling happens here; every step runs in the HIP library.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import torch

from ._lib import (AggDesc, BlockDesc, EmbedDesc, HeadDesc, ORBIT_BF16, ORBIT_F32, OrbitLib, WmseDesc)


@dataclasses.dataclass
class PassDims:
    mode: str             # "full", "blocks", "agg_blocks"
    dtype: str            # "f32" or "bf16"
    B: int
    L: int
    d: int
    blocks: int
    heads: int
    head_dim: int
    mlp: int
    qk_norm: int = 1
    eps: float = 1e-5
    V: int = 0
    grid: tuple = (0, 0)
    agg_heads: int = 0
    agg_head_dim: int = 0
    final_ln: int = 1
    patch: int = 4
    head_hidden: int = 0  # GELU layers of width d in the prediction head before its last linear map
    loss: str = "mse"     # "mse" or "wmse" (latitude-weighted, Sec. IV)

    @property
    def T(self):
        return self.B * self.L

    @property
    def out(self):
        return self.V * self.patch * self.patch


def torch_dtype(dt: str):
    return torch.bfloat16 if dt == "bf16" else torch.float32


def _code(dt: str) -> int:
    return ORBIT_BF16 if dt == "bf16" else ORBIT_F32


class ViTPass:
    """Device state of one forward+backward pass (see module docstring)."""

    def __init__(self, lib: OrbitLib, dims: PassDims, params: Dict[str, object], device="cuda",
                 checkpoint: bool = False):
        """checkpoint: activation checkpointing of the blocks (Sec. III-B): the
        forward keeps only each block's input and the backward recomputes the
        rest (orbit_vit_block_bwd with saved = NULL)."""
        self.lib, self.z, self.dev = lib, dims, torch.device(device)
        self.checkpoint = checkpoint
        z = dims
        tdt = torch_dtype(z.dtype)
        self.tdt = tdt
        code = _code(z.dtype)
        self.params = params
        self.bdesc = BlockDesc(z.B, z.L, z.d, z.heads, z.head_dim, z.mlp, z.qk_norm, z.eps, code)
        ws = lib.orbit_vit_block_workspace_bytes(self.bdesc)
        if ws == 0:
            raise ValueError(f"invalid block description: {lib.last_error()}")
        sb = lib.orbit_vit_block_saved_bytes(self.bdesc)
        E = lambda *shape, dt=tdt: torch.empty(*shape, dtype=dt, device=self.dev)
        F32 = lambda *shape: torch.zeros(*shape, dtype=torch.float32, device=self.dev)
        self.xs = [E(z.B, z.L, z.d) for _ in range(z.blocks + 1)]
        self.saved = [None if checkpoint else torch.empty(sb, dtype=torch.uint8, device=self.dev)
                      for _ in range(z.blocks)]
        self.dxa = E(z.B, z.L, z.d)
        self.dxb = E(z.B, z.L, z.d)
        self.grads: Dict[str, object] = {"blocks": [
            {k: F32(*v.shape) for k, v in bp.items()} for bp in params["blocks"]]}
        if z.mode in ("full", "agg_blocks"):
            self.adesc = AggDesc(z.B, z.L, z.V, z.d, z.agg_heads, z.agg_head_dim, code)
            ws = max(ws, lib.orbit_var_aggregate_workspace_bytes(self.adesc))
            self.asaved = torch.empty(lib.orbit_var_aggregate_saved_bytes(self.adesc), dtype=torch.uint8,
                                      device=self.dev)
            self.dtok = E(z.B, z.L, z.V, z.d)
            self.grads["agg"] = {k: F32(*v.shape) for k, v in params["agg"].items() if v is not None}
        if z.mode == "full":
            Hg, Wg = z.grid
            self.edesc = EmbedDesc(z.B, z.V, Hg, Wg, z.patch, z.d, code)
            ws = max(ws, lib.orbit_patch_embed_workspace_bytes(self.edesc))
            self.tok = E(z.B, z.L, z.V, z.d)
            self.hdesc = HeadDesc(z.B, z.L, z.d, z.out, z.final_ln, z.eps, code, z.head_hidden)
            ws = max(ws, lib.orbit_head_workspace_bytes(self.hdesc))
            self.hsaved = torch.empty(lib.orbit_head_saved_bytes(self.hdesc), dtype=torch.uint8, device=self.dev)
            self.pred = F32(z.B, z.L, z.out)
            self.dpred = F32(z.B, z.L, z.out)
            self.loss = F32(1)
            n = z.T * z.out
            ws = max(ws, lib.orbit_mse_workspace_bytes(n))
            if z.loss == "wmse":
                self.wdesc = WmseDesc(z.B, z.grid[0], z.grid[1], z.V, z.patch)
                ws = max(ws, lib.orbit_wmse_workspace_bytes(self.wdesc))
            self.grads["embed"] = {k: F32(*v.shape) for k, v in params["embed"].items() if v is not None}
            self.grads["head"] = {k: F32(*v.shape) for k, v in params["head"].items() if v is not None}
        self.ws = torch.empty(ws, dtype=torch.uint8, device=self.dev)

    # ------------------------------------------------------------------------
    def forward_backward(self, inputs: Dict[str, torch.Tensor], accumulate: int = 0, marks=None):
        """inputs: full -> img, tgt; blocks -> x, dy; agg_blocks -> tok, dy.
        Returns the loss tensor (full) or the input gradient. With a list for
        `marks`, appends (phase boundary, recorded timing event) pairs on the
        current stream: blocks_fwd / blocks_fwd_end around the block forwards,
        blocks_bwd / blocks_bwd_end around the block backwards, and agg_fwd /
        agg_fwd_end, agg_bwd / agg_bwd_end around the aggregation calls."""
        z, lib, P, G = self.z, self.lib, self.params, self.grads

        def mark(name):
            if marks is not None:
                e = torch.cuda.Event(enable_timing=True)
                e.record()
                marks.append((name, e))

        if z.mode == "full":
            e = P["embed"]
            lib.orbit_patch_embed(self.edesc, inputs["img"], e["w_pe"], e["b_pe"], e.get("ve"), self.tok)
            mark("agg_fwd")
            lib.orbit_var_aggregate(self.adesc, self.tok, P["agg"], self.xs[0], self.asaved, self.ws)
            mark("agg_fwd_end")
        elif z.mode == "agg_blocks":
            mark("agg_fwd")
            lib.orbit_var_aggregate(self.adesc, inputs["tok"], P["agg"], self.xs[0], self.asaved, self.ws)
            mark("agg_fwd_end")
        else:
            self.xs[0] = inputs["x"]
        mark("blocks_fwd")
        for i in range(z.blocks):
            lib.orbit_vit_block_fwd(self.bdesc, P["blocks"][i], self.xs[i], self.xs[i + 1], self.saved[i], self.ws)
        mark("blocks_fwd_end")
        if z.mode == "full":
            lib.orbit_head_fwd(self.hdesc, self.xs[-1], P["head"], self.pred, self.hsaved, self.ws)
            if z.loss == "wmse":
                lib.orbit_wmse_loss(self.wdesc, self.pred, inputs["tgt"], 1.0, self.loss, self.dpred, self.ws)
            else:
                lib.orbit_mse_loss(self.pred, inputs["tgt"], self.pred.numel(), 1.0, self.loss, self.dpred, self.ws)
            lib.orbit_head_bwd(self.hdesc, self.xs[-1], P["head"], self.hsaved, self.dpred, self.dxa, G["head"],
                               accumulate, self.ws)
            dy = self.dxa
        else:
            dy = inputs["dy"]
        bufs = [self.dxb, self.dxa]
        mark("blocks_bwd")
        for i in range(z.blocks - 1, -1, -1):
            dx = bufs[i % 2] if dy is not bufs[i % 2] else bufs[(i + 1) % 2]
            lib.orbit_vit_block_bwd(self.bdesc, P["blocks"][i], self.xs[i], self.saved[i], dy, dx, G["blocks"][i],
                                    accumulate, self.ws)
            dy = dx
        mark("blocks_bwd_end")
        self.dx = dy
        if z.mode in ("full", "agg_blocks"):
            tok = self.tok if z.mode == "full" else inputs["tok"]
            mark("agg_bwd")
            lib.orbit_var_aggregate_bwd(self.adesc, tok, P["agg"], self.asaved, dy, self.dtok, G["agg"], accumulate,
                                        self.ws)
            mark("agg_bwd_end")
        if z.mode == "full":
            lib.orbit_patch_embed_bwd(self.edesc, inputs["img"], self.dtok, G["embed"]["w_pe"], G["embed"]["b_pe"],
                                      G["embed"].get("ve"), accumulate, self.ws)
            return self.loss
        return self.dx


def block_flops(z: PassDims) -> float:
    """Algorithmic flops of one block forward (products only)."""
    A = z.heads * z.head_dim
    T = z.T
    return 2.0 * T * z.d * 3 * A + 4.0 * z.B * z.heads * z.L * z.L * z.head_dim + 2.0 * T * A * z.d \
        + 4.0 * T * z.d * z.mlp


def recompute_flops(z: PassDims) -> float:
    """Extra algorithmic flops of activation checkpointing per pass: each
    block's forward products again, except the last (fc2)."""
    return (block_flops(z) - 2.0 * z.T * z.mlp * z.d) * z.blocks


def pass_flops(z: PassDims) -> Dict[str, float]:
    """Algorithmic flops of one forward+backward pass (backward = 2x forward
    for every product; recomputation inside the attention backward and the
    exact refolding of the aggregation are not counted as extra work)."""
    out = {"blocks": 3.0 * block_flops(z) * z.blocks}
    T = z.T
    if z.mode in ("full", "agg_blocks"):
        A = z.agg_heads * z.agg_head_dim
        V = z.V
        # folded aggregation: scores + weighted sum over V tokens, value and output projections
        fwd = 2.0 * T * V * z.d * z.agg_heads * 2 + 2.0 * T * z.d * A * 2
        out["aggregation"] = 3.0 * fwd
    if z.mode == "full":
        out["patch_embed"] = 3.0 * 2.0 * T * z.V * 16 * z.d
        out["head"] = 3.0 * 2.0 * T * z.d * (z.out + z.head_hidden * z.d)
    out["total"] = sum(out.values())
    return out
