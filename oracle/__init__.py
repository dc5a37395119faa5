"""fp64 CPU oracle of the ORBIT ViT hot path — test infrastructure only.

Imported only by tests/, __graft_entry__.smoke() and bench.py's cpu_baseline
leg. The product path (paper_2404_14712_amd) never imports it.
"""
from .orbit_oracle import *  # noqa: F401,F403
from .orbit_oracle import (agg_bwd, agg_fwd, attention_bwd, attention_fwd, block_bwd,
                           block_fwd, gelu, gelu_grad, head_bwd, head_fwd, layer_norm_bwd,
                           layer_norm_fwd, model_fwd_bwd, mse, patch_embed_bwd,
                           patch_embed_fwd, patchify, shard_block_params, softmax)
