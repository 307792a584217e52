"""MI355X-native sharded expert-FFN MoE layer (MoEShard, arXiv 2503.08467).

The compute lives in libmoeshard.so (HIP kernels for gfx950, C ABI in
include/moeshard.h); this package only marshals torch tensors into those calls.
"""
from ._lib import LIB_PATH, MoeError, load  # noqa: F401
from .layer import (Dispatch, MoEShardLayer, PackedShard, alloc_dispatch, combine, dispatch,  # noqa: F401
                    dispatch_workspace_size, expert_ffn_shard, expert_ffn_shard_gather,
                    expert_ffn_shard_gather_combine, expert_ffn_shard_noalloc,
                    expert_ffn_shard_per_expert, expert_ffn_shard_top1, ffn_workspace_size, pack_weights,
                    padded_inner_width, route, route_dispatch)
