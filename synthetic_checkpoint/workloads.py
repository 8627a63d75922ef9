"""The resharding workloads, as plain data (model shapes and parallelism specs).

Each workload names a model shape, a trainer parallelism, a rollout
parallelism and the ranks whose pack and unpack are exercised. These are
inputs, like the synthetic values: the oracle and the library each turn them
into their own layout types.

Full-size workloads use public model shapes (Llama-3-8B, Mixtral-8x7B, the
MoE blocks of DeepSeek-V3). ``scaled`` variants keep the same structure with
small dimensions, for CPU tests and fast parity runs; some dimensions are
deliberately not multiples of the fp8 block or of 16 bytes.
"""

from __future__ import annotations

import copy

TINY = dict(family="dense", num_layers=2, hidden=256, num_heads=4, num_kv_heads=4, head_dim=64, ffn=1024, vocab=1024)
LLAMA3_8B = dict(family="dense", num_layers=32, hidden=4096, num_heads=32, num_kv_heads=8, head_dim=128, ffn=14336,
                 vocab=128256)
MIXTRAL_8X7B = dict(family="mixtral", num_layers=32, hidden=4096, num_heads=32, num_kv_heads=8, head_dim=128,
                    ffn=14336, vocab=32000, num_experts=8)
DSV3_16MOE = dict(family="moe_only", num_layers=16, hidden=7168, ffn=2048, num_experts=256, num_shared_experts=1)

WORKLOADS = {
    "tiny_fsdp2_to_tp2": dict(
        model=TINY,
        trainer=dict(style="fsdp_flat", dtype="f32", fsdp=2),
        rollout=dict(style="serving", dtype="bf16", tp=2),
        pack_rank=0, unpack_rank=1),
    "llama3_8b_fsdp8_to_tp1": dict(
        model=LLAMA3_8B,
        trainer=dict(style="fsdp_flat", dtype="bf16", fsdp=8),
        rollout=dict(style="serving", dtype="bf16", tp=1),
        pack_rank=0, unpack_rank=0),
    "llama3_8b_tp4_to_tp2": dict(
        model=LLAMA3_8B,
        trainer=dict(style="megatron", dtype="bf16", tp=4, transposed_row_parallel=True),
        rollout=dict(style="serving", dtype="bf16", tp=2),
        pack_rank=0, unpack_rank=1),
    "mixtral_ep8fsdp2_to_ep2": dict(
        model=MIXTRAL_8X7B,
        trainer=dict(style="fsdp_flat", dtype="f32", fsdp=2, ep=8),
        rollout=dict(style="serving", dtype="bf16", ep=2),
        pack_rank=0, unpack_rank=0),
    "dsv3_ep64_to_ep8_fp8": dict(
        model=DSV3_16MOE,
        trainer=dict(style="megatron", dtype="bf16", ep=64),
        rollout=dict(style="serving", dtype="bf16", ep=8, quant="f8e4m3", quant_block=128),
        pack_rank=0, unpack_rank=0),
}

ORDER = list(WORKLOADS)

_SCALED_MODELS = {
    "tiny_fsdp2_to_tp2": TINY,
    "llama3_8b_fsdp8_to_tp1": dict(family="dense", num_layers=2, hidden=192, num_heads=8, num_kv_heads=2, head_dim=24,
                                   ffn=344, vocab=1000),
    "llama3_8b_tp4_to_tp2": dict(family="dense", num_layers=2, hidden=200, num_heads=8, num_kv_heads=4, head_dim=20,
                                 ffn=344, vocab=1000),
    "mixtral_ep8fsdp2_to_ep2": dict(family="mixtral", num_layers=2, hidden=96, num_heads=8, num_kv_heads=4,
                                    head_dim=12, ffn=172, vocab=500, num_experts=8),
    "dsv3_ep64_to_ep8_fp8": dict(family="moe_only", num_layers=2, hidden=328, ffn=136, num_experts=32,
                                 num_shared_experts=1),
}
_SCALED_TRAINER = {
    "dsv3_ep64_to_ep8_fp8": dict(style="megatron", dtype="bf16", ep=16),
}
_SCALED_ROLLOUT = {
    "dsv3_ep64_to_ep8_fp8": dict(style="serving", dtype="bf16", ep=4, quant="f8e4m3", quant_block=128),
}


def scaled(name: str) -> dict:
    """Small version of workload ``name``: same styles and dtypes, small shapes."""
    w = copy.deepcopy(WORKLOADS[name])
    w["model"] = dict(_SCALED_MODELS[name])
    if name in _SCALED_TRAINER:
        w["trainer"] = dict(_SCALED_TRAINER[name])
    if name in _SCALED_ROLLOUT:
        w["rollout"] = dict(_SCALED_ROLLOUT[name])
    return w
