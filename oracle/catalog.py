"""Checkpoint catalogs: the full-model index space (WeightBridge Sec. 3.1).

The paper uses the full checkpoint as the bridge between trainer and rollout
parameters: every element has one position in it, and a worker's source map
says which checkpoint elements it holds. Here a checkpoint is an ordered list
of tensors of at most two dimensions ([rows, cols]; vectors are [1, n]).
Names and order are the reading taken here (the paper assumes a real checkpoint
and prints none); parity depends only on shapes and order.

Families:
* ``dense``    -- Llama-style decoder: embed, per layer {attn_norm, q, k, v, o,
  mlp_norm, gate, up, down}, final_norm, untied lm_head.
* ``mixtral``  -- dense attention plus, per layer, router and E experts of
  {gate_e, up_e, down_e}.
* ``moe_only`` -- DeepSeek-V3-style MoE blocks only: per layer router, shared
  expert {gate, up, down} and E routed experts of {gate_e, up_e, down_e}.
"""

from __future__ import annotations

from dataclasses import dataclass


@dataclass(frozen=True)
class ModelShapes:
    family: str
    num_layers: int
    hidden: int
    num_heads: int = 0
    num_kv_heads: int = 0
    head_dim: int = 0
    ffn: int = 0
    vocab: int = 0
    num_experts: int = 0
    num_shared_experts: int = 0


@dataclass(frozen=True)
class CkptTensor:
    name: str
    rows: int
    cols: int

    def __post_init__(self):
        # a checkpoint tensor holds at least one element (vectors are [1, n])
        if self.rows < 1 or self.cols < 1:
            raise ValueError(f"checkpoint tensor {self.name!r} needs a positive shape, got {self.rows} x {self.cols}")

    @property
    def numel(self) -> int:
        return self.rows * self.cols


TINY = ModelShapes("dense", num_layers=2, hidden=256, num_heads=4, num_kv_heads=4, head_dim=64, ffn=1024, vocab=1024)
LLAMA3_8B = ModelShapes("dense", num_layers=32, hidden=4096, num_heads=32, num_kv_heads=8, head_dim=128, ffn=14336, vocab=128256)
MIXTRAL_8X7B = ModelShapes("mixtral", num_layers=32, hidden=4096, num_heads=32, num_kv_heads=8, head_dim=128, ffn=14336,
                           vocab=32000, num_experts=8)
DSV3_16MOE = ModelShapes("moe_only", num_layers=16, hidden=7168, ffn=2048, num_experts=256, num_shared_experts=1)


def _attention(m: ModelShapes, p: str):
    h, hd = m.hidden, m.head_dim
    return [
        CkptTensor(p + "attn_norm", 1, h),
        CkptTensor(p + "q", m.num_heads * hd, h),
        CkptTensor(p + "k", m.num_kv_heads * hd, h),
        CkptTensor(p + "v", m.num_kv_heads * hd, h),
        CkptTensor(p + "o", h, m.num_heads * hd),
        CkptTensor(p + "mlp_norm", 1, h),
    ]


def _experts(m: ModelShapes, p: str):
    h, f = m.hidden, m.ffn
    out = []
    for e in range(m.num_experts):
        out += [CkptTensor(f"{p}experts.{e}.gate", f, h), CkptTensor(f"{p}experts.{e}.up", f, h),
                CkptTensor(f"{p}experts.{e}.down", h, f)]
    return out


def checkpoint_catalog(m: ModelShapes) -> list[CkptTensor]:
    """Ordered checkpoint tensors of model ``m``."""
    h = m.hidden
    cat: list[CkptTensor] = []
    if m.family in ("dense", "mixtral"):
        cat.append(CkptTensor("embed", m.vocab, h))
    for layer in range(m.num_layers):
        p = f"layers.{layer}."
        if m.family == "dense":
            cat += _attention(m, p)
            cat += [CkptTensor(p + "gate", m.ffn, h), CkptTensor(p + "up", m.ffn, h), CkptTensor(p + "down", h, m.ffn)]
        elif m.family == "mixtral":
            cat += _attention(m, p)
            cat.append(CkptTensor(p + "router", m.num_experts, h))
            cat += _experts(m, p)
        elif m.family == "moe_only":
            fs = m.ffn * m.num_shared_experts
            cat.append(CkptTensor(p + "router", m.num_experts, h))
            cat += [CkptTensor(p + "shared.gate", fs, h), CkptTensor(p + "shared.up", fs, h),
                    CkptTensor(p + "shared.down", h, fs)]
            cat += _experts(m, p)
        else:
            raise ValueError(f"unknown family {m.family!r}")
    if m.family in ("dense", "mixtral"):
        cat.append(CkptTensor("final_norm", 1, h))
        cat.append(CkptTensor("lm_head", m.vocab, h))
    return cat


def index_of(catalog: list[CkptTensor]) -> dict[str, int]:
    return {t.name: i for i, t in enumerate(catalog)}
