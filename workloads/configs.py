"""Layer shapes and decode-batch recipes of the five evaluated workloads.

Pure data: no arithmetic of the method lives here. Both the HIP path and the
CPU oracle receive tensors built from these descriptions by ``workloads.gen``.

The paper models one decode step as an ordered operator sequence and groups
layers into a repeating partition block (Appendix B.1, "Model Representation
and Partition"); a ``Workload`` is one such block plus the batch it serves.
The shapes themselves (hidden size, heads, FFN width, context mix) are
synthetic stand-ins chosen to resemble the dense 8B-class and MoE decoders the
paper's evaluation serves (Section 7 and Table 2); the paper's own context
distribution comes from a public reasoning-trace corpus that is not available
here, and uniform integer context ranges stand in for it.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Tuple

PAGE_TOKENS = 16  # tokens per KV page


@dataclass(frozen=True)
class LayerCfg:
    hidden: int
    n_q: int
    n_kv: int
    head_dim: int
    ffn: int = 0            # dense SwiGLU intermediate width (0 for MoE layers)
    n_experts: int = 0      # 0 -> dense layer
    top_k: int = 0
    moe_ffn: int = 0        # per-expert SwiGLU intermediate width
    window: int = 0         # sliding-window length in tokens, 0 -> full attention
    rope_theta: float = 10000.0
    rms_eps: float = 1e-6

    @property
    def is_moe(self) -> bool:
        return self.n_experts > 0

    @property
    def qkv_dim(self) -> int:
        return (self.n_q + 2 * self.n_kv) * self.head_dim

    @property
    def n_ops(self) -> int:
        return 14 if self.is_moe else 10


@dataclass(frozen=True)
class Workload:
    name: str
    layers: Tuple[LayerCfg, ...]
    batch: int
    ctx_lo: int             # inclusive; counts the token being decoded
    ctx_hi: int             # inclusive
    seed: int = 0
    # scale of the router weights (only used by MoE layers); see gen.layer_weights
    router_std: float = 1.0 / 64.0
    description: str = ""

    @property
    def n_ops(self) -> int:
        return sum(l.n_ops for l in self.layers)

    @property
    def max_pages(self) -> int:
        return -(-self.ctx_hi // PAGE_TOKENS)


_DENSE_8B = LayerCfg(hidden=4096, n_q=32, n_kv=8, head_dim=128, ffn=14336)

TINY = Workload(
    name="tiny",
    layers=(LayerCfg(hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=688),),
    batch=4, ctx_lo=128, ctx_hi=128,
    description="single tiny decoder layer, hidden 256, 4q/2kv heads of 64, SwiGLU 688, "
                "batch 4 x 128 tokens, full attention",
)

DENSE_8B_B64 = Workload(
    name="dense8b_b64",
    layers=(_DENSE_8B,),
    batch=64, ctx_lo=512, ctx_hi=4096,
    description="8B-shaped dense layer (hidden 4096, 32q/8kv x 128, SwiGLU 14336), "
                "batch 64, context U[512,4096], shuffled pages",
)

DENSE_8B_B256 = Workload(
    name="dense8b_b256_ctx8k",
    layers=(_DENSE_8B,),
    batch=256, ctx_lo=8192, ctx_hi=8192,
    description="8B-shaped dense layer, batch 256, every context 8192 tokens (2M cached tokens)",
)

HYBRID_4L = Workload(
    name="hybrid4_b128",
    layers=(replace(_DENSE_8B, window=1024),) * 3 + (_DENSE_8B,),
    batch=128, ctx_lo=1024, ctx_hi=32768,
    description="4-layer hybrid block: 3 sliding-window layers (window 1024) then 1 full layer, "
                "batch 128, context U[1024,32768]",
)

MOE_B512 = Workload(
    name="moe64x8_b512",
    layers=(LayerCfg(hidden=4096, n_q=32, n_kv=4, head_dim=128,
                     n_experts=64, top_k=8, moe_ffn=1536),),
    batch=512, ctx_lo=2048, ctx_hi=16384,
    description="MoE layer: hidden 4096, 32q/4kv x 128, 64 experts top-8 (SwiGLU 1536), "
                "batch 512, context U[2048,16384]",
)

ALL = (TINY, DENSE_8B_B64, DENSE_8B_B256, HYBRID_4L, MOE_B512)

# One GPU's share of the batch-256 x 8192 dense layer when the layer is split
# 8 ways by tensor parallelism: attention by KV head (one KV head with its four
# query heads, the matching slices of W_qkv and W_o), the SwiGLU FFN by
# intermediate columns (1792 of 14336), the residual stream replicated. Its
# o_proj and down products are the partial sums an all-reduce would complete;
# here they go straight into the residual (the same work per GPU), and the
# same kernels run at exactly this shape.
DENSE_8B_B256_TP8 = Workload(
    name="dense8b_b256_ctx8k_tp8",
    layers=(LayerCfg(hidden=4096, n_q=4, n_kv=1, head_dim=128, ffn=1792),),
    batch=256, ctx_lo=8192, ctx_hi=8192,
    description="one GPU's share of the batch-256 x 8192 8B-shaped layer under 8-way tensor "
                "parallelism: hidden 4096, 4q/1kv x 128, SwiGLU 1792",
)

SHARES = (DENSE_8B_B256_TP8,)
BY_NAME = {w.name: w for w in ALL + SHARES}


def shrink(w: Workload, **kw) -> Workload:
    """A copy of ``w`` with some fields replaced (reduced shapes for quick parity runs)."""
    return replace(w, **kw)
