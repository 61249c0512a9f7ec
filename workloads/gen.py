"""Seeded synthetic inputs shared by the HIP path and the CPU oracle.

Only random draws live here: context lengths, bf16 weights, the KV pool
contents and the decode-step activations. Nothing here computes any step of
the method; every tensor is produced once and handed, unchanged, to both
sides (the oracle gets a host copy).

Recipe (all draws from ``torch.Generator`` seeded by ``sub_seed``):
  * contexts: integer, inclusive range [ctx_lo, ctx_hi], drawn on the host;
    a context counts the token being decoded;
  * projection / FFN / expert weights: N(0, 0.02) rounded to bf16 (RNE);
  * RMSNorm gains: 1 + 0.02 * N(0, 1), rounded to bf16;
  * router weights: N(0, router_std), with router_std = 1/sqrt(hidden) so that
    router logits of a unit-RMS input are close to N(0, 1);
  * KV pool: every element N(0, 1) in bf16, layout-agnostic (the whole pool is
    filled, used pages or not);
  * activations: N(0, 1) in bf16.
Large tensors are drawn on the device that will hold them, so values depend
on (seed, device); both sides always see the same drawn tensor.
"""
from __future__ import annotations

import numpy as np
import torch

from .configs import PAGE_TOKENS, LayerCfg, Workload

_TAGS = {"ctx": 1, "weights": 2, "kv": 3, "x": 4, "live": 5, "misc": 6}


def sub_seed(seed: int, tag: str, *idx: int) -> int:
    """Deterministic 63-bit seed for a (seed, tag, indices...) tuple."""
    h = (seed * 0x100000001B3 + _TAGS[tag] * 0x9E3779B1) & ((1 << 63) - 1)
    for i in idx:
        h = (h * 0x100000001B3 + (i + 1) * 0xC2B2AE35) & ((1 << 63) - 1)
    return h


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=torch.device(device))
    g.manual_seed(seed)
    return g


def normal_bf16(shape, seed: int, device="cpu", std: float = 1.0, mean: float = 0.0) -> torch.Tensor:
    g = _gen(seed, device)
    t = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    if mean != 0.0:
        t.add_(mean)
    return t.to(torch.bfloat16)


def contexts(w: Workload, seed: int | None = None) -> np.ndarray:
    """Per-sequence context lengths (int32, host), uniform integers in [ctx_lo, ctx_hi]."""
    s = w.seed if seed is None else seed
    if w.ctx_lo == w.ctx_hi:
        return np.full(w.batch, w.ctx_lo, dtype=np.int32)
    g = _gen(sub_seed(s, "ctx"), "cpu")
    c = torch.randint(w.ctx_lo, w.ctx_hi + 1, (w.batch,), generator=g, dtype=torch.int64)
    return c.numpy().astype(np.int32)


def pages_needed(ctx_lens) -> int:
    return int(sum(-(-int(c) // PAGE_TOKENS) for c in ctx_lens))


def pool_pages_for(ctx_lens) -> int:
    """Pool size used by every workload: the pages the batch needs plus 25% slack."""
    n = pages_needed(ctx_lens)
    return n + -(-n // 4)


def layer_weights(cfg: LayerCfg, seed: int, layer: int, device="cpu",
                  router_std: float = 1.0 / 64.0) -> dict:
    """bf16 weights of one layer, torch "out x in" row-major layout.

    Dense:  w_gate_up [2F, H] (gate rows first, then up rows), w_down [H, F].
    MoE:    w_router [E, H], w_gate_up [E, 2I, H], w_down [E, H, I].
    Always: g_attn [H], w_qkv [(n_q + 2 n_kv) d, H] (q heads, then k, then v),
            w_o [H, n_q d], g_ffn [H].
    """
    H, d = cfg.hidden, cfg.head_dim
    k = lambda j: sub_seed(seed, "weights", layer, j)
    out = {
        "g_attn": normal_bf16((H,), k(0), device, std=0.02, mean=1.0),
        "w_qkv": normal_bf16((cfg.qkv_dim, H), k(1), device, std=0.02),
        "w_o": normal_bf16((H, cfg.n_q * d), k(2), device, std=0.02),
        "g_ffn": normal_bf16((H,), k(3), device, std=0.02, mean=1.0),
    }
    if cfg.is_moe:
        E, I = cfg.n_experts, cfg.moe_ffn
        out["w_router"] = normal_bf16((E, H), k(4), device, std=router_std)
        out["w_gate_up"] = normal_bf16((E, 2 * I, H), k(5), device, std=0.02)
        out["w_down"] = normal_bf16((E, H, I), k(6), device, std=0.02)
    else:
        F = cfg.ffn
        out["w_gate_up"] = normal_bf16((2 * F, H), k(5), device, std=0.02)
        out["w_down"] = normal_bf16((H, F), k(6), device, std=0.02)
    return out


def kv_pool(cfg: LayerCfg, pool_pages: int, seed: int, layer: int, device="cpu") -> torch.Tensor:
    """One layer's KV pool, bf16 N(0,1) everywhere: shape [P, 2, n_kv, 16 * d]."""
    shape = (pool_pages, 2, cfg.n_kv, PAGE_TOKENS * cfg.head_dim)
    return normal_bf16(shape, sub_seed(seed, "kv", layer), device)


def activations(batch: int, hidden: int, seed: int, device="cpu") -> torch.Tensor:
    """Residual-stream input of the decode step, bf16 N(0,1): [B, H]."""
    return normal_bf16((batch, hidden), sub_seed(seed, "x"), device)


def live_tensor(shape, seed: int, tag: int, device="cpu", std: float = 1.0) -> torch.Tensor:
    """A free-standing bf16 N(0, std) tensor, used to feed a single operator directly."""
    return normal_bf16(shape, sub_seed(seed, "live", tag), device, std=std)


def router_logits(batch: int, n_experts: int, seed: int, device="cpu") -> torch.Tensor:
    """Directly drawn fp32 N(0,1) router logits [B, E] for routing-only checks."""
    g = _gen(sub_seed(seed, "misc", 1), device)
    return torch.randn((batch, n_experts), generator=g, device=device, dtype=torch.float32)


def expert_choices(batch: int, n_experts: int, top_k: int, seed: int) -> np.ndarray:
    """Distinct random expert ids per token (int32 [B, k]), for permute-only checks."""
    g = _gen(sub_seed(seed, "misc", 2), "cpu")
    r = torch.rand((batch, n_experts), generator=g)
    return torch.argsort(r, dim=1)[:, :top_k].numpy().astype(np.int32)
