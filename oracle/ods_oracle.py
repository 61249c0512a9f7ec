"""CPU oracle of the operator-level-disaggregated decode step.

TEST INFRASTRUCTURE ONLY. Nothing on the product path may import, call or
execute this module: only the tests, the smoke check and the benchmark's CPU
baseline leg use it. It shares no code with the HIP library and never reads a
value the HIP library produced.

What it computes. The paper models one decode step as a fixed, ordered
sequence of kernels o_1..o_N (Appendix A.1) and a serving stage as a
contiguous slice of that sequence inside a repeating partition block
(Section 4, "Partition-block abstraction"; Appendix B.1). This module executes
any slice [op_begin, op_end) of a block's operator sequence, one plain step per
operator, in float64, with no paging tricks beyond a page-table gather, no
fusion and no splitting. Intermediates are never rounded, so running [a, c)
then [c, b) is bit-identical to running [a, b).

The paper does not define the numerics of the layer's operators (it treats
each o_i as an opaque kernel with bytes D_i(b) and flops W_i(b)). The readings
used here, each a textbook definition, are:
  * RMSNorm: x * (mean(x^2) + eps)^(-1/2) * gain;
  * RoPE: rotate-half pairing (i, i + d/2), angle p * theta^(-2i/d), p = ctx - 1;
  * attention: softmax(q K^T / sqrt(d)) V over the window [p - W + 1, p]
    (W = 0: the whole context), GQA head h reads KV head h // (n_q / n_kv);
  * SwiGLU: silu(gate) * up, silu(z) = z / (1 + exp(-z));
  * routing: softmax over all experts, top-k by probability (ties to the lower
    expert index), renormalised over the k chosen;
  * expert permutation: stable sort of (token, slot) pairs by expert id.
Parity of these conventions is pinned only by mathematical invariants and
closed forms (see tests/test_oracle.py); the paper prints no worked example.

Page allocator (splitmix64 + Fisher-Yates) and KV page layout follow the
library's documented contract; see ``kv_alloc`` and ``page_kv``.
"""
from __future__ import annotations

import math

import numpy as np

PAGE = 16
M64 = (1 << 64) - 1

DENSE_OPS = ("attn_norm", "qkv_proj", "rope", "kv_append", "attn_core", "o_proj_residual",
             "ffn_norm", "gate_up", "silu_mul", "down_residual")
MOE_OPS = DENSE_OPS[:7] + ("router", "topk_softmax", "moe_permute", "expert_gate_up",
                           "silu_mul", "expert_down", "moe_combine_residual")


def layer_ops(cfg):
    return MOE_OPS if cfg.n_experts > 0 else DENSE_OPS


# ----------------------------------------------------------------------------
# KV page allocation (setup step, integer, must agree bit-for-bit)
# ----------------------------------------------------------------------------

def splitmix64(state: int):
    """One step of Vigna's splitmix64: returns (new_state, output)."""
    state = (state + 0x9E3779B97F4A7C15) & M64
    z = state
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return state, z ^ (z >> 31)


def page_permutation(pool_pages: int, seed: int):
    """Fisher-Yates shuffle of [0, P), drawing j = next() mod (i + 1) for i = P-1 .. 1."""
    perm = list(range(pool_pages))
    state = seed & M64
    for i in range(pool_pages - 1, 0, -1):
        state, r = splitmix64(state)
        j = r % (i + 1)
        perm[i], perm[j] = perm[j], perm[i]
    return perm


def kv_alloc(ctx_lens, pool_pages: int, seed: int, max_pages: int) -> np.ndarray:
    """Page table [B, max_pages] (int32, -1 = unused): sequence b takes the next
    ceil(ctx_b / 16) entries of the shuffled page list, in batch order."""
    need = [-(-int(c) // PAGE) for c in ctx_lens]
    if sum(need) > pool_pages:
        raise MemoryError("pool too small")
    if any(n > max_pages for n in need):
        raise ValueError("context longer than the page table row")
    perm = page_permutation(pool_pages, seed)
    table = np.full((len(need), max_pages), -1, dtype=np.int32)
    off = 0
    for b, n in enumerate(need):
        table[b, :n] = perm[off:off + n]
        off += n
    return table


# ----------------------------------------------------------------------------
# KV page layout. Pool shape [P, 2, n_kv, 16 * d]: block (page, 0, g) holds the
# keys of 16 token slots row by row (slot t, dim i at t * d + i); block
# (page, 1, g) holds the values dim-major (dim i, slot t at i * 16 + t).
# ----------------------------------------------------------------------------

def page_kv(pool: np.ndarray, page_row, n_tokens: int, n_kv: int, d: int, first: int = 0):
    """Keys and values of token positions [first, n_tokens) of one sequence:
    K, V each [n_kv, n_tokens - first, d] float64. Only the pages holding
    those positions are read."""
    p0 = first // PAGE
    n_pages = -(-n_tokens // PAGE) - p0
    pages = np.asarray(page_row[p0:p0 + n_pages], dtype=np.int64)
    blk = np.asarray(pool[pages], dtype=np.float64)            # [np, 2, n_kv, 16 d]
    K = blk[:, 0].reshape(n_pages, n_kv, PAGE, d).transpose(1, 0, 2, 3)
    V = blk[:, 1].reshape(n_pages, n_kv, d, PAGE).transpose(1, 0, 3, 2)
    t0 = first - p0 * PAGE
    K = K.reshape(n_kv, n_pages * PAGE, d)[:, t0:t0 + n_tokens - first]
    V = V.reshape(n_kv, n_pages * PAGE, d)[:, t0:t0 + n_tokens - first]
    return K, V


def write_kv_slot(pool: np.ndarray, page: int, slot: int, k: np.ndarray, v: np.ndarray, d: int):
    """Store one token's k, v ([n_kv, d]) at (page, slot) of a float64 pool."""
    n_kv = k.shape[0]
    for g in range(n_kv):
        pool[page, 0, g, slot * d:(slot + 1) * d] = k[g]
        pool[page, 1, g, slot::PAGE][:d] = v[g]


# ----------------------------------------------------------------------------
# Operators (one decode step of one layer, rows independent except routing
# bookkeeping). Inputs are float64 arrays holding the bf16 input values.
# ----------------------------------------------------------------------------

def rmsnorm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """x * (mean over the row of x^2 + eps)^(-1/2) * gain."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gain


def linear(x: np.ndarray, w: np.ndarray) -> np.ndarray:
    """x @ w^T with w stored [out, in]."""
    return x @ w.T


def rope_rotate(u: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half RoPE of head vectors u [B, n_heads, d] at positions pos [B]."""
    d = u.shape[-1]
    half = d // 2
    inv = theta ** (-2.0 * np.arange(half, dtype=np.float64) / d)          # [half]
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]       # [B, half]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    a, b = u[..., :half], u[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def attention_row(q: np.ndarray, K: np.ndarray, V: np.ndarray, lo: int, hi: int) -> np.ndarray:
    """Decode attention of one sequence. q [n_q, d]; K, V [n_kv, n, d]; keys
    [lo, hi] inclusive. Returns o [n_q, d]."""
    n_q, d = q.shape
    n_kv = K.shape[0]
    group = n_q // n_kv
    o = np.empty((n_q, d))
    for h in range(n_q):
        g = h // group
        s = K[g, lo:hi + 1] @ q[h] / math.sqrt(d)
        w = np.exp(s - s.max())
        w = w / w.sum()
        o[h] = w @ V[g, lo:hi + 1]
    return o


def window_start(p: int, window: int) -> int:
    return max(0, p - window + 1) if window > 0 else 0


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def route_weights(logits: np.ndarray, ids: np.ndarray) -> np.ndarray:
    """Routing weights of a given expert choice: the softmax probabilities of
    the chosen experts renormalised over them ([B, k] float64). topk_route
    applies the same formula to its own choice."""
    out = np.empty(np.shape(ids))
    for b in range(out.shape[0]):
        z = np.asarray(logits[b], dtype=np.float64)
        p = np.exp(z - z.max())
        p = p / p.sum()
        chosen = p[np.asarray(ids[b], dtype=np.int64)]
        out[b] = chosen / chosen.sum()
    return out


def topk_route(logits: np.ndarray, k: int):
    """Softmax over all experts, top-k by probability with ties to the lower
    index, weights renormalised over the chosen k. Returns (ids int32 [B,k],
    weights float64 [B,k])."""
    B, E = logits.shape
    ids = np.empty((B, k), dtype=np.int32)
    wts = np.empty((B, k))
    for b in range(B):
        z = np.asarray(logits[b], dtype=np.float64)
        p = np.exp(z - z.max())
        p = p / p.sum()
        order = sorted(range(E), key=lambda e: (-p[e], e))[:k]
        ids[b] = order
        wts[b] = p[order] / p[order].sum()
    return ids, wts


def moe_permute(ids: np.ndarray, n_experts: int):
    """Stable sort of the (token, slot) pairs, flattened as token * k + slot,
    by expert id. Returns perm [B*k] (sorted position -> pair), expert_off
    [E+1] and slot_pos [B*k] (pair -> sorted position)."""
    flat = np.asarray(ids, dtype=np.int64).reshape(-1)
    perm = np.argsort(flat, kind="stable").astype(np.int32)
    counts = np.bincount(flat, minlength=n_experts)
    expert_off = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    slot_pos = np.empty_like(perm)
    slot_pos[perm] = np.arange(perm.size, dtype=np.int32)
    return perm, expert_off, slot_pos


# ----------------------------------------------------------------------------
# Stage execution over an operator range of a partition block
# ----------------------------------------------------------------------------

def block_op_list(cfgs):
    """[(layer, local_index, name)] for every operator of the block, in order."""
    out = []
    for l, cfg in enumerate(cfgs):
        for j, name in enumerate(layer_ops(cfg)):
            out.append((l, j, name))
    return out


def run_ops(cfgs, weights, pools, page_table, ctx_lens, live: dict, op_begin: int, op_end: int) -> dict:
    """Execute operators [op_begin, op_end) of the block on the live set.

    cfgs: per-layer configs; weights: per-layer dicts of float64 arrays (same
    names and layouts as the library's weights); pools: per-layer float64 KV
    pools [P, 2, n_kv, 16 d] (updated in place by kv_append); page_table
    [B, max_pages] int, or a list with one such table per layer (each indexing
    that layer's pool); ctx_lens [B]; live: dict of float64/int arrays keyed by
    live-buffer name (updated and returned). A sliding-window layer reads only
    the pages of its window, so its table may leave the others at -1.
    """
    ops = block_op_list(cfgs)
    if not (0 <= op_begin < op_end <= len(ops)):
        raise ValueError("bad operator range")
    ctx = np.asarray(ctx_lens, dtype=np.int64)
    pos = ctx - 1
    B = ctx.shape[0]
    for (l, _, name) in ops[op_begin:op_end]:
        cfg, w, pool = cfgs[l], weights[l], pools[l]
        table = page_table[l] if isinstance(page_table, (list, tuple)) else page_table
        H, nq, nkv, d = cfg.hidden, cfg.n_q, cfg.n_kv, cfg.head_dim
        if name == "attn_norm":
            live["xn"] = rmsnorm(live["resid"], w["g_attn"], cfg.rms_eps)
        elif name == "qkv_proj":
            live["qkv"] = linear(live["xn"], w["w_qkv"])
        elif name == "rope":
            qkv = live["qkv"].copy()
            q = qkv[:, :nq * d].reshape(B, nq, d)
            k = qkv[:, nq * d:(nq + nkv) * d].reshape(B, nkv, d)
            qkv[:, :nq * d] = rope_rotate(q, pos, cfg.rope_theta).reshape(B, -1)
            qkv[:, nq * d:(nq + nkv) * d] = rope_rotate(k, pos, cfg.rope_theta).reshape(B, -1)
            live["qkv"] = qkv
        elif name == "kv_append":
            qkv = live["qkv"]
            for b in range(B):
                p = int(pos[b])
                k = qkv[b, nq * d:(nq + nkv) * d].reshape(nkv, d)
                v = qkv[b, (nq + nkv) * d:].reshape(nkv, d)
                write_kv_slot(pool, int(table[b, p // PAGE]), p % PAGE, k, v, d)
        elif name == "attn_core":
            o = np.empty((B, nq * d))
            for b in range(B):
                p = int(pos[b])
                lo = window_start(p, cfg.window)
                K, V = page_kv(pool, table[b], p + 1, nkv, d, first=lo)   # keys lo .. p
                q = live["qkv"][b, :nq * d].reshape(nq, d)
                o[b] = attention_row(q, K, V, 0, p - lo).reshape(-1)
            live["o"] = o
        elif name == "o_proj_residual":
            live["resid"] = live["resid"] + linear(live["o"], w["w_o"])
        elif name == "ffn_norm":
            live["hn"] = rmsnorm(live["resid"], w["g_ffn"], cfg.rms_eps)
        elif name == "gate_up":
            live["gu"] = linear(live["hn"], w["w_gate_up"])
        elif name == "silu_mul":
            src, dst, F = ("gu_p", "act_p", cfg.moe_ffn) if cfg.n_experts else ("gu", "act", cfg.ffn)
            live[dst] = silu(live[src][:, :F]) * live[src][:, F:2 * F]
        elif name == "down_residual":
            live["resid"] = live["resid"] + linear(live["act"], w["w_down"])
        elif name == "router":
            live["logits"] = linear(live["hn"], w["w_router"])
        elif name == "topk_softmax":
            live["topk_ids"], live["topk_w"] = topk_route(live["logits"], cfg.top_k)
        elif name == "moe_permute":
            perm, off, slot_pos = moe_permute(live["topk_ids"], cfg.n_experts)
            live["perm"], live["expert_off"], live["slot_pos"] = perm, off, slot_pos
            live["xp"] = live["hn"][perm // cfg.top_k]
        elif name == "expert_gate_up":
            live["gu_p"] = _grouped(live["xp"], w["w_gate_up"], live["expert_off"])
        elif name == "expert_down":
            live["yp"] = _grouped(live["act_p"], w["w_down"], live["expert_off"])
        elif name == "moe_combine_residual":
            k = cfg.top_k
            yk = live["yp"][live["slot_pos"]].reshape(B, k, H)
            live["resid"] = live["resid"] + np.einsum("bk,bkh->bh", live["topk_w"], yk)
        else:  # pragma: no cover
            raise AssertionError(name)
    return live


def _grouped(x: np.ndarray, w: np.ndarray, expert_off: np.ndarray) -> np.ndarray:
    """Rows [off[e], off[e+1]) of x times w[e]^T, for every expert e."""
    out = np.zeros((x.shape[0], w.shape[1]))
    for e in range(w.shape[0]):
        a, b = int(expert_off[e]), int(expert_off[e + 1])
        if b > a:
            out[a:b] = x[a:b] @ w[e].T
    return out
