"""Analytical cost model and a small exhaustive serving planner (host side, no GPU).

Cost model (Section 3 and Appendix A). A GPU type is (c, beta, M, F): unit-time
price, memory bandwidth, memory capacity, peak compute. With alpha = c / beta
(price per byte moved) and gamma = c / F (price per flop), the per-token cost
of decoding at average sequence length s is
  homogeneous disaggregation   CPT_hom(s)   = alpha m_kv(s) + 2 gamma P_act
  heterogeneous (attn on j,
    GEMM operators on k)       CPT_het(s)   = alpha_j m_kv(s) + 2 gamma_k P_act
  colocated                    CPT_coloc(s) = alpha m_kv(s)
                                              + max(alpha M_weights / b_bar(s), 2 gamma P_act)
with b_bar(s) = (M - M_weights) / m_kv(s) the relaxed feasible batch and
b_max = floor(b_bar). GEMMs turn compute-bound at b* = M_weights F / (2 P_act beta).
Theorem 1 bounds the gain G_hom = CPT_coloc / CPT_hom by M / (M - M_weights);
Theorem 2 bounds G_het = min_j CPT_hom_j / CPT_het_* by (1 + sqrt(eta)) / 2 with
eta = beta_1 F_2 / (beta_2 F_1) >= 1, and puts its peak at the crossing
x* = 2 P_act (gamma_1 - gamma_2) / (alpha_2 - alpha_1) of x = m_kv(s).

Planner (Sections 4-5, Appendix B). A partition block of N ordered operators
is cut by a contiguous template q = (0 = q_0 < ... < q_S = N); stage j runs on
owner type sigma(j) = ((j - 1) mod K) + 1: K = S (one stage position per type)
for templates over the whole block, or, for a block of identical-structure
layers, one per-layer template of K stages tiled over every layer (S = layers
x K, each type owning one position per layer, as AFD and CAD do). Busy time,
memory and link load add up over a type's positions. Each type m has its own
per-replica microbatch b_hat_m, so a global
microbatch of B_hat requests takes n_m = B_hat / b_hat_m replicas of type m:
a type with a larger microbatch gathers the microbatches of several replicas
of the types before it (Appendix B, replica counts). Stage latency t_j sums
its operators' latencies at the microbatch of its type (roofline estimates
max(D / beta, W / F), or measured per-operator profiles); the transfer after
stage j moves the live set at that cut, u_j = b_hat * A_j / link bandwidth
with b_hat the larger of the two sides' microbatches (the side that gathers
or scatters serializes them over its link). The round-trip time of mu
microbatches over B_total blocks is taken as the larger of the two lower
bounds the paper's branch-and-bound uses: the dependency chain of one
microbatch, B_total * sum_j (t_j + u_j) (the last block's wrap-around transfer
omitted), and the serialized work of the busiest resource, mu * B_total *
t_j per replica and per link. A plan costs CPT = T_rtt * sum_m c_m / b_m with
b_m = mu * b_hat_m, subject to T_rtt <= SLO and, per type, weights of its
stages plus the KV of mu resident microbatches within M. The search is
exhaustive over S, templates (and the block's rotation, so a stage may wrap
the block boundary as CAD's rest-of-model stage does), mu and the
microbatches: one shared by every type, or (per_type_batch) one per type;
given several GPU kinds, every type also takes any kind, each with its own
price, memory and latencies (heterogeneous plans).
"""
from __future__ import annotations

import bisect
import itertools
import math
from dataclasses import dataclass, field
from typing import Callable, Sequence

BF16 = 2  # bytes per weight / activation element


# ---------------------------------------------------------------- hardware and model

@dataclass(frozen=True)
class Gpu:
    name: str
    price_per_hour: float   # c, USD per GPU-hour
    bandwidth: float        # beta, bytes / s
    memory: float           # M, bytes
    flops: float            # F, bf16 flop / s (dense)

    @property
    def c(self) -> float:
        """Unit-time cost, USD per second."""
        return self.price_per_hour / 3600.0

    @property
    def alpha(self) -> float:
        return self.c / self.bandwidth

    @property
    def gamma(self) -> float:
        return self.c / self.flops


MI355X = Gpu("MI355X", price_per_hour=1.0, bandwidth=8.0e12, memory=288e9, flops=2.5166e15)


def _is_moe(cfg) -> bool:
    return bool(getattr(cfg, "n_experts", 0))


def layer_weight_params(cfg) -> int:
    """Resident GEMM parameters of one layer (all experts for MoE)."""
    H, d = cfg.hidden, cfg.head_dim
    attn = cfg.qkv_dim * H + H * cfg.n_q * d
    if _is_moe(cfg):
        return attn + cfg.n_experts * 3 * H * cfg.moe_ffn + H * cfg.n_experts
    return attn + 3 * H * cfg.ffn


def layer_active_params(cfg) -> int:
    """GEMM parameters one token activates in one layer (top-k experts for MoE)."""
    H, d = cfg.hidden, cfg.head_dim
    attn = cfg.qkv_dim * H + H * cfg.n_q * d
    if _is_moe(cfg):
        return attn + cfg.top_k * 3 * H * cfg.moe_ffn + H * cfg.n_experts
    return attn + 3 * H * cfg.ffn


def layer_kv_bytes(cfg, s: float) -> float:
    """KV-cache bytes one request keeps in this layer at sequence length s
    (a sliding-window layer keeps at most its window)."""
    tokens = min(s, cfg.window) if getattr(cfg, "window", 0) else s
    return 2 * cfg.n_kv * cfg.head_dim * BF16 * tokens


@dataclass(frozen=True)
class Model:
    """A model as B_total repeats of a partition block of layers."""
    block: tuple
    n_blocks: int

    @property
    def p_act(self) -> float:
        return self.n_blocks * sum(layer_active_params(c) for c in self.block)

    @property
    def m_weights(self) -> float:
        return self.n_blocks * sum(layer_weight_params(c) for c in self.block) * BF16

    def m_kv(self, s: float) -> float:
        return self.n_blocks * sum(layer_kv_bytes(c, s) for c in self.block)


# ---------------------------------------------------------------- Section 3 closed forms

def cpt_hom(g: Gpu, m: Model, s: float) -> float:
    return g.alpha * m.m_kv(s) + 2 * g.gamma * m.p_act


def cpt_het(g_attn: Gpu, g_gemm: Gpu, m: Model, s: float) -> float:
    return g_attn.alpha * m.m_kv(s) + 2 * g_gemm.gamma * m.p_act


def b_bar(g: Gpu, m: Model, s: float) -> float:
    return (g.memory - m.m_weights) / m.m_kv(s)


def b_max(g: Gpu, m: Model, s: float) -> int:
    return math.floor(b_bar(g, m, s))


def cpt_coloc(g: Gpu, m: Model, s: float) -> float:
    bb = b_bar(g, m, s)
    if bb < 1:
        raise ValueError("colocation is infeasible at this sequence length (b_bar < 1)")
    return g.alpha * m.m_kv(s) + max(g.alpha * m.m_weights / bb, 2 * g.gamma * m.p_act)


def b_star(g: Gpu, m: Model) -> float:
    """Batch at which GEMM weight-loading time equals compute time."""
    return m.m_weights * g.flops / (2 * m.p_act * g.bandwidth)


def g_hom(g: Gpu, m: Model, s: float) -> float:
    return cpt_coloc(g, m, s) / cpt_hom(g, m, s)


def g_hom_bound(g: Gpu, m: Model) -> float:
    return g.memory / (g.memory - m.m_weights)


def eta(g1: Gpu, g2: Gpu) -> float:
    """Hardware ratio beta_1 F_2 / (beta_2 F_1), taken >= 1 by labelling."""
    r = (g1.bandwidth * g2.flops) / (g2.bandwidth * g1.flops)
    return max(r, 1.0 / r)


def g_het(gpus: Sequence[Gpu], m: Model, s: float) -> float:
    hom = min(cpt_hom(g, m, s) for g in gpus)
    het = min(g.alpha for g in gpus) * m.m_kv(s) + min(g.gamma for g in gpus) * 2 * m.p_act
    return hom / het


def g_het_bound(e: float) -> float:
    return (1.0 + math.sqrt(e)) / 2.0


def x_star(g1: Gpu, g2: Gpu, m: Model) -> float:
    """KV bytes per request at which the two homogeneous costs cross; the
    types are labelled so that g1 is the cheaper one per byte."""
    if g1.alpha > g2.alpha:
        g1, g2 = g2, g1
    return 2 * m.p_act * (g1.gamma - g2.gamma) / (g2.alpha - g1.alpha)


# ---------------------------------------------------------------- operators of a block

OP_NAMES_DENSE = ("attn_norm", "qkv_proj", "rope", "kv_append", "attn_core", "o_proj_residual",
                  "ffn_norm", "gate_up", "silu_mul", "down_residual")
OP_NAMES_MOE = OP_NAMES_DENSE[:7] + ("router", "topk_softmax", "moe_permute", "expert_gate_up", "silu_mul",
                                     "expert_down", "moe_combine_residual")


def layer_op_names(cfg) -> tuple:
    return OP_NAMES_MOE if _is_moe(cfg) else OP_NAMES_DENSE


def handoff_bytes_per_token(cfg) -> list:
    """Bytes per request of the live set that crosses a cut after each local
    operator of a layer (the activation interface A_j): the residual stream
    plus whatever later operators of the layer still read."""
    H, nq, d = cfg.hidden, cfg.n_q, cfg.head_dim
    resid, qkv, q, o = 2 * H, 2 * cfg.qkv_dim, 2 * nq * d, 2 * nq * d
    if not _is_moe(cfg):
        F = cfg.ffn
        return [resid + 2 * H, resid + qkv, resid + qkv, resid + q, resid + o, resid,
                resid + 2 * H, resid + 4 * F, resid + 2 * F, resid]
    E, k, I = cfg.n_experts, cfg.top_k, cfg.moe_ffn
    route = 4 * k + 4 * k  # routing weights and slots, read by the combine
    return [resid + 2 * H, resid + qkv, resid + qkv, resid + q, resid + o, resid,
            resid + 2 * H, resid + 2 * H + 4 * E, resid + 2 * H + 8 * k,
            resid + 2 * k * H + route, resid + 4 * k * I + route, resid + 2 * k * I + route,
            resid + 2 * k * H + route, resid]


def op_bytes_flops(cfg, op: str, b: float, s: float):
    """(D, W, resident weight bytes, KV bytes per request) of one operator of a
    layer at batch b and sequence length s, per the roofline accounting of
    Appendix A (weights read once per call, activations in and out)."""
    H, nq, nkv, d = cfg.hidden, cfg.n_q, cfg.n_kv, cfg.head_dim
    qd = cfg.qkv_dim
    if op in ("attn_norm", "ffn_norm"):
        return 2 * BF16 * b * H, 4 * b * H, 0, 0
    if op == "qkv_proj":
        w = qd * H * BF16
        return w + BF16 * b * (H + qd), 2 * b * H * qd, w, 0
    if op == "rope":
        return 2 * BF16 * b * (nq + nkv) * d, 6 * b * (nq + nkv) * d, 0, 0
    if op == "kv_append":
        return BF16 * b * 2 * nkv * d, 0, 0, 0
    if op == "attn_core":
        kv = layer_kv_bytes(cfg, s)
        tokens = kv / (2 * nkv * d * BF16)
        return b * kv + 2 * BF16 * b * nq * d, 4 * b * nq * d * tokens, 0, kv
    if op == "o_proj_residual":
        w = H * nq * d * BF16
        return w + BF16 * b * (nq * d + 2 * H), 2 * b * H * nq * d, w, 0
    if _is_moe(cfg):
        E, k, I = cfg.n_experts, cfg.top_k, cfg.moe_ffn
        touched = E * (1.0 - (1.0 - k / E) ** b)  # experts hit by at least one of b tokens
        if op == "router":
            w = E * H * BF16
            return w + BF16 * b * H + 4 * b * E, 2 * b * H * E, w, 0
        if op == "topk_softmax":
            return 4 * b * E + 8 * b * k, 8 * b * E, 0, 0
        if op == "moe_permute":
            return 2 * BF16 * b * k * H, 0, 0, 0
        if op == "expert_gate_up":
            return touched * 2 * I * H * BF16 + BF16 * b * k * (H + 2 * I), 2 * b * k * H * 2 * I, E * 2 * I * H * BF16, 0
        if op == "silu_mul":
            return BF16 * b * k * 3 * I, 4 * b * k * I, 0, 0
        if op == "expert_down":
            return touched * H * I * BF16 + BF16 * b * k * (I + H), 2 * b * k * H * I, E * H * I * BF16, 0
        if op == "moe_combine_residual":
            return BF16 * b * (k * H + 2 * H) + 4 * b * k, 2 * b * k * H, 0, 0
    else:
        F = cfg.ffn
        if op == "gate_up":
            w = 2 * F * H * BF16
            return w + BF16 * b * (H + 2 * F), 2 * b * H * 2 * F, w, 0
        if op == "silu_mul":
            return BF16 * b * 3 * F, 4 * b * F, 0, 0
        if op == "down_residual":
            w = H * F * BF16
            return w + BF16 * b * (F + 2 * H), 2 * b * H * F, w, 0
    raise ValueError(f"unknown operator {op}")


@dataclass(frozen=True)
class BlockOp:
    layer: int
    local: int
    name: str
    cfg: object


def block_ops(block: Sequence) -> list:
    return [BlockOp(l, j, n, c) for l, c in enumerate(block) for j, n in enumerate(layer_op_names(c))]


def roofline_latency(g: Gpu) -> Callable:
    """Operator latency max(D / beta, W / F) of Appendix A."""
    def lat(op: BlockOp, b: float, s: float) -> float:
        D, W, _, _ = op_bytes_flops(op.cfg, op.name, b, s)
        return max(D / g.bandwidth, W / g.flops)
    return lat


class ProfiledLatency:
    """Measured single-operator latencies t(op, b, s) per layer shape (the
    layer's attention window: 0 for full attention), interpolated linearly in
    batch and sequence length (clamped at the ends). rows: iterable of dicts
    with keys local (operator index), batch, ctx, us and optionally window."""

    def __init__(self, rows):
        table = {}
        for r in rows:
            key = (int(r.get("window", 0)), int(r["local"]))
            table.setdefault(key, {}).setdefault(float(r["ctx"]), []).append((float(r["batch"]), float(r["us"])))
        self.table = {j: {c: sorted(v) for c, v in per.items()} for j, per in table.items()}

    @staticmethod
    def _interp(pts, x):
        xs = [p[0] for p in pts]
        i = bisect.bisect_left(xs, x)
        if i == 0:
            return pts[0][1]
        if i == len(pts):
            return pts[-1][1]
        (x0, y0), (x1, y1) = pts[i - 1], pts[i]
        return y0 + (y1 - y0) * (x - x0) / (x1 - x0)

    def __call__(self, op: BlockOp, b: float, s: float) -> float:
        per = self.table[(int(getattr(op.cfg, "window", 0)), op.local)]
        ctxs = sorted(per)
        i = bisect.bisect_left(ctxs, s)
        if i == 0 or i == len(ctxs):
            c = ctxs[0] if i == 0 else ctxs[-1]
            return self._interp(per[c], b) * 1e-6
        c0, c1 = ctxs[i - 1], ctxs[i]
        y0, y1 = self._interp(per[c0], b), self._interp(per[c1], b)
        return (y0 + (y1 - y0) * (s - c0) / (c1 - c0)) * 1e-6


# ---------------------------------------------------------------- templates and plans

def templates(n_ops: int, S: int):
    """Every contiguous template q = (0, q_1, ..., q_{S-1}, n_ops)."""
    for cut in itertools.combinations(range(1, n_ops), S - 1):
        yield (0,) + cut + (n_ops,)


def count_templates(n_ops: int, S: int) -> int:
    return math.comb(n_ops - 1, S - 1)


def subblock_templates(n_ops: int, n_rep: int, K: int):
    """Templates chosen inside one of n_rep identical sub-blocks and tiled over
    the block (S = n_rep * K stages)."""
    if n_ops % n_rep:
        raise ValueError("the sub-block must divide the block")
    sub = n_ops // n_rep
    for q in templates(sub, K):
        out = [0]
        for r in range(n_rep):
            out.extend(r * sub + x for x in q[1:])
        yield tuple(out)


@dataclass
class Plan:
    rotation: int
    q: tuple
    mu: int
    b_hat: int            # the largest per-replica microbatch of the plan's types
    t: list
    u: list
    t_rtt: float
    cpt: float
    memory: list = field(default_factory=list)   # per type
    b_hats: tuple = ()    # per-replica microbatch of each type
    K: int = 0            # device-group types; stage j runs on type j mod K (0: one type per stage)
    tiled: int = 0        # > 0: q tiles one per-layer template over this many layers
    kinds: tuple = ()     # GPU kind of each type

    @property
    def types(self) -> int:
        return self.K or self.S

    @property
    def S(self) -> int:
        return len(self.q) - 1


class _Tables:
    """Per-batch operator latencies, weights, KV bytes and cut handoffs of a
    block, doubled so a rotated block is a plain slice, with prefix sums."""

    def __init__(self, model: Model, g: Gpu, s: float, latency: Callable, b_hats, link_bw: float):
        ops = block_ops(model.block)
        self.N = len(ops)
        self.by_b = {}
        for b in b_hats:
            lat = [latency(op, b, s) for op in ops] * 2
            w = [op_bytes_flops(op.cfg, op.name, b, s)[2] for op in ops] * 2
            kv = [op_bytes_flops(op.cfg, op.name, b, s)[3] for op in ops] * 2
            hand = [b * handoff_bytes_per_token(op.cfg)[op.local] / link_bw for op in ops] * 2
            pre = lambda xs: list(itertools.accumulate(xs, initial=0.0))
            self.by_b[b] = (pre(lat), pre(w), pre(kv), hand)


def _plan_from_tables(model: Model, g, tab, q: tuple, mu: int, b_hat, rotation: int,
                      K: int = 0, tiled: int = 0):
    """Stage j of template q runs on device-group type j mod K (K = 0: one
    type per stage, K = S). b_hat: one per-replica microbatch for every type,
    or a tuple with one per type. g, tab: one GPU kind (and its tables) for
    every type, or tuples with one per type (heterogeneous plans)."""
    S = len(q) - 1
    T = K or S
    if S % T:
        raise ValueError("the stages must fill every type the same number of times")
    bs = tuple(b_hat) if isinstance(b_hat, tuple) else (b_hat,) * T
    gs = tuple(g) if isinstance(g, (tuple, list)) else (g,) * T
    tabs = tuple(tab) if isinstance(tab, (tuple, list)) else (tab,) * T
    t, u = [], []
    mem = [0.0] * T
    for j in range(S):
        m, m_next = j % T, (j + 1) % S % T
        plat, pw, pkv, _ = tabs[m].by_b[bs[m]]
        lo, hi = rotation + q[j], rotation + q[j + 1]
        t.append(plat[hi] - plat[lo])
        # the live set crosses to the next stage's type (none when it stays on one replica)
        u.append(tabs[m].by_b[max(bs[m], bs[m_next])][3][hi - 1] if m != m_next else 0.0)
        mem[m] += (pw[hi] - pw[lo]) * model.n_blocks + mu * bs[m] * (pkv[hi] - pkv[lo]) * model.n_blocks
    if any(x > gm.memory for x, gm in zip(mem, gs)):
        return None
    Bt = model.n_blocks
    chain = Bt * sum(t) + Bt * sum(u) - u[-1]
    busy = [sum(t[j] for j in range(m, S, T)) for m in range(T)]
    link = [sum(u[j] for j in range(m, S, T)) for m in range(T)]
    loads = [mu * Bt * x for x in busy] + [mu * Bt * x - (mu * u[-1] if m == (S - 1) % T else 0.0)
                                           for m, x in enumerate(link)]
    t_rtt = max([chain] + loads)
    cpt = t_rtt * sum(gm.c / (mu * b) for gm, b in zip(gs, bs))
    return Plan(rotation, q, mu, max(bs), t, u, t_rtt, cpt, mem, bs, K, tiled, tuple(gm.name for gm in gs))


def evaluate(model: Model, g: Gpu, q: tuple, mu: int, b_hat: int, s: float, latency: Callable | None = None,
             link_bw: float = 153e9, rotation: int = 0):
    """Round-trip time, cost per token and per-owner memory of one plan on one
    GPU type (owner m runs stage m of every block); None if a stage's memory
    does not fit."""
    tab = _Tables(model, g, s, latency or roofline_latency(g), (b_hat,), link_bw)
    return _plan_from_tables(model, g, tab, q, mu, b_hat, rotation)


def layer_ops_count(model: Model) -> int:
    """Operators per layer when every layer of the block has the same count, else 0."""
    counts = {len(layer_op_names(c)) for c in model.block}
    return counts.pop() if len(counts) == 1 else 0


def search(model: Model, g, s: float, slo: float, latency=None, S_max: int = 3,
           mus=(1, 2, 4, 8), b_hats=(1, 2, 4, 8, 16, 32, 64, 128, 256, 512), link_bw: float = 153e9,
           rotations: bool = True, per_type_batch: bool = False, per_type_S_max: int = 2, tiled_K=(2, 3)):
    """Every plan over the grid that meets the SLO and fits memory, cheapest
    first: contiguous templates of 1 to S_max stages over the block, one type
    per stage, and, for a block of several layers with the same operator
    sequence, one per-layer template of K stages tiled over every layer, its
    stages placed round-robin on K types (S = layers x K). With
    per_type_batch, plans of up to per_type_S_max types also try every
    combination of per-replica microbatches over their types. g is one GPU
    kind or a sequence of kinds, in which case every type takes any of them
    (the heterogeneous plans of Section 3.3); latency is one callable for
    every kind or a dict from kind name to callable (default: each kind's
    roofline)."""
    kinds = tuple(g) if isinstance(g, (tuple, list)) else (g,)

    def lat_of(k):
        if isinstance(latency, dict):
            return latency[k.name]
        return latency or roofline_latency(k)

    tabs = {k.name: _Tables(model, k, s, lat_of(k), b_hats, link_bw) for k in kinds}
    N = next(iter(tabs.values())).N

    def combos(T):
        return list(itertools.product(b_hats, repeat=T)) if per_type_batch and 1 < T <= per_type_S_max else list(b_hats)

    out = []

    def consider(q, r, K, tiled):
        T = K or len(q) - 1
        for ks in itertools.product(kinds, repeat=T):
            tk = tuple(tabs[k.name] for k in ks)
            for mu in mus:
                for b in combos(T):
                    p = _plan_from_tables(model, ks, tk, q, mu, b, r, K, tiled)
                    if p is not None and p.t_rtt <= slo:
                        out.append(p)

    for S in range(1, S_max + 1):
        for r in (range(N) if (rotations and S > 1) else (0,)):
            for q in templates(N, S):
                consider(q, r, 0, 0)
    L, n = layer_ops_count(model), len(model.block)
    if L and n > 1:
        for K in tiled_K:
            for r in (range(L) if rotations else (0,)):
                for q in subblock_templates(N, n, K):
                    consider(q, r, K, n)
    out.sort(key=lambda p: p.cpt)
    return out


# ---------------------------------------------------------------- plans from a measured profile

def named_plans(model: Model):
    """(label, rotation, q, K, tiled) of the templates the paper names: AFD
    cuts every layer after its output projection, CAD isolates every layer's
    core attention (kv_append, attn_core) and lets the rest-of-model stage wrap
    the layer boundary (a rotation by five operators); both alternate two
    device-group types over the block's layers. Colocated is one stage."""
    N = len(block_ops(model.block))
    n = len(model.block)
    if n == 1 or not layer_ops_count(model):
        return [("colocated", 0, (0, N), 0, 0), ("AFD", 0, (0, 6, N), 0, 0), ("CAD", 5, (0, N - 2, N), 0, 0)]
    L = layer_ops_count(model)
    tile = lambda sub: tuple([0] + [r * L + x for r in range(n) for x in sub[1:]])
    return [("colocated", 0, (0, N), 0, 0), ("AFD", 0, tile((0, 6, L)), 2, n), ("CAD", 5, tile((0, L - 2, L)), 2, n)]


def profile_report(profile: dict, model: Model, g: Gpu, s: float, slo: float, S_max: int = 3,
                   mus=(1, 2, 4, 8), b_hats=(1, 8, 32, 64, 128, 256), per_type_batch: bool = False) -> str:
    """Markdown table: the cheapest plan of the exhaustive search and the best
    point of each named template, with per-operator latencies measured on the
    GPU (profile["op_latency"]). With per_type_batch, plans of two stages
    choose a per-replica microbatch per type."""
    lat = ProfiledLatency(profile["op_latency"])
    plans = search(model, g, s, slo, lat, S_max=S_max, mus=mus, b_hats=b_hats, per_type_batch=per_type_batch)
    rows = []
    if plans:
        p = plans[0]
        rows.append(("search optimum", p))
    tab = _Tables(model, g, s, lat, b_hats, 153e9)
    for label, r, q, K, tiled in named_plans(model):
        T = K or len(q) - 1
        combos = list(itertools.product(b_hats, repeat=T)) if per_type_batch and T > 1 else list(b_hats)
        best = None
        for mu in mus:
            for b in combos:
                p = _plan_from_tables(model, g, tab, q, mu, b, r, K, tiled)
                if p is not None and p.t_rtt <= slo and (best is None or p.cpt < best.cpt):
                    best = p
        if best is not None:
            rows.append((label, best))
    return _plan_table(model, g, rows)


def _plan_table(model: Model, g: Gpu, rows) -> str:
    bops = block_ops(model.block)
    N = len(bops)
    name = lambda i: (f"L{bops[i % N].layer}." if len(model.block) > 1 else "") + bops[i % N].name
    out = [f"| plan | stages (operators, block rotated by r) | mu | b_hat per type | T_rtt ms | busy per type us | "
           f"GPU-seconds per 1k tokens |", "|---|---|---:|---:|---:|---|---:|"]
    for label, p in rows:
        if p.tiled:
            per = p.S // p.tiled
            stages = (" / ".join(f"{name(p.rotation + p.q[j])}..{name(p.rotation + p.q[j + 1] - 1)}"
                                 for j in range(per)) + f" (every layer, {p.types} types)")
        else:
            stages = " / ".join(f"{name(p.rotation + p.q[j])}..{name(p.rotation + p.q[j + 1] - 1)}"
                                for j in range(p.S))
        busy = [sum(p.t[j] for j in range(m, p.S, p.types)) for m in range(p.types)]
        out.append(f"| {label} | r={p.rotation}: {stages} | {p.mu} | {', '.join(str(b) for b in p.b_hats)} | "
                   f"{p.t_rtt * 1e3:.2f} | {', '.join(f'{t * 1e6:.0f}' for t in busy)} | {p.cpt / g.c * 1e3:.3f} |")
    return "\n".join(out)


if __name__ == "__main__":
    import argparse
    import json
    import sys as _sys
    import os as _os

    _sys.path.insert(0, _os.path.dirname(_os.path.dirname(_os.path.abspath(__file__))))
    import workloads as _W

    ap = argparse.ArgumentParser(description="serving plans for a model of repeated one-layer blocks from a "
                                             "measured per-operator profile")
    ap.add_argument("--profile", required=True, help="JSON written by bench.py --latency-table")
    ap.add_argument("--workload", default="dense8b_b64", help="one-layer workload whose layer the model repeats "
                                                              "(the layer the profile was measured on)")
    ap.add_argument("--layers", type=int, default=32)
    ap.add_argument("--slo-ms", type=float, default=50.0)
    ap.add_argument("--common-batch", action="store_true",
                    help="one per-replica microbatch for every stage type (default: one per type for "
                         "two-stage plans)")
    args = ap.parse_args()
    prof = json.load(open(args.profile))
    block = _W.BY_NAME[args.workload].layers
    if args.layers % len(block):
        _sys.exit(f"--layers must be a multiple of the block's {len(block)} layers")
    model = Model(block, args.layers // len(block))
    b_hats = tuple(sorted({int(r["batch"]) for r in prof["op_latency"]}))
    for s in (1024, 4096, 16384):
        print(f"\n### context {s}, {args.layers} layers, TPOT SLO {args.slo_ms:g} ms, MI355X\n")
        print(profile_report(prof, model, MI355X, s, args.slo_ms * 1e-3, b_hats=b_hats,
                             per_type_batch=not args.common_batch))
