"""Parity at the full evaluated sizes, in the launch configuration the
benchmark times (per layer: ops [0,4), [4,5), [5,6), [6,end)).

Tiled weights (the layout the benchmark runs) are checked on every row:
  * attention stage [0, 6): every row's residual, attention output and the
    K / V written to the appended slot;
  * FFN stage [6, end): every row's residual (and the dense SiLU-gated
    activation the stage materialises);
  * core attention [3, 5) from a fresh qkv, and the chained block run as the
    benchmark runs it: at least 64 rows covering every 64-row group of the
    batch plus its longest and shortest contexts.
Row-major weights run the same checks on a handful of sampled rows (the FFN
stage on every row). The oracle recomputes rows in chunks, reading only their
pages (only the window's pages for sliding-window layers).

Bars. A stage that starts from the same live set on both sides is held to
1e-2 per row (max |gpu - oracle| / max |oracle| of the row). A chained block
rounds every live buffer to bf16 at every layer, which compounds: its final
residual and its last attention output are held to a bar measured on these
inputs with a stated margin (CHAINED_BAR). Element-wise errors
(|gpu - oracle| / (|oracle| + 1e-3 max |oracle|)) are reported beside the
normwise ones.

Routing. The GPU's expert choice must equal the oracle's top-k of the GPU's
own fp32 logits for every token (the same decision on the same numbers).
Against the oracle's own logits, a token's choice is fixed beyond the
rounding of the GPU's bf16 input once its k-th / (k+1)-th logit gap exceeds
twice that token's measured max |GPU logit - oracle logit|: such tokens must
choose the same experts, and at least 90% of tokens must be such tokens. Any
other token's residual is compared against the oracle evaluated with the
GPU's expert set. Page tables and permutations are compared bit for bit."""
import sys
import time

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from workloads import gen
from harness import Setup, assert_rows_close, f64, report, routing_check

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

# The attention output inside a stage that starts from the residual carries
# the bf16 rounding of xn, qkv and the rotated q (a float64 emulation of just
# those roundings gives up to 9e-3 per row on the 8B-shaped layer). Measured
# against the oracle from the residual, the worst row over all configurations
# was 1.60e-2 (hybrid block, layer 0); the bar is 1.5 times that, rounded up.
O_BAR = 2.5e-2

# Chained blocks, as the benchmark runs them: the worst row measured on these
# inputs (tiled and row-major weights) times 1.5, rounded up, at least the
# per-stage 1e-2. Measured worst rows: one 8B-shaped layer, resid 5.8e-3 and
# last o 1.07e-2; the 4-layer hybrid block, resid 1.21e-2 and last o 2.59e-2;
# the MoE layer, resid 5.4e-3 and last o 8.3e-3.
CHAINED_BAR = {
    "dense8b_b64": {"resid": 1e-2, "o": O_BAR},
    "dense8b_b256_ctx8k": {"resid": 1e-2, "o": O_BAR},
    "hybrid4_b128": {"resid": 2e-2, "o": 4e-2},
    "moe64x8_b512": {"resid": 1e-2, "o": O_BAR},
    "dense8b_b256_ctx8k_tp8": {"resid": 1e-2, "o": O_BAR},
}


def say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


def layer_ops(c):
    return 14 if c.n_experts else 10


def bench_ranges(cfgs):
    out, off = [], 0
    for c in cfgs:
        n = layer_ops(c)
        out += [(off, off + 4), (off + 4, off + 5), (off + 5, off + 6), (off + 6, off + n)]
        off += n
    return out


def group_rows(ctx, per_batch, seed):
    """At least per_batch rows: an equal seeded share of every 64-row group of
    the batch, plus the longest and the shortest context."""
    B = len(ctx)
    rng = np.random.default_rng(seed)
    groups = [np.arange(g, min(g + 64, B)) for g in range(0, B, 64)]
    share = max(1, -(-per_batch // len(groups)))
    rows = {int(np.argmax(ctx)), int(np.argmin(ctx))}
    for g in groups:
        rows.update(int(r) for r in rng.choice(g, min(share, g.size), replace=False))
    return np.array(sorted(rows))


def host(t, rows=None):
    if rows is not None:
        t = t[torch.from_numpy(np.asarray(rows)).to(t.device)]
    return f64(t)


class FullSize:
    def __init__(self, w, tiled):
        say("full size", w.name, "setup", "tiled" if tiled else "row-major")
        self.w = w
        self.tiled = tiled
        self.tag = f"{w.name} {'tiled' if tiled else 'rows'}"
        self.s = Setup(w, seed=w.seed, tiled=tiled)
        np.testing.assert_array_equal(self.s.page_table,
                                      O.kv_alloc(self.s.ctx, self.s.pool_pages, w.seed, self.s.max_pages))
        B = w.batch
        self.all_rows = np.arange(B) if tiled else group_rows(self.s.ctx, 8, 1)
        self.sub_rows = group_rows(self.s.ctx, 64, 2) if tiled else self.all_rows

    def oracle_rows(self, rows, live_of, a, b):
        """Run the oracle over [a, b) chunk by chunk; live_of(chunk) gives the
        chunk's starting live set. Yields (chunk, result, chunk inputs)."""
        cfgs = list(self.w.layers)
        for chunk in self.s.row_chunks(rows):
            inp = self.s.oracle_inputs_windowed(chunk)
            ref = O.run_ops(cfgs, inp["weights"], inp["pools"], inp["page_table"], inp["ctx"], live_of(chunk), a, b)
            yield chunk, ref, inp


def appended_slots(s, layer, cfg, rows):
    """K (post-RoPE) and V the GPU wrote at each row's position ctx - 1: [rows, n_kv, d] each."""
    d, nkv = cfg.head_dim, cfg.n_kv
    pool = s.pools[layer].view(s.pool_pages, 2, nkv, 16 * d)
    ks, vs = [], []
    for b in rows:
        p = int(s.ctx[b]) - 1
        page, slot = int(s.page_table[b, p // 16]), p % 16
        ks.append(pool[page, 0, :, slot * d:(slot + 1) * d])
        vs.append(pool[page, 1, :, slot::16])
    return f64(torch.stack(ks)), f64(torch.stack(vs))


def oracle_slots(inp, layer, cfg, chunk_pos):
    """The oracle's appended K, V of chunk row i (after its kv_append)."""
    c = int(inp["ctx"][chunk_pos])
    K, V = O.page_kv(inp["pools"][layer], inp["page_table"][layer][chunk_pos], c, cfg.n_kv, cfg.head_dim,
                     first=c - 1)
    return K[:, 0], V[:, 0]


def attention_stage(f, l, off):
    """Attention stage [0, 6) of layer l from a fresh residual, every row of
    f.all_rows: the residual and the appended K / V (the stage's outputs)
    against the oracle from the same residual; the attention output against
    the oracle's core attention on the GPU's own rotated qkv (identical
    inputs), and against the oracle from the residual (which also carries the
    bf16 rounding of xn and qkv; bar O_BAR)."""
    w, s, cfg = f.w, f.s, f.w.layers[l]
    H = cfg.hidden
    say(f.tag, "layer", l, "attention stage", len(f.all_rows), "rows")
    t0 = time.time()
    x = gen.live_tensor((w.batch, H), w.seed + 100 + l, 10, "cuda")
    s.reset_resid(x)
    for a, b in bench_ranges(w.layers)[4 * l:4 * l + 3]:
        s.run(a, b)
    torch.cuda.synchronize()
    rows = f.all_rows
    h = host(s.buf("resid", w.batch, H), rows)
    o = host(s.buf("o", w.batch, cfg.n_q * cfg.head_dim), rows)
    qkv = host(s.buf("qkv", w.batch, cfg.qkv_dim), rows)
    k_gpu, v_gpu = appended_slots(s, l, cfg, rows)
    x64 = host(x)
    pos = {int(b): i for i, b in enumerate(rows)}
    ref_h, ref_o, own_o = np.empty_like(h), np.empty_like(o), np.empty_like(o)
    ref_k, ref_v = np.empty_like(k_gpu), np.empty_like(v_gpu)
    for chunk, ref, inp in f.oracle_rows(rows, lambda c: {"resid": x64[c].copy()}, off, off + 6):
        idx = [pos[b] for b in chunk]
        ref_h[idx], ref_o[idx] = ref["resid"], ref["o"]
        for i, j in enumerate(idx):
            ref_k[j], ref_v[j] = oracle_slots(inp, l, cfg, i)
        # core attention on the GPU's own rotated qkv (its k, v appended by the oracle)
        own = O.run_ops(list(w.layers), inp["weights"], inp["pools"], inp["page_table"], inp["ctx"],
                        {"qkv": qkv[idx].copy()}, off + 3, off + 5)
        own_o[idx] = own["o"]
    n = len(rows)
    eh = assert_rows_close(f"{f.tag} layer {l} attention stage resid", h, ref_h)
    ek = assert_rows_close(f"{f.tag} layer {l} appended K", k_gpu.reshape(n, -1), ref_k.reshape(n, -1))
    ev = assert_rows_close(f"{f.tag} layer {l} appended V", v_gpu.reshape(n, -1), ref_v.reshape(n, -1))
    ec = assert_rows_close(f"{f.tag} layer {l} attention o (oracle on the GPU's qkv)", o, own_o)
    eo = assert_rows_close(f"{f.tag} layer {l} attention o (oracle from the residual)", o, ref_o, O_BAR)
    report(f"{f.tag} L{l} attention stage, {n} rows: resid {eh[0]:.2e} (elem {eh[1]:.2e}), appended K {ek[0]:.2e} "
           f"/ V {ev[0]:.2e}; o vs oracle on GPU qkv {ec[0]:.2e} (elem {ec[1]:.2e}), o vs oracle from resid "
           f"{eo[0]:.2e} (bar {O_BAR:.1e})  [{time.time() - t0:.0f}s]")


def core_attention(f, l, off):
    """Core attention [3, 5) from a fresh qkv on f.sub_rows."""
    w, s, cfg = f.w, f.s, f.w.layers[l]
    say(f.tag, "layer", l, "core attention", len(f.sub_rows), "rows")
    qkv = gen.live_tensor((w.batch, cfg.qkv_dim), w.seed + 200 + l, 11, "cuda")
    s.buf("qkv", w.batch, cfg.qkv_dim).copy_(qkv)
    s.run(off + 3, off + 5)
    torch.cuda.synchronize()
    rows = f.sub_rows
    o = host(s.buf("o", w.batch, cfg.n_q * cfg.head_dim), rows)
    q64 = host(qkv)
    pos = {int(b): i for i, b in enumerate(rows)}
    ref_o = np.empty_like(o)
    for chunk, ref, _ in f.oracle_rows(rows, lambda c: {"qkv": q64[c].copy()}, off + 3, off + 5):
        for i, b in enumerate(chunk):
            ref_o[pos[b]] = ref["o"][i]
    e = assert_rows_close(f"{f.tag} layer {l} core attention o", o, ref_o)
    report(f"{f.tag} L{l} core attention, {len(rows)} rows (every 64-row group, longest and shortest "
           f"context): o {e[0]:.2e} (elem {e[1]:.2e})")


def ffn_stage(f, l, off):
    """FFN / MoE stage [6, end) of layer l from a fresh residual, every row."""
    w, s, cfg = f.w, f.s, f.w.layers[l]
    H, n = cfg.hidden, layer_ops(cfg)
    say(f.tag, "layer", l, "ffn stage")
    hx = gen.live_tensor((w.batch, H), w.seed + 300 + l, 12, "cuda")
    s.reset_resid(hx)
    s.run(off + 6, off + n)
    torch.cuda.synchronize()
    cfgs = list(w.layers)
    weights = s.oracle_weights()
    none = [None] * len(cfgs)
    x64 = host(hx)
    ref = O.run_ops(cfgs, weights, none, None, s.ctx, {"resid": x64.copy()}, off + 6, off + n)
    y = host(s.buf("resid", w.batch, H))
    if not cfg.n_experts:
        e = assert_rows_close(f"{f.tag} layer {l} ffn stage resid", y, ref["resid"])
        act = host(s.buf("act", w.batch, cfg.ffn))
        ref_act = O.silu(ref["gu"][:, :cfg.ffn]) * ref["gu"][:, cfg.ffn:]
        ea = assert_rows_close(f"{f.tag} layer {l} ffn stage act", act, ref_act)
        report(f"{f.tag} L{l} FFN stage, {w.batch} rows: resid {e[0]:.2e} (elem {e[1]:.2e}), "
               f"act {ea[0]:.2e} (elem {ea[1]:.2e})")
        return
    k, E = cfg.top_k, cfg.n_experts
    logits = host(s.buf("logits", w.batch, E))
    ids = s.buf("topk_ids", w.batch, k).cpu().numpy().astype(np.int64)
    wts = host(s.buf("topk_w", w.batch, k))
    forced, summary = routing_check(f"{f.tag} layer {l}", ids, wts, logits, ref, k)
    perm, eoff, slot = O.moe_permute(ids, E)
    np.testing.assert_array_equal(s.buf("perm", w.batch * k).cpu().numpy(), perm)
    np.testing.assert_array_equal(s.buf("expert_off", E + 1).cpu().numpy(), eoff)
    np.testing.assert_array_equal(s.buf("slot_pos", w.batch * k).cpu().numpy(), slot)
    # every token's residual, against the oracle run with the GPU's expert set
    # where the sets differ (near-ties)
    live = {"resid": x64.copy(), "hn": ref["hn"], "logits": ref["logits"], "topk_ids": forced,
            "topk_w": O.route_weights(ref["logits"], forced)}
    ref2 = O.run_ops(cfgs, weights, none, None, s.ctx, live, off + 9, off + n)
    e = assert_rows_close(f"{f.tag} layer {l} moe stage resid", y, ref2["resid"])
    report(f"{f.tag} L{l} MoE stage, {w.batch} tokens: resid {e[0]:.2e} (elem {e[1]:.2e}); routing: {summary}")


def chained(f):
    """The whole block as the benchmark runs it, from x, on f.sub_rows."""
    w, s = f.w, f.s
    say(f.tag, "chained block", len(f.sub_rows), "rows")
    s.reset_resid()
    for a, b in bench_ranges(w.layers):
        s.run(a, b)
    torch.cuda.synchronize()
    cfg = w.layers[-1]
    rows = f.sub_rows
    resid = host(s.buf("resid", w.batch, cfg.hidden), rows)
    o = host(s.buf("o", w.batch, cfg.n_q * cfg.head_dim), rows)
    ids = s.buf("topk_ids", w.batch, cfg.top_k).cpu().numpy()[rows] if cfg.n_experts else None
    x64 = host(s.x)
    pos = {int(b): i for i, b in enumerate(rows)}
    ref_r, ref_o = np.empty_like(resid), np.empty_like(o)
    ref_ids = np.empty_like(ids) if ids is not None else None
    ref_logits = np.empty((len(rows), cfg.n_experts)) if ids is not None else None
    n_ops = sum(layer_ops(c) for c in w.layers)
    for chunk, ref, _ in f.oracle_rows(rows, lambda c: {"resid": x64[c].copy()}, 0, n_ops):
        for i, b in enumerate(chunk):
            j = pos[b]
            ref_r[j], ref_o[j] = ref["resid"][i], ref["o"][i]
            if ids is not None:
                ref_ids[j], ref_logits[j] = ref["topk_ids"][i], ref["logits"][i]
    keep = np.ones(len(rows), dtype=bool)
    if ids is not None:
        # a chained MoE token is compared where its routing is the oracle's
        keep = np.array([set(a) == set(b) for a, b in zip(ids, ref_ids)])
    bar = CHAINED_BAR[w.name]
    er = assert_rows_close(f"{f.tag} chained resid", resid[keep], ref_r[keep], bar["resid"])
    eo = assert_rows_close(f"{f.tag} chained last-layer o", o, ref_o, bar["o"])
    extra = f", {int((~keep).sum())} tokens routed differently (not compared)" if ids is not None else ""
    report(f"{f.tag} chained {len(w.layers)}-layer block, {len(rows)} rows: resid {er[0]:.2e} (elem {er[1]:.2e}, "
           f"bar {bar['resid']:.1e}), last o {eo[0]:.2e} (elem {eo[1]:.2e}, bar {bar['o']:.1e}){extra}")


@pytest.mark.parametrize("tiled", [True, False], ids=["tiled", "rows"])
@pytest.mark.parametrize("name", ["dense8b_b64", "dense8b_b256_ctx8k", "hybrid4_b128", "moe64x8_b512",
                                  "dense8b_b256_ctx8k_tp8"])
def test_fullsize(name, tiled):
    w = W.BY_NAME[name]
    f = FullSize(w, tiled)
    chained(f)
    off = 0
    for l, cfg in enumerate(w.layers):
        attention_stage(f, l, off)
        core_attention(f, l, off)
        ffn_stage(f, l, off)
        off += layer_ops(cfg)
    del f
    torch.cuda.empty_cache()
