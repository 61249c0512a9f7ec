"""Parity on seeded random layer shapes, through the C ABI.

Hand-picked shapes elsewhere aim at particular tiles and tails; these draw
the shape itself: head size 64 or 128, one to four KV heads with one to eight
query heads each, hidden sizes that are or are not multiples of 64, dense or
top-k MoE FFNs of assorted widths, full or sliding-window attention, batches
from 1 to 300 with ragged contexts, and row-major or tiled weights wherever
the tiled layout applies. Each case runs the whole layer in one call and
again cut at two seeded operator indices, and compares every live buffer
with the oracle (1e-2 per buffer, max |gpu - oracle| / max |oracle|); MoE
routing is checked as in the other parity tests (ids equal to the top-k of
the GPU's own logits, the oracle's choice wherever no near-tie can flip it),
and the residual against the oracle evaluated with the GPU's experts."""
import sys

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from harness import Setup, assert_close, f64, oracle_run, report, routing_check

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)


def say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


def fresh(inp):
    out = dict(inp)
    out["pools"] = [p.copy() for p in inp["pools"]]
    return out


def draw(i):
    rng = np.random.default_rng(1000 + i)
    D = int(rng.choice([64, 128]))
    n_kv = int(rng.choice([1, 2, 4, 8]))
    group = int(rng.choice([1, 2, 4, 8]))
    hidden = 64 * int(rng.integers(2, 17)) + (8 * int(rng.integers(1, 8)) if rng.random() < 0.3 else 0)
    window = int(16 * rng.integers(1, 12) + rng.integers(0, 16)) if rng.random() < 0.3 else 0
    if rng.random() < 0.35:
        E = int(rng.choice([8, 16, 32]))
        cfg = W.LayerCfg(hidden=hidden, n_q=group * n_kv, n_kv=n_kv, head_dim=D, n_experts=E,
                         top_k=int(rng.integers(1, min(8, E) + 1)),
                         moe_ffn=64 * int(rng.integers(1, 5)) + (8 if rng.random() < 0.3 else 0), window=window)
    else:
        cfg = W.LayerCfg(hidden=hidden, n_q=group * n_kv, n_kv=n_kv, head_dim=D, window=window,
                         ffn=64 * int(rng.integers(2, 33)) + (8 * int(rng.integers(1, 8)) if rng.random() < 0.3 else 0))
    batch = int(rng.choice([1, 5, 33, 64, 100, 200, 300]))
    w = W.Workload(f"random{i}", (cfg,), batch=batch, ctx_lo=1, ctx_hi=int(rng.integers(2, 400)),
                   router_std=hidden ** -0.5)
    n = cfg.n_ops
    cut = sorted(rng.choice(np.arange(1, n), 2, replace=False).tolist())
    tiled = bool(rng.random() < 0.8) and hidden % 64 == 0 and (cfg.moe_ffn or cfg.ffn) % 64 == 0
    return w, cut, tiled


CASES = [draw(i) for i in range(24)]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_random_layer_shape(case):
    w, cut, tiled = CASES[case]
    cfg = w.layers[0]
    n = cfg.n_ops
    say(f"random shape {case}: {cfg}, batch {w.batch}, contexts 1..{w.ctx_hi}, cut {cut}, "
        f"{'tiled' if tiled else 'row-major'}")
    s = Setup(w, seed=50 + case, tiled=tiled)
    inp = s.oracle_inputs()
    ref = oracle_run(fresh(inp), w.layers, 0, n)
    B, H, d = w.batch, cfg.hidden, cfg.head_dim
    for bounds in ([0, n], [0] + cut + [n]):
        s.reset_resid()
        for a, b in zip(bounds[:-1], bounds[1:]):
            s.run(a, b)
        torch.cuda.synchronize()
        tag = f"shape {case} cuts {bounds[1:-1]}"
        assert_close(f"{tag} xn", f64(s.buf("xn", B, H)), ref["xn"])
        assert_close(f"{tag} qkv", f64(s.buf("qkv", B, cfg.qkv_dim)), ref["qkv"])
        assert_close(f"{tag} o", f64(s.buf("o", B, cfg.n_q * d)), ref["o"])
        assert_close(f"{tag} hn", f64(s.buf("hn", B, H)), ref["hn"])
        if not cfg.n_experts:
            assert_close(f"{tag} resid", f64(s.buf("resid", B, H)), ref["resid"])
            continue
        logits = f64(s.buf("logits", B, cfg.n_experts))
        ids = s.buf("topk_ids", B, cfg.top_k).cpu().numpy()
        wts = f64(s.buf("topk_w", B, cfg.top_k))
        forced, summary = routing_check(tag, ids, wts, logits, ref, cfg.top_k, min_fixed=0.0)
        assert_close(f"{tag} logits", logits, ref["logits"])
        pre = oracle_run(fresh(inp), w.layers, 0, 9)
        live = {"resid": pre["resid"].copy(), "hn": pre["hn"], "topk_ids": forced,
                "topk_w": O.route_weights(ref["logits"], forced)}
        ref2 = oracle_run(fresh(inp), w.layers, 9, n, live)
        assert_close(f"{tag} resid", f64(s.buf("resid", B, H)), ref2["resid"])
        report(f"{tag}: routing {summary}")
