"""Window-only KV page ring for sliding-window layers.

A sliding-window layer reads only the most recent `window` tokens, so its KV
pages can live in a ring of R >= ceil(window / 16) + 1 pages per sequence:
token position t goes to page ring_table[b][(t // 16) % R]. The ring is a pure
storage reorganisation, so (1) a block run with the ring must equal, bit for
bit, the same block run with full page tables holding the same logical pages,
and (2) the oracle, reading K/V through the logical table t // 16 ->
ring_table[b][(t // 16) % R] (the ring's definition, written out here), must
agree with the ring run, also for contexts no full table of the test covers.
Ring pages that hold logical pages older than the window are filled with NaN,
so a read outside the window shows up in the output."""
import sys
from dataclasses import replace

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from harness import Setup, assert_close, f64, oracle_run
from workloads import gen

pytestmark = pytest.mark.gpu

PAGE = 16


def say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


def ring_alloc(ctx, R, seed):
    from paper_2609_14237_amd import binding as B
    rctx = np.minimum(np.asarray(ctx, dtype=np.int64), PAGE * R).astype(np.int32)
    pool_pages = int(sum(-(-int(c) // PAGE) for c in rctx))
    table = np.zeros((len(ctx), R), dtype=np.int32)
    assert B.ods_kv_alloc(pool_pages, rctx, len(ctx), seed, R, table) == 0, B.ods_last_error()
    return table, pool_pages


def window_pages(c, window):
    p = int(c) - 1
    lo = max(0, p - window + 1)
    return lo // PAGE, p // PAGE


def fill_ring(full_pool, page_table, ctx, ring_table, ring_pages_total, window, R):
    """Ring pool holding, for each sequence, the logical pages the ring keeps
    (the last R of them); pages older than the window are NaN."""
    ring = torch.full((ring_pages_total,) + tuple(full_pool.shape[1:]), float("nan"), dtype=full_pool.dtype,
                      device=full_pool.device)
    for b, c in enumerate(ctx):
        first_w, last = window_pages(c, window)
        for lp in range(max(0, last - R + 1), last + 1):
            if lp >= first_w:
                ring[int(ring_table[b, lp % R])] = full_pool[int(page_table[b, lp])]
    return ring


CFG = W.LayerCfg(hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=512)


@pytest.mark.parametrize("R_extra", [0, 3])
def test_ring_block_equals_full_tables_and_oracle(R_extra):
    """Sliding-window layer (window 64) then a full layer; contexts 1..400
    (shorter than, equal to and far beyond the window, so rings wrap)."""
    from paper_2609_14237_amd import runtime as Rt
    window = 64
    cfgs = (replace(CFG, window=window), CFG)
    w = W.Workload("ring_small", cfgs, batch=16, ctx_lo=1, ctx_hi=400)
    ctx = np.array([1, 15, 16, 17, 63, 64, 65, 80, 127, 129, 200, 255, 256, 257, 333, 400], dtype=np.int32)
    R = -(-window // PAGE) + 1 + R_extra
    say("ring block, R =", R)
    s = Setup(w, seed=21, ctx=ctx, nan_trap=True)
    inp = s.oracle_inputs()
    ref = oracle_run(inp, cfgs, 0, 20)
    pools0 = [p.clone() for p in s.pools]
    ring_table, ring_pages_total = ring_alloc(ctx, R, seed=77)
    ring_pool = fill_ring(pools0[0], s.page_table, ctx, ring_table, ring_pages_total, window, R)

    # full page tables
    s.reset_resid()
    s.run(0, 20)
    torch.cuda.synchronize()
    resid_full = s.buf("resid", w.batch, 256).clone()
    o_full = s.buf("o", w.batch, 256).clone()
    pool_full_after = s.pools[0]

    # the same block with the window-only ring for layer 0
    block = Rt.DeviceBlock(cfgs, s.weights, [ring_pool, pools0[1]], [ring_pages_total, s.pool_pages])
    batch = Rt.DeviceBatch(s.batch.ctx_lens, s.batch.page_table, ring_table=torch.from_numpy(ring_table).cuda())
    state = Rt.DeviceState(block, batch, "cuda", fill=float("nan"))
    for cuts in ((0, 20), (0, 4, 5, 6, 10, 14, 15, 20)):
        state.view("resid", w.batch, 256).copy_(s.x)
        for a, b in zip(cuts, cuts[1:]):
            Rt.run_partition(block, a, b, batch, state)
        torch.cuda.synchronize()
        assert torch.equal(state.view("resid", w.batch, 256), resid_full), f"resid differs, cuts {cuts}"
        assert torch.equal(state.view("o", w.batch, 256), o_full), f"o differs, cuts {cuts}"
    assert_close("ring resid vs oracle", f64(state.view("resid", w.batch, 256)), ref["resid"])
    # the appended K/V of layer 0 landed in the ring slot of the decoded position
    d, nkv = CFG.head_dim, CFG.n_kv
    rv = ring_pool.view(-1, 2, nkv, PAGE * d)
    fv = pool_full_after.view(-1, 2, nkv, PAGE * d)
    for b, c in enumerate(ctx):
        p = int(c) - 1
        rp, fp, t = int(ring_table[b, (p // PAGE) % R]), int(s.page_table[b, p // PAGE]), p % PAGE
        assert torch.equal(rv[rp, 0, :, t * d:(t + 1) * d], fv[fp, 0, :, t * d:(t + 1) * d]), f"K slot, seq {b}"
        assert torch.equal(rv[rp, 1, :, t::PAGE], fv[fp, 1, :, t::PAGE]), f"V slot, seq {b}"


def test_ring_long_contexts_against_oracle():
    """Contexts up to 20k tokens on a 9-page ring (window 128): the oracle reads
    the logical pages through t // 16 -> ring_table[b][(t // 16) % R]."""
    from paper_2609_14237_amd import runtime as Rt
    window = 128
    cfg = W.LayerCfg(hidden=512, n_q=8, n_kv=2, head_dim=128, ffn=512, window=window)
    ctx = np.array([1, 7, 128, 129, 300, 4097, 9999, 20000], dtype=np.int32)
    B = len(ctx)
    R = -(-window // PAGE) + 1
    say("ring long contexts, R =", R)
    ring_table, ring_pages_total = ring_alloc(ctx, R, seed=5)
    weights = {k: v.cuda() for k, v in gen.layer_weights(cfg, 3, 0, "cpu").items()}
    pool = gen.kv_pool(cfg, ring_pages_total, 3, 0, "cpu").cuda()
    pool_before = f64(pool)
    x = gen.activations(B, cfg.hidden, 3, "cpu").cuda()
    block = Rt.DeviceBlock((cfg,), [weights], [pool], ring_pages_total)
    ctx_t = torch.from_numpy(ctx).cuda()
    rt = torch.from_numpy(ring_table).cuda()
    batch = Rt.DeviceBatch(ctx_t, rt, ring_table=rt)
    state = Rt.DeviceState(block, batch, "cuda", fill=float("nan"))
    state.view("resid", B, cfg.hidden).copy_(x)
    Rt.run_partition(block, 0, 10, batch, state)
    torch.cuda.synchronize()
    # logical page table for the oracle: every logical page through the ring
    n_log = int(-(-int(ctx.max()) // PAGE))
    logical = np.array([[ring_table[b, lp % R] for lp in range(n_log)] for b in range(B)], dtype=np.int32)
    wts = {k: f64(v) for k, v in weights.items()}
    live = {"resid": f64(x)}
    pool_o = pool_before.copy()
    ref = O.run_ops([cfg], [wts], [pool_o], logical, ctx.copy(), live, 0, 10)
    assert_close("ring long o", f64(state.view("o", B, cfg.n_q * cfg.head_dim)), ref["o"])
    assert_close("ring long resid", f64(state.view("resid", B, cfg.hidden)), ref["resid"])
    # appended slots match the oracle's pool after its kv_append
    d = cfg.head_dim
    gv = f64(pool).reshape(-1, 2, cfg.n_kv, PAGE * d)
    ov = pool_o.reshape(-1, 2, cfg.n_kv, PAGE * d)
    for b, c in enumerate(ctx):
        p = int(c) - 1
        pg, t = int(ring_table[b, (p // PAGE) % R]), p % PAGE
        np.testing.assert_allclose(gv[pg, 0, :, t * d:(t + 1) * d], ov[pg, 0, :, t * d:(t + 1) * d], rtol=1e-2,
                                   atol=1e-2)
        np.testing.assert_allclose(gv[pg, 1, :, t::PAGE], ov[pg, 1, :, t::PAGE], rtol=1e-2, atol=1e-2)
