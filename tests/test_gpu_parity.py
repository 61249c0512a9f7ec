"""GPU parity of the HIP decode path against the CPU oracle, through the C ABI.

Bar: every floating-point live buffer within max |gpu - oracle| / max |oracle|
<= 1e-2 (bf16 storage, fp32 accumulation); page tables, routing ids and the
expert permutation bit-exact. Shapes here are small enough for the oracle to
run whole, and still span several GEMM tiles, split-K work items and ragged
page tails."""
import copy
import sys
from dataclasses import replace

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from workloads import gen
from harness import Setup, assert_close, f64, oracle_run, rel_err, report, routing_check

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)


def say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


def fresh(inp):
    out = dict(inp)
    out["pools"] = [p.copy() for p in inp["pools"]]
    return out


def n_ops(cfgs):
    return sum(14 if c.n_experts else 10 for c in cfgs)


# ---------------------------------------------------------------- tiny layer

@pytest.fixture(scope="module")
def tiny():
    say("tiny setup")
    s = Setup(W.TINY, seed=0)
    inp = s.oracle_inputs()
    ref = oracle_run(fresh(inp), W.TINY.layers, 0, 10)
    return s, inp, ref


def _check_layer_buffers(s, ref, cfg, B):
    H, d = cfg.hidden, cfg.head_dim
    assert_close("resid", f64(s.buf("resid", B, H)), ref["resid"])
    assert_close("xn", f64(s.buf("xn", B, H)), ref["xn"])
    assert_close("qkv", f64(s.buf("qkv", B, cfg.qkv_dim)), ref["qkv"])
    assert_close("o", f64(s.buf("o", B, cfg.n_q * d)), ref["o"])
    assert_close("hn", f64(s.buf("hn", B, H)), ref["hn"])


def test_tiny_colocated_layer(tiny):
    s, inp, ref = tiny
    say("tiny colocated [0,10)")
    s.reset_resid()
    s.run(0, 10)
    torch.cuda.synchronize()
    _check_layer_buffers(s, ref, W.TINY.layers[0], 4)
    cfg = W.TINY.layers[0]
    act = O.silu(ref["gu"][:, :cfg.ffn]) * ref["gu"][:, cfg.ffn:]
    assert_close("act", f64(s.buf("act", 4, cfg.ffn)), act)


def test_tiny_appended_slot(tiny):
    s, inp, ref = tiny
    say("tiny kv slot after [0,4)")
    s.reset_resid()
    s.run(0, 4)
    torch.cuda.synchronize()
    cfg = W.TINY.layers[0]
    nq, nkv, d = cfg.n_q, cfg.n_kv, cfg.head_dim
    qkv = s.buf("qkv", 4, cfg.qkv_dim)
    pool = s.pools[0].view(-1, 2, nkv, 16 * d)
    ref_pool = oracle_run(fresh(inp), W.TINY.layers, 0, 4)
    for b, c in enumerate(s.ctx):
        p = int(c) - 1
        page = int(s.page_table[b, p // 16])
        k = pool[page, 0, :, (p % 16) * d:(p % 16 + 1) * d]
        v = pool[page, 1, :, (p % 16)::16]
        # the cache holds exactly the bf16 values the rope step produced
        assert torch.equal(k.reshape(-1), qkv[b, nq * d:(nq + nkv) * d])
        assert torch.equal(v.reshape(-1), qkv[b, (nq + nkv) * d:])
        assert_close("k slot", f64(k), ref_pool["qkv"][b, nq * d:(nq + nkv) * d].reshape(nkv, d))


def test_tiny_every_cut_composes(tiny):
    s, inp, ref = tiny
    cfg = W.TINY.layers[0]
    cuts = [[c] for c in range(1, 10)] + [[a, b] for a in range(1, 10) for b in range(a + 1, 10)]
    for cut in cuts:
        say("tiny cut", cut)
        s.reset_resid()
        bounds = [0] + cut + [10]
        for a, b in zip(bounds[:-1], bounds[1:]):
            s.run(a, b)
        torch.cuda.synchronize()
        assert_close(f"resid cut {cut}", f64(s.buf("resid", 4, cfg.hidden)), ref["resid"])
        assert_close(f"o cut {cut}", f64(s.buf("o", 4, cfg.n_q * cfg.head_dim)), ref["o"])


def test_tiny_stage_entry_points(tiny):
    s, inp, ref = tiny
    say("tiny attn_stage + ffn_stage")
    s.reset_resid()
    s.R.attn_stage(s.block, 0, s.batch, s.state)
    h = s.buf("resid", 4, 256).clone()
    s.R.ffn_stage(s.block, 0, s.batch, s.state)
    torch.cuda.synchronize()
    ref_h = oracle_run(fresh(inp), W.TINY.layers, 0, 6)["resid"]
    assert_close("h after attention stage", f64(h), ref_h)
    assert_close("resid after ffn stage", f64(s.buf("resid", 4, 256)), ref["resid"])


# ---------------------------------------------------------------- attention core alone

ATTN_CFG = W.LayerCfg(hidden=256, n_q=8, n_kv=2, head_dim=128, ffn=256)


def _attn_setup(ctx, window=0, split_pages=0, seed=3, alloc_seed=None, nan_trap=False, cfg=ATTN_CFG):
    cfg = replace(cfg, window=window)
    w = W.Workload("attn", (cfg,), batch=len(ctx), ctx_lo=1, ctx_hi=int(max(ctx)), seed=seed)
    s = Setup(w, seed=seed, ctx=np.asarray(ctx, dtype=np.int32), split_pages=split_pages,
              alloc_seed=alloc_seed, nan_trap=nan_trap)
    qkv = gen.live_tensor((len(ctx), cfg.qkv_dim), seed, 1, "cuda")
    s.buf("qkv", len(ctx), cfg.qkv_dim).copy_(qkv)
    return s, cfg, qkv


def _attn_ref(s, cfg, qkv, rows=None):
    inp = s.oracle_inputs(rows)
    live = {"qkv": f64(qkv) if rows is None else f64(qkv)[rows]}
    return O.run_ops([cfg], inp["weights"], inp["pools"], inp["page_table"], inp["ctx"], live, 4, 5)["o"]


RAGGED = [1, 2, 15, 16, 17, 31, 33, 100, 255, 256, 257, 700, 1025, 2000]


@pytest.mark.parametrize("window", [0, 1, 16, 17, 100])
@pytest.mark.parametrize("split_pages", [0, 1, 3])
def test_attention_core_matches_oracle(window, split_pages):
    say("attn_core window", window, "split", split_pages)
    s, cfg, qkv = _attn_setup(RAGGED, window, split_pages)
    s.run(4, 5)
    torch.cuda.synchronize()
    o = f64(s.buf("o", len(RAGGED), cfg.n_q * cfg.head_dim))
    ref = _attn_ref(s, cfg, qkv)
    for b in range(len(RAGGED)):
        assert_close(f"o row {b} ctx {RAGGED[b]}", o[b], ref[b])


@pytest.mark.parametrize("head_dim,n_q,n_kv", [(64, 4, 2), (128, 32, 4), (128, 16, 16), (64, 16, 1)])
def test_attention_core_head_shapes(head_dim, n_q, n_kv):
    say("attn_core shapes", head_dim, n_q, n_kv)
    cfg = W.LayerCfg(hidden=256, n_q=n_q, n_kv=n_kv, head_dim=head_dim, ffn=256)
    s, cfg, qkv = _attn_setup([5, 16, 129, 600], cfg=cfg)
    s.run(4, 5)
    torch.cuda.synchronize()
    o = f64(s.buf("o", 4, cfg.n_q * cfg.head_dim))
    ref = _attn_ref(s, cfg, qkv)
    for b in range(4):
        assert_close(f"o row {b}", o[b], ref[b])


def test_attention_softmax_rows_sum_to_one():
    say("attn V == 1")
    s, cfg, qkv = _attn_setup(RAGGED, 0, 2)
    s.pools[0].view(-1, 2, cfg.n_kv, 16 * cfg.head_dim)[:, 1] = 1.0
    s.run(4, 5)
    torch.cuda.synchronize()
    o = f64(s.buf("o", len(RAGGED), cfg.n_q * cfg.head_dim))
    assert np.abs(o - 1.0).max() <= 2 ** -8


def test_attention_single_key_returns_its_value_row():
    say("attn ctx == 1")
    s, cfg, qkv = _attn_setup([1, 1, 1])
    s.run(4, 5)
    torch.cuda.synchronize()
    o = s.buf("o", 3, cfg.n_q * cfg.head_dim)
    d, group = cfg.head_dim, cfg.n_q // cfg.n_kv
    pool = s.pools[0].view(-1, 2, cfg.n_kv, 16 * d)
    for b in range(3):
        page = int(s.page_table[b, 0])
        for h in range(cfg.n_q):
            v0 = pool[page, 1, h // group, 0::16][:d]
            assert torch.equal(o[b, h * d:(h + 1) * d], v0)


def test_attention_window_covering_context_equals_full():
    say("attn window >= ctx")
    outs = []
    for window in (0, 2000, 5000):
        s, cfg, qkv = _attn_setup(RAGGED, window, 3)   # same split size so the merge order matches
        s.run(4, 5)
        torch.cuda.synchronize()
        outs.append(s.buf("o", len(RAGGED), cfg.n_q * cfg.head_dim).clone())
    assert torch.equal(outs[0], outs[1]) and torch.equal(outs[0], outs[2])


def test_attention_page_shuffle_invariance():
    say("attn page shuffle")
    outs = []
    for alloc_seed in (11, 12):
        s, cfg, qkv = _attn_setup(RAGGED, 0, 0, alloc_seed=alloc_seed)
        # write one logical cache (drawn per token) through each page table
        d, nkv = cfg.head_dim, cfg.n_kv
        pool = s.pools[0].view(-1, 2, nkv, 16, d)
        for b, c in enumerate(RAGGED):
            kv = gen.normal_bf16((int(c), 2, nkv, d), 1000 + b, "cuda")
            for t0 in range(0, int(c), 16):
                page = int(s.page_table[b, t0 // 16])
                n = min(16, int(c) - t0)
                pool[page, 0, :, :n] = kv[t0:t0 + n, 0].transpose(0, 1)
                vblk = s.pools[0].view(-1, 2, nkv, d, 16)
                vblk[page, 1, :, :, :n] = kv[t0:t0 + n, 1].permute(1, 2, 0)
        s.run(4, 5)
        torch.cuda.synchronize()
        outs.append(s.buf("o", len(RAGGED), cfg.n_q * d).clone())
    assert torch.equal(outs[0], outs[1])


def test_attention_ignores_stale_slots_and_pages():
    say("attn NaN traps")
    outs = []
    for trap in (False, True):
        s, cfg, qkv = _attn_setup(RAGGED, 0, 3, nan_trap=trap)
        s.run(4, 5)
        torch.cuda.synchronize()
        outs.append(s.buf("o", len(RAGGED), cfg.n_q * cfg.head_dim).clone())
    assert torch.isfinite(outs[1].float()).all()
    assert torch.equal(outs[0], outs[1])


def test_attention_split_size_invariance():
    say("attn split sizes")
    outs = []
    for sp in (1, 2, 7, 64):
        s, cfg, qkv = _attn_setup(RAGGED, 0, sp)
        s.run(4, 5)
        torch.cuda.synchronize()
        outs.append(f64(s.buf("o", len(RAGGED), cfg.n_q * cfg.head_dim)))
    for o in outs[1:]:
        assert rel_err(o, outs[0]) <= 8e-3


# ---------------------------------------------------------------- routing and permutation

MOE_SMALL = W.Workload("moe_small", (W.LayerCfg(hidden=512, n_q=8, n_kv=2, head_dim=64, n_experts=64, top_k=8,
                                                moe_ffn=96),), batch=40, ctx_lo=1, ctx_hi=300,
                       router_std=512 ** -0.5)


def test_topk_routing_bit_exact():
    say("topk on drawn logits")
    w = replace(MOE_SMALL, batch=512)
    s = Setup(w, seed=5)
    cfg = w.layers[0]
    logits = gen.router_logits(512, 64, 5, "cuda")
    logits[3, 10] = logits[3, 20] = logits[3].max() + 1.0   # exact tie at the top
    s.buf("logits", 512, 64).copy_(logits)
    s.run(8, 9)
    torch.cuda.synchronize()
    ids = s.buf("topk_ids", 512, 8).cpu().numpy()
    wts = f64(s.buf("topk_w", 512, 8))
    ref_ids, ref_w = O.topk_route(f64(logits), 8)
    np.testing.assert_array_equal(ids, ref_ids)
    assert ids[3, 0] == 10 and ids[3, 1] == 20
    assert np.abs(wts - ref_w).max() <= 1e-6


def test_permute_bit_exact():
    say("permute on drawn ids")
    w = replace(MOE_SMALL, batch=512)
    s = Setup(w, seed=6)
    ids = gen.expert_choices(512, 64, 8, 6)
    s.buf("topk_ids", 512, 8).copy_(torch.from_numpy(ids))
    hn = gen.live_tensor((512, 512), 6, 2, "cuda")
    s.buf("hn", 512, 512).copy_(hn)
    s.run(9, 10)
    torch.cuda.synchronize()
    perm, off, slot = O.moe_permute(ids, 64)
    np.testing.assert_array_equal(s.buf("perm", 4096).cpu().numpy(), perm)
    np.testing.assert_array_equal(s.buf("expert_off", 65).cpu().numpy(), off)
    np.testing.assert_array_equal(s.buf("slot_pos", 4096).cpu().numpy(), slot)
    xp = s.buf("xp", 4096, 512)
    assert torch.equal(xp, hn[torch.from_numpy(perm // 8).long().cuda()])


def test_moe_layer_small_and_cuts():
    w = MOE_SMALL
    cfg = w.layers[0]
    s = Setup(w, seed=7)
    inp = s.oracle_inputs()
    ref = oracle_run(fresh(inp), w.layers, 0, 14)
    pre = oracle_run(fresh(inp), w.layers, 0, 9)   # residual after the attention half, hn, logits
    rng = np.random.default_rng(7)
    cut_sets = [[], [6], [3, 5], [7], [8], [9], [10], [11], [12], [13]] + \
               [sorted(rng.choice(np.arange(1, 14), 3, replace=False).tolist()) for _ in range(4)]
    first_logits = None
    for cut in cut_sets:
        say("moe cut", cut)
        s.reset_resid()
        bounds = [0] + cut + [14]
        for a, b in zip(bounds[:-1], bounds[1:]):
            s.run(a, b)
        torch.cuda.synchronize()
        # the router's split-K sum is the same whether the reduce kernel or the
        # top-k kernel (router and top-k in one range) does it: bit for bit
        raw = s.buf("logits", w.batch, 64).clone()
        if first_logits is None:
            first_logits = raw
        assert torch.equal(raw.view(torch.int32), first_logits.view(torch.int32)), f"logits differ at cut {cut}"
        ids = s.buf("topk_ids", w.batch, cfg.top_k).cpu().numpy()
        wts = f64(s.buf("topk_w", w.batch, cfg.top_k))
        logits = f64(raw)
        forced, summary = routing_check(f"moe cut {cut}", ids, wts, logits, ref, cfg.top_k)
        assert_close(f"logits {cut}", logits, ref["logits"])
        # the residual of every token, with the oracle evaluated on the GPU's
        # expert set where a near-tie made the sets differ
        live = {"resid": pre["resid"].copy(), "hn": pre["hn"], "topk_ids": forced,
                "topk_w": O.route_weights(ref["logits"], forced)}
        ref2 = oracle_run(fresh(inp), w.layers, 9, 14, live)
        assert_close(f"topk_w {cut}", wts, O.route_weights(ref["logits"], ids))
        assert_close(f"resid {cut}", f64(s.buf("resid", w.batch, cfg.hidden)), ref2["resid"])
    report(f"moe_small (batch {w.batch}) cuts: routing {summary}")


MOE_K8 = W.Workload("moe_k8", (W.LayerCfg(hidden=520, n_q=8, n_kv=2, head_dim=64, n_experts=16, top_k=4,
                                           moe_ffn=136),), batch=40, ctx_lo=1, ctx_hi=200, router_std=520 ** -0.5)


def test_moe_layer_hidden_not_multiple_of_64():
    """hidden 520 and expert width 136 (multiples of 8, not of 64): the expert
    GEMMs take the register-staged large-M tile, so moe_permute gathers xp
    even when expert_gate_up shares its range; the whole layer and the cut
    after moe_permute against the oracle, and bit for bit against each other."""
    w = MOE_K8
    cfg = w.layers[0]
    s = Setup(w, seed=9)
    inp = s.oracle_inputs()
    ref = oracle_run(fresh(inp), w.layers, 0, 14)
    pre = oracle_run(fresh(inp), w.layers, 0, 9)
    outs = []
    for cut in ([], [10]):
        say("moe hidden 520 cut", cut)
        s.reset_resid()
        bounds = [0] + cut + [14]
        for a, b in zip(bounds[:-1], bounds[1:]):
            s.run(a, b)
        torch.cuda.synchronize()
        ids = s.buf("topk_ids", w.batch, cfg.top_k).cpu().numpy()
        wts = f64(s.buf("topk_w", w.batch, cfg.top_k))
        logits = f64(s.buf("logits", w.batch, cfg.n_experts))
        forced, summary = routing_check(f"moe hidden 520 cut {cut}", ids, wts, logits, ref, cfg.top_k)
        live = {"resid": pre["resid"].copy(), "hn": pre["hn"], "topk_ids": forced,
                "topk_w": O.route_weights(ref["logits"], forced)}
        ref2 = oracle_run(fresh(inp), w.layers, 9, 14, live)
        out = s.buf("resid", w.batch, cfg.hidden).clone()
        assert_close(f"resid {cut}", f64(out), ref2["resid"])
        outs.append(out)
    assert torch.equal(outs[0].view(torch.int16), outs[1].view(torch.int16))
    report(f"moe_k8 (hidden 520, batch {w.batch}): routing {summary}")


# ---------------------------------------------------------------- hybrid block and real shapes

HYBRID_SMALL = W.Workload("hybrid_small",
                          tuple([W.LayerCfg(hidden=512, n_q=8, n_kv=2, head_dim=128, ffn=1376, window=40)] * 3 +
                                [W.LayerCfg(hidden=512, n_q=8, n_kv=2, head_dim=128, ffn=1376)]),
                          batch=8, ctx_lo=20, ctx_hi=500)


def test_hybrid_block_random_cuts():
    w = HYBRID_SMALL
    s = Setup(w, seed=8)
    inp = s.oracle_inputs()
    ref = oracle_run(fresh(inp), w.layers, 0, 40)
    rng = np.random.default_rng(8)
    cut_sets = [[], [6, 16, 26, 36], [3, 5, 13, 15, 23, 25, 33, 35]] + \
               [sorted(rng.choice(np.arange(1, 40), int(rng.integers(1, 7)), replace=False).tolist())
                for _ in range(5)]
    for cut in cut_sets:
        say("hybrid cut", cut)
        s.reset_resid()
        bounds = [0] + cut + [40]
        for a, b in zip(bounds[:-1], bounds[1:]):
            s.run(a, b)
        torch.cuda.synchronize()
        assert_close(f"resid {cut}", f64(s.buf("resid", w.batch, 512)), ref["resid"])
        assert_close(f"o {cut}", f64(s.buf("o", w.batch, 1024)), ref["o"])


def test_dense_8b_shape_small_batch():
    w = replace(W.DENSE_8B_B64, batch=5)
    say("dense 8B shape, batch 5")
    s = Setup(w, seed=9)
    inp = s.oracle_inputs()
    ref = oracle_run(fresh(inp), w.layers, 0, 10)
    s.reset_resid()
    s.run(0, 6)
    s.run(6, 10)
    torch.cuda.synchronize()
    _check_layer_buffers(s, ref, w.layers[0], 5)


# ---------------------------------------------------------------- GEMM tile paths

@pytest.mark.parametrize("batch", [65, 100, 128, 200, 300])
def test_layer_across_gemm_tile_paths(batch):
    """Batches above 64 rows take the 512-thread large-M GEMM tiles up to 128
    rows; past 128 the streaming kernel runs every GEMM whose K is a multiple
    of 64, on 64-row tiles at these narrow widths, and down (K = 688) stays on
    the 256-row large-M tile. F = 688 leaves K and SiLU-N tails, H = 640 an N
    tail of the 128-column tile."""
    cfg = W.LayerCfg(hidden=640, n_q=10, n_kv=2, head_dim=64, ffn=688)
    w = W.Workload("gemm_paths", (cfg,), batch=batch, ctx_lo=1, ctx_hi=70)
    say("gemm tile paths, batch", batch)
    s = Setup(w, seed=12)
    inp = s.oracle_inputs()
    ref = oracle_run(fresh(inp), w.layers, 0, 10)
    s.reset_resid()
    s.run(0, 10)
    torch.cuda.synchronize()
    _check_layer_buffers(s, ref, cfg, batch)
    act = O.silu(ref["gu"][:, :cfg.ffn]) * ref["gu"][:, cfg.ffn:]
    assert_close("act", f64(s.buf("act", batch, cfg.ffn)), act)
    # unfused gate_up (bf16 epilogue) and the standalone SiLU
    s.reset_resid()
    s.run(0, 8)
    s.run(8, 10)
    torch.cuda.synchronize()
    assert_close("gu", f64(s.buf("gu", batch, 2 * cfg.ffn)), ref["gu"])
    assert_close("resid (split at silu)", f64(s.buf("resid", batch, cfg.hidden)), ref["resid"])


@pytest.mark.parametrize("ffn,tiled", [(9000, False), (8960, True)], ids=["rows", "tiled"])
def test_wide_gated_ffn_on_256_row_stream_tiles(ffn, tiled):
    """An FFN wide enough to fill the compute units with 256-row streaming
    tiles at 200 rows: 141 gated tiles of 64 columns (row-major F = 9000
    leaves a 40-column tail; tiled F = 8960 gives 140) for gate_up + SiLU,
    and as many 128-column tiles (an 80-column tail row-major) for the
    unfused gate_up's bf16 epilogue."""
    cfg = W.LayerCfg(hidden=512, n_q=8, n_kv=2, head_dim=64, ffn=ffn)
    w = W.Workload("wide_ffn", (cfg,), batch=200, ctx_lo=1, ctx_hi=60)
    say("wide gated FFN on 256-row stream tiles, batch 200, ffn", ffn, "tiled" if tiled else "rows")
    s = Setup(w, seed=14, tiled=tiled)
    ref = oracle_run(fresh(s.oracle_inputs()), w.layers, 0, 10)
    s.reset_resid()
    s.run(0, 10)
    torch.cuda.synchronize()
    _check_layer_buffers(s, ref, cfg, 200)
    act = O.silu(ref["gu"][:, :cfg.ffn]) * ref["gu"][:, cfg.ffn:]
    assert_close("act", f64(s.buf("act", 200, cfg.ffn)), act)
    s.reset_resid()
    s.run(0, 8)
    s.run(8, 10)
    torch.cuda.synchronize()
    assert_close("gu", f64(s.buf("gu", 200, 2 * cfg.ffn)), ref["gu"])
    assert_close("resid (split at silu)", f64(s.buf("resid", 200, cfg.hidden)), ref["resid"])


@pytest.mark.parametrize("batch", [33, 47, 64])
def test_layer_on_64_row_stream_tiles(batch):
    """33 to 64 rows send qkv, o_proj and down (K a multiple of 64) to the
    64-row streaming tile; H = 704 and qkv N = 832 leave N tails of the
    128-column tile, and split-K partials are reduced both fused into RoPE
    (qkv) and on their own (o_proj, down)."""
    cfg = W.LayerCfg(hidden=704, n_q=11, n_kv=1, head_dim=64, ffn=768)
    w = W.Workload("stream64", (cfg,), batch=batch, ctx_lo=1, ctx_hi=90)
    say("64-row stream tiles, batch", batch)
    s = Setup(w, seed=21)
    inp = s.oracle_inputs()
    ref = oracle_run(fresh(inp), w.layers, 0, 10)
    s.reset_resid()
    s.run(0, 10)
    torch.cuda.synchronize()
    _check_layer_buffers(s, ref, cfg, batch)
    # every stage boundary: the unfused qkv and o_proj outputs
    s.reset_resid()
    for a, b in [(0, 2), (2, 3), (3, 5), (5, 6), (6, 10)]:
        s.run(a, b)
    torch.cuda.synchronize()
    _check_layer_buffers(s, ref, cfg, batch)


# ---------------------------------------------------------------- fusions

def test_qkv_split_reduce_fused_into_rope_is_bit_exact():
    """With split-K on the qkv projection and RoPE in the same range, the RoPE /
    KV-append kernel sums the partials itself. Same order, same rounding: the
    fused range [0, 4) must leave qkv and the KV pool byte-identical to the
    unfused cuts [0, 2) + [2, 4), and the layer must match the oracle."""
    from paper_2609_14237_amd import binding as Bd
    cfg = W.LayerCfg(hidden=2048, n_q=16, n_kv=4, head_dim=128, ffn=1024)
    w = W.Workload("fused_qkv", (cfg,), batch=48, ctx_lo=1, ctx_hi=200)
    assert Bd.lib.ods_workspace_bytes  # library loaded
    say("qkv reduce fused into rope")
    s = Setup(w, seed=31)
    inp = s.oracle_inputs()
    ref = oracle_run(fresh(inp), w.layers, 0, 10)
    pool0 = s.pools[0].clone()
    s.reset_resid()
    s.run(0, 4)
    torch.cuda.synchronize()
    qkv_fused, pool_fused = s.buf("qkv", w.batch, cfg.qkv_dim).clone(), s.pools[0].clone()
    s.pools[0].copy_(pool0)
    s.reset_resid()
    s.run(0, 2)
    s.run(2, 4)
    torch.cuda.synchronize()
    assert torch.equal(s.buf("qkv", w.batch, cfg.qkv_dim), qkv_fused)
    assert torch.equal(s.pools[0], pool_fused)
    s.pools[0].copy_(pool0)
    s.reset_resid()
    s.run(0, 10)
    torch.cuda.synchronize()
    _check_layer_buffers(s, ref, cfg, w.batch)
