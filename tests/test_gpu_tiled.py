"""Tiled projection weights (ODS_WEIGHTS_TILED), through the C ABI.

- ods_tile_weight is a pure permutation: its output equals, bit for bit, a
  numpy rearrangement written from the layout's definition in include/ods.h.
- A layer run on tiled weights matches the oracle (which takes the row-major
  weights) to the same 1e-2 bar as the row-major path, at batches that take
  64-row streaming tiles (one and several per N tile: at these narrow widths
  a 256-row grid would leave most compute units idle), with N tails, split-K
  partials and the unfused gate_up (whose plain epilogue un-pairs the gate
  and up rows). The 256-row tile on tiled weights is covered by the wide-FFN
  parity test and at full size.
- Where the row-major path runs the same streaming kernel with the same
  split, both layouts give bit-identical results."""
import sys
from dataclasses import replace

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from workloads import gen
from harness import Setup, assert_close, f64, oracle_run, report, routing_check

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

from paper_2609_14237_amd import binding as B  # noqa: E402


def say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


def fresh(inp):
    out = dict(inp)
    out["pools"] = [p.copy() for p in inp["pools"]]
    return out


def tiled_reference(w: np.ndarray, out: int, gated: bool) -> np.ndarray:
    """[groups, rows, in] uint16 -> the tiled layout as a flat uint16 array:
    per slab, N tile and 64-wide K step, 128 rows x 8 chunks of 8 columns, with
    chunk c of row r at position c ^ (r % 8); rows past `out` are zero."""
    groups, _, k_in = w.shape
    per = 64 if gated else 128
    n_tiles, ks = -(-out // per), k_in // 64
    r = np.arange(128)
    n = np.arange(n_tiles)[:, None] * per + (r % 64 if gated else r)[None, :]  # [nt, 128]
    valid = n < out
    src_row = np.where(gated & (r[None, :] >= 64), out + n, n)
    src_row = np.where(valid, src_row, 0)
    pos = np.arange(8)
    chunk = pos[None, :] ^ (r[:, None] % 8)                                      # [128, 8] chunk at position
    cols = np.arange(ks)[:, None, None, None] * 64 + chunk[None, :, :, None] * 8 + np.arange(8)  # [ks,128,8,8]
    res = np.zeros((groups, n_tiles, ks, 128, 8, 8), dtype=np.uint16)
    for g in range(groups):
        rows = w[g][src_row]                                                      # [nt, 128, in]
        # rows[nt, r, cols[s, r, p, e]] -> [nt, s, r, p, e]
        gathered = np.take_along_axis(rows[:, None, :, :],
                                      np.broadcast_to(cols.reshape(1, ks, 128, 64), (n_tiles, ks, 128, 64)),
                                      axis=3).reshape(n_tiles, ks, 128, 8, 8)
        gathered[~np.broadcast_to(valid[:, None, :, None, None], gathered.shape)] = 0
        res[g] = gathered
    return res.reshape(-1)


@pytest.mark.parametrize("out,k_in,gated,groups", [(300, 192, 0, 1), (100, 128, 1, 1), (130, 64, 0, 3),
                                                   (70, 256, 1, 2), (4096, 128, 0, 1)])
def test_tile_weight_is_the_documented_permutation(out, k_in, gated, groups):
    say("tile weight", out, k_in, gated, groups)
    rows = (2 if gated else 1) * out
    gen_ = torch.Generator().manual_seed(out * 7 + k_in)
    src = torch.randint(-32768, 32767, (groups, rows, k_in), generator=gen_, dtype=torch.int32).to(torch.int16)
    n = B.ods_tiled_weight_bytes(out, k_in, gated, groups)
    dev_src = src.cuda()
    dst = torch.full((n // 2,), -1, dtype=torch.int16, device="cuda")
    st = B.ods_tile_weight(dev_src.data_ptr(), dst.data_ptr(), out, k_in, gated, groups,
                           torch.cuda.current_stream().cuda_stream)
    assert st == B.ODS_OK, B.ods_last_error()
    torch.cuda.synchronize()
    got = dst.cpu().numpy().view(np.uint16)
    ref = tiled_reference(src.numpy().view(np.uint16), out, bool(gated))
    np.testing.assert_array_equal(got, ref)


# hidden 576 and qkv width 960 leave N tails of the 128-row tiles; ffn 704 is 11 gated tiles
CFG = W.LayerCfg(hidden=576, n_q=9, n_kv=3, head_dim=64, ffn=704)


def _check(s, ref, cfg, batch):
    H = cfg.hidden
    assert_close("resid", f64(s.buf("resid", batch, H)), ref["resid"])
    assert_close("qkv", f64(s.buf("qkv", batch, cfg.qkv_dim)), ref["qkv"])
    assert_close("o", f64(s.buf("o", batch, cfg.n_q * cfg.head_dim)), ref["o"])
    assert_close("hn", f64(s.buf("hn", batch, H)), ref["hn"])


# hidden 1024 gives 16 K steps: split-K partials also for the unfused gate_up,
# whose split epilogue writes the un-paired gate and up columns
CFG_K16 = W.LayerCfg(hidden=1024, n_q=8, n_kv=2, head_dim=128, ffn=704)


@pytest.mark.parametrize("cfg,batch", [(CFG, 1), (CFG, 33), (CFG, 64), (CFG, 100), (CFG, 200),
                                       (CFG_K16, 1), (CFG_K16, 64), (CFG_K16, 150)])
def test_layer_on_tiled_weights_matches_oracle(cfg, batch):
    w = W.Workload("tiled", (cfg,), batch=batch, ctx_lo=1, ctx_hi=80)
    say("tiled layer, hidden", cfg.hidden, "batch", batch)
    s = Setup(w, seed=31, tiled=True)
    ref = oracle_run(fresh(s.oracle_inputs()), w.layers, 0, 10)
    s.reset_resid()
    s.run(0, 10)
    torch.cuda.synchronize()
    _check(s, ref, cfg, batch)
    act = O.silu(ref["gu"][:, :cfg.ffn]) * ref["gu"][:, cfg.ffn:]
    assert_close("act", f64(s.buf("act", batch, cfg.ffn)), act)
    # unfused gate_up: gate and up columns back in their row-major places
    s.reset_resid()
    for a, b in [(0, 2), (2, 5), (5, 6), (6, 8), (8, 10)]:
        s.run(a, b)
    torch.cuda.synchronize()
    assert_close("gu", f64(s.buf("gu", batch, 2 * cfg.ffn)), ref["gu"])
    _check(s, ref, cfg, batch)


@pytest.mark.parametrize("batch", [64, 200])
def test_tiled_and_row_major_agree_bitwise_on_the_streaming_kernel(batch):
    """qkv, o_proj and down run the streaming kernel with the same split on
    either layout at 33-64 rows (gate_up too past 128 rows), so the outputs are
    the same bits."""
    w = W.Workload("tiled_vs_rows", (CFG,), batch=batch, ctx_lo=1, ctx_hi=80)
    say("tiled vs row-major, batch", batch)
    out = {}
    for tiled in (False, True):
        s = Setup(w, seed=32, tiled=tiled)
        s.reset_resid()
        s.run(0, 6)
        torch.cuda.synchronize()
        out[tiled] = {"qkv": s.buf("qkv", batch, CFG.qkv_dim).clone(), "h": s.buf("resid", batch, CFG.hidden).clone()}
        s.run(6, 10)
        torch.cuda.synchronize()
        out[tiled]["y"] = s.buf("resid", batch, CFG.hidden).clone()
    for k in ("qkv", "h") + (("y",) if batch > 128 else ()):
        assert torch.equal(out[False][k].view(torch.int16), out[True][k].view(torch.int16)), k


MOE_TILED = W.Workload("moe_tiled", (W.LayerCfg(hidden=512, n_q=8, n_kv=2, head_dim=64, n_experts=16, top_k=4,
                                                moe_ffn=128),), batch=48, ctx_lo=1, ctx_hi=200,
                       router_std=512 ** -0.5)


@pytest.mark.parametrize("batch", [48, 300])
def test_moe_layer_on_tiled_weights(batch):
    """Expert slabs in tile order (64-row tiles at 12 rows per expert, 128-row
    tiles at 75), fused and unfused expert gate_up."""
    w = replace(MOE_TILED, batch=batch)
    cfg = w.layers[0]
    say("tiled moe, batch", batch)
    s = Setup(w, seed=33, tiled=True)
    inp = s.oracle_inputs()
    ref = oracle_run(fresh(inp), w.layers, 0, 14)
    pre = oracle_run(fresh(inp), w.layers, 0, 9)   # residual after the attention half, hn, logits
    for cut in ([], [11], [7, 12]):
        say("tiled moe cut", cut)
        s.reset_resid()
        bounds = [0] + cut + [14]
        for a, b in zip(bounds[:-1], bounds[1:]):
            s.run(a, b)
        torch.cuda.synchronize()
        ids = s.buf("topk_ids", batch, cfg.top_k).cpu().numpy()
        wts = f64(s.buf("topk_w", batch, cfg.top_k))
        logits = f64(s.buf("logits", batch, cfg.n_experts))
        forced, summary = routing_check(f"tiled moe batch {batch} cut {cut}", ids, wts, logits, ref, cfg.top_k)
        # every token's residual, the oracle taking the GPU's expert set where a near-tie made them differ
        live = {"resid": pre["resid"].copy(), "hn": pre["hn"], "topk_ids": forced,
                "topk_w": O.route_weights(ref["logits"], forced)}
        ref2 = oracle_run(fresh(inp), w.layers, 9, 14, live)
        assert_close(f"resid {cut}", f64(s.buf("resid", batch, cfg.hidden)), ref2["resid"])
    report(f"moe_tiled (batch {batch}) cuts: routing {summary}")


@pytest.mark.parametrize("batch", [300, 450])
@pytest.mark.parametrize("tiled", [False, True])
def test_moe_skewed_groups(batch, tiled):
    """The expert half [9, 14) on a routing where expert 0 takes 200 rows,
    expert 1 none (an empty group) and the rest share the remainder. At batch
    300 (75 rows per expert on average) the 128-row tile takes expert 0 in two
    passes; at batch 450 (112.5) the 256-row tile takes it in one. Every
    token's residual against the oracle on the same ids and weights, and bit
    for bit the same whether the expert GEMM gathers its rows of hn through
    perm (one range) or reads the materialised xp (cut after moe_permute)."""
    w = replace(MOE_TILED, batch=batch)
    cfg = w.layers[0]
    E, k, H = cfg.n_experts, cfg.top_k, cfg.hidden
    say("skewed moe groups, batch", batch, "tiled", tiled)
    s = Setup(w, seed=41, tiled=tiled)
    ids = gen.expert_choices(batch, E - 2, k, 41) + 2
    ids[:200, k - 1] = 0
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    rng = np.random.default_rng(41)
    wts = rng.uniform(0.1, 1.0, (batch, k)).astype(np.float32)
    wts /= wts.sum(axis=1, keepdims=True)
    counts = np.bincount(ids.ravel(), minlength=E)
    assert counts[0] == 200 and counts[1] == 0
    hn = gen.live_tensor((batch, H), 41, 3, "cuda")
    s.reset_resid()
    s.buf("hn", batch, H).copy_(hn)
    s.buf("topk_ids", batch, k).copy_(torch.from_numpy(ids))
    s.buf("topk_w", batch, k).copy_(torch.from_numpy(wts))
    s.run(9, 14)
    torch.cuda.synchronize()
    fused = s.buf("resid", batch, H).clone()
    # cut after moe_permute: xp is materialised and the expert GEMM reads it
    # instead of gathering hn rows through perm; the result must not change
    s.reset_resid()
    s.run(9, 10)
    s.run(10, 14)
    torch.cuda.synchronize()
    xp = s.buf("xp", batch * k, H)
    perm = s.buf("perm", batch * k).long()
    assert torch.equal(xp, hn[perm // k])
    assert torch.equal(s.buf("resid", batch, H).view(torch.int16), fused.view(torch.int16))
    inp = s.oracle_inputs()
    live = {"resid": inp["x"].copy(), "hn": f64(hn), "topk_ids": ids.astype(np.int64),
            "topk_w": wts.astype(np.float64)}
    ref = oracle_run(fresh(inp), w.layers, 9, 14, live)
    e = assert_close(f"skewed resid batch {batch}", f64(s.buf("resid", batch, H)), ref["resid"])
    report(f"moe skewed groups (batch {batch}, rows per expert {counts.min()}..{counts.max()}, "
           f"{'tiled' if tiled else 'row-major'}): resid {e:.2e}")
