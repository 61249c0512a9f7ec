"""Degenerate inputs of the decode path on the GPU, through the C ABI.

- An empty batch (batch = 0) enqueues nothing: every live buffer, the
  workspace-fed outputs and the KV pool keep their bytes, for whole layers,
  the stage entry points and a graph captured at batch 0.
- Rows with no context (ctx_lens < 1) are no-ops for KV append and attention:
  their attention output is exactly zero, so the attention stage leaves their
  residual rows unchanged; the pool keeps every byte outside the slots the
  other rows append; the other rows match the oracle run on those rows alone.
- attn_core at its batch limit (4096 sequences, ragged short contexts, so the
  per-sequence prefix in LDS is at its largest): sampled rows match the oracle,
  and rows whose whole context fits one wave's range come out of the attention
  kernel directly while long ones go through the merge."""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from workloads import gen
from harness import Setup, assert_close, f64, oracle_run

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)


def say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


def snapshot(s):
    bufs = {k: v.clone() for k, v in s.state.buffers.items()}
    pools = [p.clone() for p in s.pools]
    return bufs, pools


def assert_unchanged(s, snap):
    bufs, pools = snap
    for k, v in s.state.buffers.items():
        assert torch.equal(v.view(torch.uint8), bufs[k].view(torch.uint8)), k
    for l, p in enumerate(s.pools):
        assert torch.equal(p.view(torch.uint8), pools[l].view(torch.uint8)), f"pool {l}"


@pytest.mark.parametrize("wl", [W.TINY, W.Workload("moe_e", (W.LayerCfg(hidden=256, n_q=4, n_kv=2, head_dim=64,
                                                                        n_experts=8, top_k=2, moe_ffn=128),),
                                                   batch=6, ctx_lo=1, ctx_hi=90)],
                         ids=["dense", "moe"])
def test_empty_batch_enqueues_nothing(wl):
    say("empty batch", wl.name)
    s = Setup(wl, seed=5)
    s.reset_resid()
    torch.cuda.synchronize()
    snap = snapshot(s)
    empty = s.R.DeviceBatch(s.batch.ctx_lens[:0], s.batch.page_table[:0])
    assert empty.batch == 0
    n = wl.n_ops
    s.R.run_partition(s.block, 0, n, empty, s.state)
    s.R.run_partition(s.block, 4, 5, empty, s.state)
    s.R.attn_stage(s.block, 0, empty, s.state)
    s.R.ffn_stage(s.block, 0, empty, s.state)
    torch.cuda.synchronize()
    assert_unchanged(s, snap)
    # a graph captured at batch 0 holds no work: replays leave every byte alone
    g = s.R.PartitionGraph(s.block, 0, n, empty, s.state)
    for _ in range(2):
        g.launch()
        torch.cuda.synchronize()
    g.close()
    assert_unchanged(s, snap)


ZERO_CFG = W.LayerCfg(hidden=256, n_q=8, n_kv=2, head_dim=128, ffn=256)
ZERO_CTX = [0, 5, 0, 40, 17, 0, 300, 1, -3, 64, 16, 0]


def appended_slots_mask(s, cfg, rows):
    """True at the pool bytes (as a [P, 2, n_kv, 16 d] view) of the slot each
    listed row appends: K is slot-major [16][d] per KV head, V is [d][16]."""
    d, nkv = cfg.head_dim, cfg.n_kv
    mask = torch.zeros(s.pool_pages, 2, nkv, 16 * d, dtype=torch.bool, device="cuda")
    for b in rows:
        p = int(s.ctx[b]) - 1
        page, slot = int(s.page_table[b, p // 16]), p % 16
        mask[page, 0, :, slot * d:(slot + 1) * d] = True
        mask[page, 1, :, slot::16] = True
    return mask


@pytest.mark.parametrize("split_pages", [0, 2])
def test_rows_without_context(split_pages):
    say("rows with ctx < 1, split", split_pages)
    cfg = ZERO_CFG
    w = W.Workload("zero_ctx", (cfg,), batch=len(ZERO_CTX), ctx_lo=1, ctx_hi=300)
    # pages are allocated as for a context of 1 (the allocator takes contexts >= 1);
    # the device sees the true contexts
    s = Setup(w, seed=41, ctx=np.maximum(np.asarray(ZERO_CTX), 1).astype(np.int32), split_pages=split_pages)
    s.batch.ctx_lens.copy_(torch.tensor(ZERO_CTX, dtype=torch.int32))
    live_rows = [b for b, c in enumerate(ZERO_CTX) if c >= 1]
    dead_rows = [b for b, c in enumerate(ZERO_CTX) if c < 1]
    ref = oracle_run(s.oracle_inputs(live_rows), w.layers, 0, 10)
    pool0 = s.pools[0].clone()
    B, H = len(ZERO_CTX), cfg.hidden
    s.reset_resid()
    s.run(0, 6)
    torch.cuda.synchronize()
    dead = torch.tensor(dead_rows, device="cuda")
    o = s.buf("o", B, cfg.n_q * cfg.head_dim)
    assert torch.count_nonzero(o.index_select(0, dead).float()) == 0
    assert torch.equal(s.buf("resid", B, H).index_select(0, dead).view(torch.int16),
                       s.x.index_select(0, dead).view(torch.int16))
    s.run(6, 10)
    torch.cuda.synchronize()
    live = torch.tensor(live_rows, device="cuda")
    for name, width in (("resid", H), ("o", cfg.n_q * cfg.head_dim), ("hn", H)):
        assert_close(name, f64(s.buf(name, B, width).index_select(0, live)), ref[name])
    mask = appended_slots_mask(s, cfg, live_rows)
    view = lambda p: p.view(s.pool_pages, 2, cfg.n_kv, 16 * cfg.head_dim).view(torch.int16)
    assert torch.equal(view(s.pools[0])[~mask], view(pool0)[~mask])
    # the appended slots hold the rows' rotated k and their v
    assert not torch.equal(view(s.pools[0])[mask], view(pool0)[mask])


LIMIT_CFG = W.LayerCfg(hidden=256, n_q=8, n_kv=2, head_dim=128, ffn=256)


def test_attention_at_the_batch_limit():
    B = 4096
    say("attn_core at batch", B)
    w = W.Workload("attn_limit", (LIMIT_CFG,), batch=B, ctx_lo=1, ctx_hi=70, seed=7)
    ctx = gen.contexts(w, 7).copy()
    ctx[-1] = 2000          # one long sequence at the end: split over several waves, merged
    ctx[B // 2] = 900
    s = Setup(w, seed=7, ctx=ctx)
    qkv = gen.live_tensor((B, LIMIT_CFG.qkv_dim), 7, 1, "cuda")
    s.buf("qkv", B, LIMIT_CFG.qkv_dim).copy_(qkv)
    s.run(4, 5)
    torch.cuda.synchronize()
    rng = np.random.default_rng(7)
    rows = np.unique(np.concatenate([[0, 1, B // 2, B - 2, B - 1], rng.choice(B, 59, replace=False)]))
    inp = s.oracle_inputs(rows)
    live = {"qkv": f64(qkv)[rows]}
    from oracle import run_ops
    ref = run_ops([LIMIT_CFG], inp["weights"], inp["pools"], inp["page_table"], inp["ctx"], live, 4, 5)["o"]
    o = f64(s.buf("o", B, LIMIT_CFG.n_q * LIMIT_CFG.head_dim))[rows]
    for i, b in enumerate(rows):
        assert_close(f"o row {b} ctx {ctx[b]}", o[i], ref[i])
