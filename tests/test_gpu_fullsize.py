"""Parity at the full evaluated sizes, in the launch configuration the
benchmark times (per layer: ops [0,4), [4,5), [5,6), [6,end); tiled weights,
and row-major weights as well). The oracle
recomputes a handful of sampled sequences one by one (their pages only).

Two kinds of check:
  * stage parity: each stage (attention [0,6), FFN [6,end), core attention
    [3,5)) starts from the same freshly drawn live set on both sides and its
    output live set must match to 1e-2 (max |gpu - oracle| / max |oracle| per
    row);
  * chained block: the whole block runs as the benchmark runs it; bf16
    rounding of the live buffers at every layer compounds, so the final
    residual of an L-layer block is held to max(1e-2, 5e-3 * L) and the
    attention output of its last layer, an intermediate that inherits the
    rounding of q, to twice that.
The FFN stage also checks its SiLU-gated activation (an intermediate the
stage materialises), since the residual it returns is dominated by its input.
The page table is compared bit-exactly in full."""
import sys

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from workloads import gen
from harness import Setup, assert_close, f64

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)


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


def sample_rows(ctx, k, seed):
    rng = np.random.default_rng(seed)
    rows = {0, int(np.argmax(ctx)), int(np.argmin(ctx))}
    while len(rows) < k:
        rows.add(int(rng.integers(0, len(ctx))))
    return sorted(rows)


def chained_bar(n_layers):
    return max(1e-2, 5e-3 * n_layers)


def routing_clear(logits, k, gap=3e-2):
    srt = -np.sort(-logits, axis=1)
    return (srt[:, k - 1] - srt[:, k]) > gap


class FullSize:
    def __init__(self, w, n_rows, tiled=False):
        say("full size", w.name, "setup", "tiled" if tiled else "row-major")
        self.w = w
        self.s = Setup(w, seed=w.seed, tiled=tiled)
        np.testing.assert_array_equal(self.s.page_table,
                                      O.kv_alloc(self.s.ctx, self.s.pool_pages, w.seed, self.s.max_pages))
        self.rows = sample_rows(self.s.ctx, n_rows, 1)
        self.tr = torch.from_numpy(np.asarray(self.rows)).cuda()

    def snapshot(self):
        return self.s.oracle_inputs(self.rows)   # before the step appends to the cache

    def rows_of(self, name, width):
        return f64(self.s.buf(name, self.w.batch, width)[self.tr])


def _chained(w, n_rows, moe=False, tiled=False):
    f = FullSize(w, n_rows, tiled)
    s, rows = f.s, f.rows
    inp = f.snapshot()
    say("chained", w.name, "rows", rows)
    s.reset_resid()
    for a, b in bench_ranges(w.layers):
        s.run(a, b)
    torch.cuda.synchronize()
    n_ops = sum(layer_ops(c) for c in w.layers)
    ref = O.run_ops(list(w.layers), inp["weights"], inp["pools"], inp["page_table"], inp["ctx"],
                    {"resid": inp["x"].copy()}, 0, n_ops)
    cfg = w.layers[-1]
    bar = chained_bar(len(w.layers))
    keep = np.ones(len(rows), dtype=bool)
    if moe:
        keep = routing_clear(ref["logits"], cfg.top_k)
        assert keep.sum() >= 3, "too few sampled tokens clear of routing near-ties"
        ids = f.rows_of("topk_ids", cfg.top_k).astype(np.int64)
        np.testing.assert_array_equal(ids[keep], ref["topk_ids"][keep])
    resid = f.rows_of("resid", cfg.hidden)
    o = f.rows_of("o", cfg.n_q * cfg.head_dim)
    for i, b in enumerate(rows):
        if keep[i]:
            assert_close(f"{w.name} chained resid row {b}", resid[i], ref["resid"][i], bar)
        assert_close(f"{w.name} chained last-layer o row {b}", o[i], ref["o"][i], 2 * bar)
    return f


def _stages(f, moe=False):
    """Each layer's attention, core-attention and FFN stage from fresh inputs."""
    w, s, rows = f.w, f.s, f.rows
    off = 0
    for l, cfg in enumerate(w.layers):
        H, n = cfg.hidden, layer_ops(cfg)
        # attention stage [0, 6) from a fresh residual stream
        x = gen.live_tensor((w.batch, H), w.seed + 100 + l, 10, "cuda")
        inp = f.snapshot()
        s.reset_resid(x)
        s.run(off, off + 4)
        s.run(off + 4, off + 5)
        s.run(off + 5, off + 6)
        torch.cuda.synchronize()
        xr = f64(x[f.tr])
        ref = O.run_ops(list(w.layers), inp["weights"], inp["pools"], inp["page_table"], inp["ctx"],
                        {"resid": xr.copy()}, off, off + 6)
        h = f.rows_of("resid", H)
        for i, b in enumerate(rows):
            assert_close(f"{w.name} layer {l} attention stage resid row {b}", h[i], ref["resid"][i])
        # core-attention stage [3, 5) from a fresh qkv
        say("stages", w.name, "layer", l, "core attention")
        qkv = gen.live_tensor((w.batch, cfg.qkv_dim), w.seed + 200 + l, 11, "cuda")
        inp = f.snapshot()
        s.buf("qkv", w.batch, cfg.qkv_dim).copy_(qkv)
        s.run(off + 3, off + 5)
        torch.cuda.synchronize()
        ref = O.run_ops(list(w.layers), inp["weights"], inp["pools"], inp["page_table"], inp["ctx"],
                        {"qkv": f64(qkv[f.tr])}, off + 3, off + 5)
        o = f.rows_of("o", cfg.n_q * cfg.head_dim)
        for i, b in enumerate(rows):
            assert_close(f"{w.name} layer {l} core attention o row {b}", o[i], ref["o"][i])
        # FFN stage [6, end) from a fresh residual stream
        say("stages", w.name, "layer", l, "ffn")
        hx = gen.live_tensor((w.batch, H), w.seed + 300 + l, 12, "cuda")
        s.reset_resid(hx)
        s.run(off + 6, off + n)
        torch.cuda.synchronize()
        ref = O.run_ops(list(w.layers), inp["weights"], inp["pools"], inp["page_table"], inp["ctx"],
                        {"resid": f64(hx[f.tr])}, off + 6, off + n)
        y = f.rows_of("resid", H)
        keep = routing_clear(ref["logits"], cfg.top_k) if cfg.n_experts else np.ones(len(rows), dtype=bool)
        if cfg.n_experts:
            ids = f.rows_of("topk_ids", cfg.top_k).astype(np.int64)
            np.testing.assert_array_equal(ids[keep], ref["topk_ids"][keep])
        for i, b in enumerate(rows):
            if keep[i]:
                assert_close(f"{w.name} layer {l} ffn stage resid row {b}", y[i], ref["resid"][i])
        if not cfg.n_experts:
            act = f.rows_of("act", cfg.ffn)
            ref_act = O.silu(ref["gu"][:, :cfg.ffn]) * ref["gu"][:, cfg.ffn:]
            for i, b in enumerate(rows):
                assert_close(f"{w.name} layer {l} ffn stage act row {b}", act[i], ref_act[i])
        off += n


@pytest.mark.parametrize("tiled", [True, False], ids=["tiled", "rows"])
@pytest.mark.parametrize("name,n_rows", [("dense8b_b64", 4), ("dense8b_b256_ctx8k", 3), ("hybrid4_b128", 3),
                                         ("moe64x8_b512", 8)])
def test_fullsize(name, n_rows, tiled):
    """The benchmark runs tiled weights; the row-major layout is the other
    supported one."""
    w = W.BY_NAME[name]
    moe = w.layers[0].n_experts > 0
    f = _chained(w, n_rows, moe, tiled)
    _stages(f, moe)
    del f
    torch.cuda.empty_cache()
