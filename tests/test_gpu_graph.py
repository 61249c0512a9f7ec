"""HIP-graph replay of partitions against eager execution (Section 6: stages
bound once as graphs, only token, position and KV metadata rewritten between
iterations). Each graph is replayed several times with eager work and
synchronisations in between; every replay must equal the eager run of the
same inputs bit for bit (same kernels, same order)."""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from harness import Setup

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

MOE_SMALL = W.Workload("moe_small_graph", (W.LayerCfg(hidden=512, n_q=8, n_kv=2, head_dim=64, n_experts=64,
                                                       top_k=8, moe_ffn=96),),
                       batch=40, ctx_lo=1, ctx_hi=300, router_std=512 ** -0.5)
DENSE_MID = W.Workload("dense_mid_graph", (W.LayerCfg(hidden=640, n_q=8, n_kv=2, head_dim=128, ffn=1376),),
                       batch=96, ctx_lo=1, ctx_hi=1500)


def say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


def snapshot(s, names):
    w, B = s.w, s.w.batch
    c = w.layers[0]
    shapes = {"resid": (B, c.hidden), "qkv": (B, c.qkv_dim), "o": (B, c.n_q * c.head_dim), "hn": (B, c.hidden)}
    return {n: s.buf(n, *shapes[n]).clone() for n in names}


def eager(s, a, b, names):
    s.reset_resid()
    s.run(a, b)
    torch.cuda.synchronize()
    return snapshot(s, names)


def replay_and_compare(s, graph, ref, names, reps=3):
    side = torch.randn(1 << 20, device="cuda")
    for rep in range(reps):
        s.reset_resid()                  # eager work between replays ...
        side.mul_(1.0001).add_(rep)      # ... and an unrelated kernel
        torch.cuda.synchronize()
        graph.launch()
        torch.cuda.synchronize()
        got = snapshot(s, names)
        for n in names:
            assert torch.equal(got[n], ref[n]), f"replay {rep}: {n} differs from the eager run"


@pytest.mark.parametrize("wl,ranges", [(W.TINY, [(0, 10)]), (W.TINY, [(0, 6), (6, 10)]),
                                       (DENSE_MID, [(0, 6), (6, 10)]), (MOE_SMALL, [(0, 14)]),
                                       (MOE_SMALL, [(0, 6), (6, 14)])])
def test_graph_replays_match_eager(wl, ranges):
    say("graph", wl.name, ranges)
    s = Setup(wl, seed=5)
    names = ["resid", "o"]
    s.reset_resid()
    for a, b in ranges:
        s.run(a, b)
    torch.cuda.synchronize()
    ref = snapshot(s, names)
    graphs = [s.R.PartitionGraph(s.block, a, b, s.batch, s.state) for a, b in ranges]

    class Chain:
        def launch(self):
            for g in graphs:
                g.launch()

    replay_and_compare(s, Chain(), ref, names)
    for g in graphs:
        g.close()


def test_graph_sees_rewritten_metadata():
    """The captured stage reads ctx_lens at launch: shorter contexts written
    into the same device buffer change the replayed result exactly as they
    change an eager run (pages of the shorter contexts are already mapped)."""
    say("graph metadata")
    s = Setup(DENSE_MID, seed=6)
    names = ["resid", "o"]
    g = s.R.PartitionGraph(s.block, 0, 6, s.batch, s.state)
    ctx0 = s.batch.ctx_lens.clone()
    for step, delta in enumerate((0, 7, 33)):
        s.batch.ctx_lens.copy_(torch.clamp(ctx0 - delta, min=1))
        ref = eager(s, 0, 6, names)
        s.state.view("o", DENSE_MID.batch, 8 * 128).fill_(float("nan"))
        replay_and_compare(s, g, ref, names, reps=2)
    g.close()


def test_graph_of_attention_core_with_forced_split():
    say("graph attn_core split 3")
    s = Setup(DENSE_MID, seed=7, split_pages=3)
    s.reset_resid()
    s.run(0, 4)
    torch.cuda.synchronize()
    names = ["o"]
    ref = eager(s, 4, 5, names)
    g = s.R.PartitionGraph(s.block, 4, 5, s.batch, s.state)
    replay_and_compare(s, g, ref, names)
    g.close()


def test_graph_capture_rejects_bad_range_without_enqueueing():
    s = Setup(W.TINY, seed=0)
    from paper_2609_14237_amd import binding as B
    st, h = B.ods_partition_graph(s.block.c, 3, 99, s.batch.c, s.state.c)
    assert st == B.ODS_ERANGE and h is None
