"""HIP-graph replay of partitions (Section 6: stages bound once as graphs,
only token, position and KV metadata rewritten between iterations). Each graph
is replayed several times with eager work and synchronisations in between;
every replay must equal the eager run of the same inputs bit for bit (same
kernels, same order), and every replay's outputs must match the CPU oracle on
the same inputs (1e-2 per row, max |gpu - oracle| / max |oracle|)."""
import sys

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from harness import Setup, assert_rows_close, f64, report

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


def replay_and_compare(s, graph, ref, names, reps=3, oracle=None, rows=None, tag=""):
    """Replay `reps` times; each replay must equal the eager snapshot `ref` bit
    for bit and, when `oracle` (name -> float64 rows) is given, match it on
    `rows` (all rows by default) to 1e-2 per row."""
    side = torch.randn(1 << 20, device="cuda")
    worst = {}
    for rep in range(reps):
        s.reset_resid()                  # eager work between replays ...
        side.mul_(1.0001).add_(rep)      # ... and an unrelated kernel
        torch.cuda.synchronize()
        graph.launch()
        torch.cuda.synchronize()
        got = snapshot(s, names)
        for n in names:
            assert torch.equal(got[n], ref[n]), f"replay {rep}: {n} differs from the eager run"
            if oracle is not None and n in oracle:
                g = f64(got[n])
                g = g if rows is None else g[rows]
                worst[n] = max(worst.get(n, 0.0), assert_rows_close(f"{tag} replay {rep} {n} vs oracle", g,
                                                                    oracle[n])[0])
    if worst:
        report(f"graph {tag}: {reps} replays vs oracle, worst row " +
               ", ".join(f"{n} {e:.2e}" for n, e in worst.items()))


def oracle_of(s, a, b, ctx=None):
    """Oracle outputs of ops [a, b) from x (fresh pools; optional new contexts)."""
    inp = s.oracle_inputs()
    if ctx is not None:
        inp["ctx"] = np.asarray(ctx, dtype=np.int32)
    return O.run_ops(list(s.w.layers), inp["weights"], inp["pools"], inp["page_table"], inp["ctx"],
                     {"resid": inp["x"].copy()}, a, b)


def routed_as_oracle(s, ref):
    """Rows whose GPU expert set is the oracle's (all rows for a dense layer)."""
    c = s.w.layers[-1]
    if not c.n_experts:
        return np.arange(s.w.batch)
    ids = s.buf("topk_ids", s.w.batch, c.top_k).cpu().numpy()
    return np.array([b for b in range(s.w.batch) if set(ids[b]) == set(ref["topk_ids"][b])])


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

    orc = oracle_of(s, ranges[0][0], ranges[-1][1])
    keep = routed_as_oracle(s, orc)
    assert len(keep) >= 0.9 * s.w.batch
    replay_and_compare(s, Chain(), ref, names, oracle={n: orc[n][keep] for n in names}, rows=keep,
                       tag=f"{wl.name} {ranges}")
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
        orc = oracle_of(s, 0, 6, ctx=np.maximum(s.ctx - delta, 1))
        replay_and_compare(s, g, ref, names, reps=2, oracle=orc, tag=f"{DENSE_MID.name} ctx - {delta}")
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
    replay_and_compare(s, g, ref, names, oracle=oracle_of(s, 0, 5), tag=f"{DENSE_MID.name} attn_core split 3")
    g.close()


def test_graph_capture_rejects_bad_range_without_enqueueing():
    s = Setup(W.TINY, seed=0)
    from paper_2609_14237_amd import binding as B
    st, h = B.ods_partition_graph(s.block.c, 3, 99, s.batch.c, s.state.c)
    assert st == B.ODS_ERANGE and h is None
