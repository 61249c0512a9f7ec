"""ods_run_partition_scratch (the library's own static workspace, for callers
that cannot allocate) against ods_run_partition on a caller workspace.

Both entry points run the same kernels with the same split plans, so every
live buffer must agree bit for bit. Each case makes two calls in a row
through the scratch entry point, the second on a smaller batch, so the
second call runs on what the first left in the shared array."""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from harness import Setup
from paper_2609_14237_amd import binding as B

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

# 8B-shaped dense layer and the MoE layer, short contexts (parity of the
# kernels is covered elsewhere; this exercises the workspace routing).
DENSE = W.shrink(W.DENSE_8B_B64, name="dense8b_scratch", batch=64, ctx_lo=1, ctx_hi=700)
MOE = W.shrink(W.MOE_B512, name="moe_scratch", batch=128, ctx_lo=1, ctx_hi=500)


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


def live_names(s):
    return [n for n in ("resid", "xn", "qkv", "o", "hn", "gu", "act", "logits", "topk_ids", "topk_w", "perm",
                        "slot_pos", "expert_off", "xp", "act_p", "yp") if n in s.state.buffers]


def reset(s):
    """Live set to NaN (int buffers to -7), residual to x."""
    for t in s.state.buffers.values():
        t.fill_(float("nan") if t.dtype != torch.int32 else -7)
    s.reset_resid()


def run_all(s, runner, ranges=None):
    """Run the block range by range with `runner` from a reset live set;
    returns every live buffer."""
    reset(s)
    for a, b in ranges or bench_ranges(s.w.layers):
        runner(a, b)
    torch.cuda.synchronize()
    return {n: s.state.buffers[n].clone() for n in live_names(s)}


def compare(tag, got, ref):
    for n in ref:
        g, r = got[n], ref[n]
        same = torch.equal(g, r) or (g.dtype != torch.int32 and torch.equal(torch.isnan(g), torch.isnan(r))
                                     and torch.equal(torch.nan_to_num(g, 0.0), torch.nan_to_num(r, 0.0)))
        assert same, f"{tag}: live buffer {n} differs between the scratch and caller workspaces"


@pytest.mark.parametrize("wl,small", [(DENSE, 16), (MOE, 40)], ids=["dense", "moe"])
def test_scratch_entry_point_matches_caller_workspace(wl, small):
    for batch in (wl.batch, small):  # second call on a smaller input
        w = W.shrink(wl, batch=batch)
        say("scratch", w.name, "batch", batch)
        s = Setup(w, seed=w.seed, tiled=True)
        assert s.state.ws_bytes <= B.SCRATCH_BYTES
        ref = run_all(s, s.run)
        got = run_all(s, lambda a, b: s.R.run_partition_scratch(s.block, a, b, s.batch, s.state))
        compare(f"{w.name} batch {batch}", got, ref)
        # one call over the whole block as well
        whole = [(0, s.block.num_ops())]
        ref = run_all(s, s.run, whole)
        got = run_all(s, lambda a, b: s.R.run_partition_scratch(s.block, a, b, s.batch, s.state), whole)
        compare(f"{w.name} batch {batch} whole block", got, ref)
        del s
        torch.cuda.empty_cache()


def test_scratch_ignores_the_caller_workspace_pointer():
    s = Setup(DENSE, seed=DENSE.seed, tiled=True)
    ref = run_all(s, s.run)
    s.state.c.ws = None
    s.state.c.ws_bytes = 0
    got = run_all(s, lambda a, b: s.R.run_partition_scratch(s.block, a, b, s.batch, s.state))
    compare("ws = NULL", got, ref)
    np.testing.assert_equal(B.ods_run_partition(s.block.c, 0, 4, s.batch.c, s.state.c, 0), B.ODS_EINVAL)
