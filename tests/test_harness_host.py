"""Host checks of the parity harness itself (no GPU): the chunked, window-only
oracle inputs the full-size tests use reproduce the oracle on whole inputs
(to float64 rounding: a matrix product over fewer rows may sum in another
order), and the routing check accepts what it should and rejects a
wrong expert choice."""

import numpy as np
import pytest

import oracle as O
import workloads as W

pytest.importorskip("paper_2609_14237_amd.binding")
from harness import Setup, routing_check  # noqa: E402

HYBRID = W.Workload("hybrid_host", tuple([W.LayerCfg(hidden=128, n_q=4, n_kv=2, head_dim=64, ffn=256, window=40)] * 2
                                         + [W.LayerCfg(hidden=128, n_q=4, n_kv=2, head_dim=64, ffn=256)]),
                    batch=9, ctx_lo=1, ctx_hi=300)


def test_windowed_chunks_reproduce_whole_inputs():
    s = Setup(HYBRID, seed=3, device="cpu")
    cfgs = list(HYBRID.layers)
    full = s.oracle_inputs()
    ref = O.run_ops(cfgs, full["weights"], full["pools"], full["page_table"], full["ctx"],
                    {"resid": full["x"].copy()}, 0, 30)
    chunks = s.row_chunks(np.arange(HYBRID.batch), budget_bytes=3 * 2 * 2 * 16 * 64 * 8 * 12)
    assert len(chunks) > 1 and sorted(sum(chunks, [])) == list(range(HYBRID.batch))
    for chunk in chunks:
        inp = s.oracle_inputs_windowed(chunk)
        # sliding-window layers carry no page before each row's window
        for i, b in enumerate(chunk):
            c = int(s.ctx[b])
            first = max(0, c - 40) // 16
            assert (inp["page_table"][0][i, :first] == -1).all()
            assert (inp["page_table"][2][i, :-(-c // 16)] >= 0).all()
        got = O.run_ops(cfgs, inp["weights"], inp["pools"], inp["page_table"], inp["ctx"],
                        {"resid": inp["x"].copy()}, 0, 30)
        for name in ("resid", "o", "qkv"):
            np.testing.assert_allclose(got[name], ref[name][chunk], rtol=1e-12, atol=1e-13)


def test_routing_check_accepts_noise_and_rejects_a_wrong_choice():
    rng = np.random.default_rng(8)
    B, E, k = 200, 16, 4
    ref_logits = rng.normal(size=(B, E))
    ref_ids, ref_w = O.topk_route(ref_logits, k)
    ref = {"logits": ref_logits, "topk_ids": ref_ids}
    # the "GPU" sees logits with 1e-4 noise, rounded to fp32, and decides on them
    gl = (ref_logits + rng.normal(scale=1e-4, size=(B, E))).astype(np.float32).astype(np.float64)
    ids, w = O.topk_route(gl, k)
    forced, summary = routing_check("noise", ids, w, gl, ref, k)
    assert "near-tie" in summary
    same = np.array([set(a) == set(b) for a, b in zip(ids, ref_ids)])
    np.testing.assert_array_equal(forced[same], ref_ids[same])
    np.testing.assert_array_equal(forced[~same], ids[~same])
    # a token that swaps a clearly chosen expert for a clearly rejected one fails
    bad = ids.copy()
    srt = np.argsort(-ref_logits[0], kind="stable")
    bad[0, k - 1] = srt[-1]
    with pytest.raises(AssertionError):
        routing_check("wrong", bad, w, gl, ref, k)
    # so does a choice that is not the top-k of the GPU's own logits
    with pytest.raises(AssertionError):
        routing_check("not top-k", ids[:, ::-1].copy(), w, gl, ref, k)
    # and too many near-ties: noise as large as the gaps
    noisy = ref_logits + rng.normal(scale=0.5, size=(B, E))
    nids, nw = O.topk_route(noisy, k)
    with pytest.raises(AssertionError):
        routing_check("noisy", nids, nw, noisy, ref, k)
