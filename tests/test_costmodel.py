"""Cost model and planner (host side) against the paper's printed values and
against brute force: the hardware ratios and gain bounds quoted from the GPU
table, Theorems 1 and 2 checked numerically, b* against the operator-level
roofline, template counts against enumeration, and plan invariants."""
import math
import os

import numpy as np
import pytest

import workloads as W
from paper_2609_14237_amd import costmodel as CM

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_gpu_table.txt")


def paper_gpus():
    gpus, pairs = {}, {}
    for line in open(GOLDEN):
        f = line.split()
        if not f or f[0].startswith("#"):
            continue
        if "+" in f[0]:
            pairs[f[0]] = (float(f[1]), float(f[2]))
        else:
            name, bw, mem, tf, price = f[0], *map(float, f[1:])
            gpus[name] = CM.Gpu(name, price, bw * 1e9, mem * 1e9, tf * 1e12)
    return gpus, pairs


DENSE32 = CM.Model(W.BY_NAME["dense8b_b64"].layers, 32)


def test_eta_and_gain_bounds_match_the_printed_examples():
    gpus, pairs = paper_gpus()
    for key, (eta_p, bound_p) in pairs.items():
        a, b = key.split("+")
        e = CM.eta(gpus[a], gpus[b])
        assert round(e, 2) == eta_p
        assert round(CM.g_het_bound(e), 2) == bound_p


def test_b_star_is_where_the_operator_roofline_turns_compute_bound():
    """b* from the closed form equals the batch at which the per-operator
    roofline of the GEMM operators turns compute-bound when, as in Section
    3's scaling approximations, only weight bytes count as traffic; the
    activations each GEMM also reads and writes push the crossing higher."""
    g = CM.MI355X
    gemm = [op for op in CM.block_ops(DENSE32.block) if op.name in ("qkv_proj", "o_proj_residual", "gate_up",
                                                                    "down_residual")]

    def crossing(with_activations):
        def excess(b):  # compute time minus memory time of the GEMM class at batch b
            D = sum(CM.op_bytes_flops(op.cfg, op.name, b, 1)[0 if with_activations else 2] for op in gemm)
            Wf = sum(CM.op_bytes_flops(op.cfg, op.name, b, 1)[1] for op in gemm)
            return Wf / g.flops - D / g.bandwidth
        lo, hi = 1.0, 1e5
        for _ in range(200):
            mid = (lo + hi) / 2
            lo, hi = (mid, hi) if excess(mid) < 0 else (lo, mid)
        return lo

    bstar = CM.b_star(g, DENSE32)
    assert crossing(False) == pytest.approx(bstar, rel=1e-9)
    assert bstar < crossing(True) < 1.2 * bstar
    assert abs(bstar - 314.6) < 0.1  # 8B-shaped layer x 32 on MI355X


def test_theorem_1_homogeneous_gain():
    g = CM.MI355X
    bstar, bound = CM.b_star(g, DENSE32), CM.g_hom_bound(g, DENSE32)
    s_max = (g.memory - DENSE32.m_weights) / DENSE32.m_kv(1)  # b_bar = 1
    ss = np.geomspace(64, s_max * 0.999, 400)
    gains = np.array([CM.g_hom(g, DENSE32, s) for s in ss])
    bb = np.array([CM.b_bar(g, DENSE32, s) for s in ss])
    assert np.all(gains[bb >= bstar] == 1.0)
    inc = gains[bb < bstar]
    assert np.all(inc > 1.0) and np.all(np.diff(inc) > 0)
    assert np.all(gains < bound) and gains[-1] > 1 + 0.99 * (bound - 1)


def test_theorem_2_heterogeneous_gain_is_unimodal_and_bounded():
    gpus, _ = paper_gpus()
    for a, b in (("H100", "L40S"), ("H100", "A100")):
        g1, g2 = gpus[a], gpus[b]
        e = CM.eta(g1, g2)
        xs = CM.x_star(g1, g2, DENSE32)
        # gain as a function of x = m_kv(s): m_kv is linear in s for full attention
        per_s = DENSE32.m_kv(1.0)
        s_star = xs / per_s
        ss = np.geomspace(s_star / 50, s_star * 50, 801)
        gains = np.array([CM.g_het([g1, g2], DENSE32, s) for s in ss])
        assert np.all(gains >= 1.0) and np.all(gains <= CM.g_het_bound(e) + 1e-12)
        k = int(np.argmax(gains))
        assert np.all(np.diff(gains[:k + 1]) > 0) and np.all(np.diff(gains[k:]) < 0)
        assert abs(ss[k] / s_star - 1) < 0.02
        assert CM.g_het([g1, g2], DENSE32, s_star) >= gains.max() - 1e-12


def test_theorem_2_bound_is_the_supremum_over_prices():
    """Brute force over the price ratio and x reaches (1 + sqrt(eta)) / 2."""
    gpus, _ = paper_gpus()
    g1, g2 = gpus["H100"], gpus["A100"]
    e = CM.eta(g1, g2)
    best = 0.0
    for ratio in np.geomspace(0.05, 20, 801):
        g2r = CM.Gpu("x", g1.price_per_hour * ratio, g2.bandwidth, g2.memory, g2.flops)
        if not (min(g1.alpha, g2r.alpha) < max(g1.alpha, g2r.alpha)):
            continue
        try:
            xs = CM.x_star(g1, g2r, DENSE32)
        except ZeroDivisionError:
            continue
        if xs <= 0:
            continue
        best = max(best, CM.g_het([g1, g2r], DENSE32, xs / DENSE32.m_kv(1.0)))
    assert abs(best - CM.g_het_bound(e)) < 2e-3


def test_no_heterogeneous_gain_under_dominance():
    g1 = CM.Gpu("a", 1.0, 4e12, 80e9, 1e15)
    g2 = CM.Gpu("b", 2.0, 3e12, 80e9, 0.9e15)  # costlier per byte and per flop
    for s in (512, 8192, 65536):
        assert CM.g_het([g1, g2], DENSE32, s) == pytest.approx(1.0, abs=1e-15)


@pytest.mark.parametrize("N,S", [(10, 1), (10, 2), (10, 3), (14, 4), (9, 5)])
def test_template_count(N, S):
    qs = list(CM.templates(N, S))
    assert len(qs) == len(set(qs)) == CM.count_templates(N, S) == math.comb(N - 1, S - 1)
    assert all(q[0] == 0 and q[-1] == N and all(a < b for a, b in zip(q, q[1:])) for q in qs)


def test_subblock_templates_tile_one_repetition():
    N, n, K = 40, 4, 3  # the hybrid block: 4 layers of 10 operators
    qs = list(CM.subblock_templates(N, n, K))
    assert len(qs) == math.comb(N // n - 1, K - 1)
    for q in qs:
        assert len(q) - 1 == n * K
        sub = q[:K + 1]
        assert all(q[r * K + i] == r * (N // n) + sub[i] for r in range(n) for i in range(K + 1))


def test_colocated_plan_is_the_roofline_step_cost():
    """One stage, one microbatch: T_rtt is B_total times the summed operator
    roofline latencies (Appendix A's step cost) and CPT = T_rtt c / b."""
    g, s, b = CM.MI355X, 4096, 64
    p = CM.evaluate(DENSE32, g, (0, 10), 1, b, s)
    lat = CM.roofline_latency(g)
    step = DENSE32.n_blocks * sum(lat(op, b, s) for op in CM.block_ops(DENSE32.block))
    assert p.t_rtt == pytest.approx(step, rel=1e-12)
    assert p.cpt == pytest.approx(step * g.c / b, rel=1e-12)


def test_search_beats_the_named_templates_and_respects_the_slo():
    g, s = CM.MI355X, 16384
    block = W.BY_NAME["hybrid4_b128"].layers
    m = CM.Model(block, 8)
    mus, bs = (1, 2, 4), (8, 16, 32, 64, 128)
    plans = CM.search(m, g, s, slo=0.03, S_max=2, mus=mus, b_hats=bs)
    assert plans and all(p.t_rtt <= 0.03 for p in plans)
    named = []
    for q, r in (((0, 40), 0), ((0, 6, 40), 0), ((0, 38, 40), 5)):  # colocated, AFD-like, CAD-like (core attention isolated)
        for mu in mus:
            for b in bs:
                p = CM.evaluate(m, g, q, mu, b, s, rotation=r)
                if p is not None and p.t_rtt <= 0.03:
                    named.append(p.cpt)
    assert plans[0].cpt <= min(named) + 1e-18
    looser = CM.search(m, g, s, slo=0.06, S_max=2, mus=mus, b_hats=bs)
    assert looser[0].cpt <= plans[0].cpt


def test_plans_that_do_not_fit_memory_are_dropped():
    small = CM.Gpu("small", 1.0, 8e12, 12e9, 2.5e15)  # 12 GB: the 14 GB of weights cannot sit on one owner
    assert CM.evaluate(DENSE32, small, (0, 10), 1, 8, 4096) is None
    two = CM.evaluate(DENSE32, small, (0, 7, 10), 1, 8, 4096)  # attention side / FFN side each fit
    assert two is not None and all(mem <= small.memory for mem in two.memory)


def test_profiled_latency_interpolates_between_measured_points():
    rows = [{"local": 0, "batch": 1, "ctx": 1024, "us": 10.0}, {"local": 0, "batch": 9, "ctx": 1024, "us": 18.0},
            {"local": 0, "batch": 1, "ctx": 4096, "us": 20.0}, {"local": 0, "batch": 9, "ctx": 4096, "us": 36.0}]
    lat = CM.ProfiledLatency(rows)
    op = CM.block_ops(W.TINY.layers)[0]
    assert lat(op, 1, 1024) == pytest.approx(10e-6)
    assert lat(op, 5, 1024) == pytest.approx(14e-6)
    assert lat(op, 5, 2560) == pytest.approx(21e-6)  # 14 us at 1024, 28 us at 4096
    assert lat(op, 100, 99999) == pytest.approx(36e-6)


# ---------------------------------------------------------------- per-type microbatches (Appendix B replicas)

MOE32 = CM.Model(W.BY_NAME["moe64x8_b512"].layers, 32)


def test_equal_per_type_microbatches_give_the_common_plan():
    g = CM.MI355X
    for model, N in ((DENSE32, 10), (MOE32, 14)):
        for s, q, mu, b, r in ((4096, (0, 6, N), 2, 64, 0), (16384, (0, N - 2, N), 4, 32, 5),
                               (1024, (0, 3, 9, N), 1, 128, 2)):
            one = CM.evaluate(model, g, q, mu, b, s, rotation=r)
            tab = CM._Tables(model, g, s, CM.roofline_latency(g), (b,), 153e9)
            per = CM._plan_from_tables(model, g, tab, q, mu, (b,) * (len(q) - 1), r)
            assert (one is None) == (per is None)
            if one is not None:
                assert (per.t, per.u, per.t_rtt, per.cpt) == (one.t, one.u, one.t_rtt, one.cpt)
                assert per.b_hats == (b,) * (len(q) - 1)


def test_per_type_cost_counts_the_replicas():
    """A global microbatch of B_hat requests takes B_hat / b_hat_m replicas of
    type m; every replica is paid for T_rtt per round trip, which completes
    mu * B_hat tokens (Appendix B, cost-per-token derivation)."""
    g, s = CM.MI355X, 1024
    tab = CM._Tables(MOE32, g, s, CM.roofline_latency(g), (64, 128, 1024), 153e9)
    for bs, mu in (((128, 1024), 2), ((1024, 64), 1), ((64, 128), 4)):
        p = CM._plan_from_tables(MOE32, g, tab, (0, 6, 14), mu, bs, 0)
        assert p is not None and p.b_hats == bs and p.b_hat == max(bs)
        B_hat = math.lcm(*bs)
        replicas = [B_hat // b for b in bs]
        gpu_seconds = p.t_rtt * g.c * sum(replicas)
        assert p.cpt == pytest.approx(gpu_seconds / (mu * B_hat), rel=1e-12)


def test_each_type_holds_the_kv_of_its_own_microbatches():
    g, s = CM.MI355X, 16384  # 1 GB of KV per request over 32 layers
    tab = CM._Tables(MOE32, g, s, CM.roofline_latency(g), (128, 512, 1024), 153e9)
    # attention side at 512 requests needs 512 GB of KV: no plan, whatever the FFN side gathers
    assert CM._plan_from_tables(MOE32, g, tab, (0, 6, 14), 1, (512, 128), 0) is None
    p = CM._plan_from_tables(MOE32, g, tab, (0, 6, 14), 1, (128, 1024), 0)
    assert p is not None and p.memory[0] <= g.memory and p.memory[1] <= g.memory
    assert p.memory[1] == pytest.approx(MOE32.n_blocks * sum(
        CM.op_bytes_flops(op.cfg, op.name, 1, s)[2] for op in CM.block_ops(MOE32.block)[6:]))


def test_per_type_search_contains_the_common_one():
    g, s = CM.MI355X, 4096
    kw = dict(S_max=2, mus=(1, 2), b_hats=(32, 128, 512))
    common = CM.search(DENSE32, g, s, slo=0.05, **kw)
    per = CM.search(DENSE32, g, s, slo=0.05, per_type_batch=True, **kw)
    assert per and per[0].cpt <= common[0].cpt
    assert len(per) > len(common)


def test_gathering_pays_only_where_the_colocated_batch_is_memory_bound():
    """Theorem 1's regimes on the roofline latencies: while the colocated batch
    can reach b* (short contexts) no disaggregated plan is cheaper; once memory
    caps it below b*, a type that gathers several replicas' microbatches for
    the expert GEMMs is."""
    g = CM.MI355X
    bs = (64, 128, 512, 1024, 2048, 4096)
    assert CM.b_bar(g, MOE32, 256) > 2 * CM.b_star(g, MOE32) and CM.b_bar(g, MOE32, 16384) < CM.b_star(g, MOE32)
    gains = {}
    for s in (256, 16384):
        col = CM.search(MOE32, g, s, slo=10.0, S_max=1, mus=(1,), b_hats=bs)[0]
        best = CM.search(MOE32, g, s, slo=10.0, S_max=2, mus=(1, 2, 4), b_hats=bs, per_type_batch=True)[0]
        gains[s] = col.cpt / best.cpt
        if s == 16384:
            assert best.S == 2 and len(set(best.b_hats)) == 2
    assert gains[256] == pytest.approx(1.0)
    assert gains[16384] > 1.2


# ---------------------------------------------------------------- per-layer templates over several device-group types

def test_tiled_plan_is_the_same_deployment_as_the_one_layer_block():
    """Four identical layers per block, AFD cut in every layer, stages
    alternating over two types, eight blocks: the same deployment as a
    one-layer block cut once over 32 blocks, so the same round trip, memory
    and cost."""
    g, s = CM.MI355X, 4096
    layer = W.BY_NAME["dense8b_b64"].layers[0]
    four = CM.Model((layer,) * 4, 8)
    label, r, q, K, tiled = [p for p in CM.named_plans(four) if p[0] == "AFD"][0]
    assert (r, q, K, tiled) == (0, (0, 6, 10, 16, 20, 26, 30, 36, 40), 2, 4)
    for mu, bs in ((1, (64, 64)), (2, (32, 128)), (4, (128, 8))):
        t4 = CM._Tables(four, g, s, CM.roofline_latency(g), set(bs), 153e9)
        t1 = CM._Tables(DENSE32, g, s, CM.roofline_latency(g), set(bs), 153e9)
        a = CM._plan_from_tables(four, g, t4, q, mu, bs, r, K, tiled)
        b = CM._plan_from_tables(DENSE32, g, t1, (0, 6, 10), mu, bs, 0)
        assert a is not None and b is not None and a.types == b.types == 2
        assert a.t_rtt == pytest.approx(b.t_rtt, rel=1e-12)
        assert a.cpt == pytest.approx(b.cpt, rel=1e-12)
        assert a.memory == pytest.approx(b.memory, rel=1e-12)


def test_tiled_plan_sums_each_type_over_the_layers():
    g, s = CM.MI355X, 16384
    m = CM.Model(W.BY_NAME["hybrid4_b128"].layers, 8)
    lat = CM.roofline_latency(g)
    ops = CM.block_ops(m.block)
    label, r, q, K, tiled = [p for p in CM.named_plans(m) if p[0] == "CAD"][0]
    assert (r, K, tiled) == (5, 2, 4) and len(q) == 9
    tab = CM._Tables(m, g, s, lat, (16, 64), 153e9)
    p = CM._plan_from_tables(m, g, tab, q, 2, (64, 16), r, K, tiled)
    core = [i for i, op in enumerate(ops) if op.name in ("kv_append", "attn_core")]
    rest = [i for i in range(len(ops)) if i not in core]
    busy = [sum(p.t[j] for j in range(mm, p.S, 2)) for mm in range(2)]
    assert busy[0] == pytest.approx(sum(lat(ops[i], 64, s) for i in rest), rel=1e-12)
    assert busy[1] == pytest.approx(sum(lat(ops[i], 16, s) for i in core), rel=1e-12)
    kv = sum(CM.op_bytes_flops(ops[i].cfg, ops[i].name, 1, s)[3] for i in core)
    assert p.memory[1] == pytest.approx(2 * 16 * kv * m.n_blocks, rel=1e-12)  # core attention holds all the KV
    assert p.cpt == pytest.approx(p.t_rtt * g.c * (1 / (2 * 64) + 1 / (2 * 16)), rel=1e-12)


def test_profiled_latency_keeps_window_and_full_layers_apart():
    rows = [{"local": 4, "window": 0, "batch": 8, "ctx": 16384, "us": 100.0},
            {"local": 4, "window": 1024, "batch": 8, "ctx": 16384, "us": 10.0}]
    lat = CM.ProfiledLatency(rows)
    ops = CM.block_ops(W.BY_NAME["hybrid4_b128"].layers)
    swa, full = ops[4], ops[34]
    assert (swa.name, full.name, swa.cfg.window, full.cfg.window) == ("attn_core", "attn_core", 1024, 0)
    assert lat(swa, 8, 16384) == pytest.approx(10e-6) and lat(full, 8, 16384) == pytest.approx(100e-6)


# ---------------------------------------------------------------- heterogeneous plans (a GPU kind per type)

def test_one_kind_is_the_homogeneous_search():
    g, s = CM.MI355X, 4096
    kw = dict(S_max=2, mus=(1, 2), b_hats=(32, 128, 256), per_type_batch=True)
    a = CM.search(DENSE32, g, s, 0.05, **kw)
    b = CM.search(DENSE32, (g,), s, 0.05, **kw)
    assert [p.cpt for p in a] == [p.cpt for p in b] and set(b[0].kinds) == {"MI355X"}


def test_a_dominated_kind_is_never_chosen():
    """Theorem 2's dominance case: a kind costlier per byte and per flop (with
    the same memory) never lowers a plan's cost, so the cheapest plan uses
    only the dominant kind."""
    gpus, _ = paper_gpus()
    a = gpus["H100"]
    b = CM.Gpu("H100x", a.price_per_hour * 1.3, a.bandwidth * 0.9, a.memory, a.flops * 0.95)
    assert b.alpha > a.alpha and b.gamma > a.gamma
    for s in (1024, 16384):
        kw = dict(S_max=2, mus=(1, 2, 4), b_hats=(8, 64, 256), per_type_batch=True)
        hom = CM.search(DENSE32, a, s, 0.2, **kw)[0]
        het = CM.search(DENSE32, (a, b), s, 0.2, **kw)[0]
        assert set(het.kinds) == {"H100"} and het.cpt == pytest.approx(hom.cpt, rel=1e-12)


def test_complementary_kinds_split_attention_from_the_gemms():
    """H100 with A100 (the paper's pair, eta = 1.93): A100 is cheaper per byte,
    H100 per flop. The cheapest plan puts the KV-bound core attention on A100
    and the GEMM operators on H100, beats either kind alone, and stays within
    Theorem 2's (1 + sqrt(eta)) / 2."""
    gpus, pairs = paper_gpus()
    h, a = gpus["H100"], gpus["A100"]
    assert a.alpha < h.alpha and h.gamma < a.gamma
    bound = CM.g_het_bound(CM.eta(h, a))
    ops = CM.block_ops(DENSE32.block)
    for s in (1024, 4096):
        kw = dict(S_max=2, mus=(1, 2, 4, 8), b_hats=(8, 32, 64, 128, 256, 512), per_type_batch=True)
        best_hom = min(CM.search(DENSE32, k, s, 1.0, **kw)[0].cpt for k in (h, a))
        het = CM.search(DENSE32, (h, a), s, 1.0, **kw)[0]
        assert 1.05 < best_hom / het.cpt <= bound
        assert set(het.kinds) == {"H100", "A100"}
        for j in range(het.S):
            names = {ops[(het.rotation + i) % len(ops)].name for i in range(het.q[j], het.q[j + 1])}
            kind = het.kinds[j % het.types]
            if "attn_core" in names:
                assert kind == "A100"
            if names & {"qkv_proj", "o_proj_residual", "gate_up", "down_residual"}:
                assert kind == "H100"
