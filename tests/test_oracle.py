"""Pins of the CPU oracle against facts that do not come from the oracle itself:
published generator outputs, closed forms, invariants, library routines on
special cases and brute force on tiny inputs. CPU only."""
import math
import os
from dataclasses import dataclass

import numpy as np
import pytest

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@dataclass(frozen=True)
class Cfg:
    hidden: int
    n_q: int
    n_kv: int
    head_dim: int
    ffn: int = 0
    n_experts: int = 0
    top_k: int = 0
    moe_ffn: int = 0
    window: int = 0
    rope_theta: float = 10000.0
    rms_eps: float = 1e-6


# ---------------------------------------------------------------- allocator

def test_splitmix64_matches_published_sequence():
    lines = [l.split() for l in open(os.path.join(GOLDEN, "splitmix64_reference.txt"))
             if l.strip() and not l.startswith("#")]
    assert lines[0][0] == "seed"
    state = int(lines[0][1])
    for (val,) in lines[1:]:
        state, out = O.splitmix64(state)
        assert out == int(val)


def test_fisher_yates_small_case_by_hand():
    # P = 3: i = 2 draws j = out1 mod 3, then i = 1 draws j = out2 mod 2.
    s, o1 = O.splitmix64(7)
    s, o2 = O.splitmix64(s)
    perm = [0, 1, 2]
    j = o1 % 3
    perm[2], perm[j] = perm[j], perm[2]
    j = o2 % 2
    perm[1], perm[j] = perm[j], perm[1]
    assert O.page_permutation(3, 7) == perm


def load_kv_alloc_example():
    ex = {"pages": []}
    for line in open(os.path.join(GOLDEN, "kv_alloc_worked_example.txt")):
        if not line.strip() or line.startswith("#"):
            continue
        key, *vals = line.split()
        vals = [int(v, 0) for v in vals]
        if key == "pages":
            ex["pages"].append(vals)
        else:
            ex[key] = vals
    return ex


def test_kv_alloc_worked_example():
    ex = load_kv_alloc_example()
    state = 0
    for want in ex["splitmix64_seed0"]:
        state, out = O.splitmix64(state)
        assert out == want
    P, seed = ex["pool_pages"][0], ex["seed"][0]
    assert O.page_permutation(P, seed) == ex["permutation"]
    table = O.kv_alloc(ex["contexts"], P, seed, 3)
    for b, pages in enumerate(ex["pages"]):
        np.testing.assert_array_equal(table[b, :len(pages)], pages)
        assert (table[b, len(pages):] == -1).all()


@pytest.mark.parametrize("seed", [0, 1, 12345])
def test_kv_alloc_invariants(seed):
    rng = np.random.default_rng(seed)
    ctx = rng.integers(1, 200, size=23)
    need = [-(-int(c) // 16) for c in ctx]
    P = sum(need) + 7
    t = O.kv_alloc(ctx, P, seed, max(need) + 2)
    used = []
    for b, n in enumerate(need):
        assert (t[b, :n] >= 0).all() and (t[b, :n] < P).all()
        assert (t[b, n:] == -1).all()
        used.extend(t[b, :n].tolist())
    assert len(set(used)) == len(used) == sum(need)
    # contiguous assignment of the shuffled list
    assert used == O.page_permutation(P, seed)[:sum(need)]


def test_kv_alloc_errors():
    with pytest.raises(MemoryError):
        O.kv_alloc([33, 33], 5, 0, 4)
    with pytest.raises(ValueError):
        O.kv_alloc([33], 10, 0, 2)


# ---------------------------------------------------------------- operators

def test_rmsnorm_closed_form():
    H, c, eps = 16, 0.37, 1e-6
    g = np.linspace(0.5, 1.5, H)
    y = O.rmsnorm(np.full((1, H), c), g, eps)
    np.testing.assert_allclose(y[0], g * c / math.sqrt(c * c + eps), rtol=1e-15)
    # eps -> 0: output depends only on the direction of x
    x = np.random.default_rng(0).normal(size=(3, H))
    np.testing.assert_allclose(O.rmsnorm(5 * x, g, 0.0), O.rmsnorm(x, g, 0.0), rtol=1e-13)


def test_linear_integer_example():
    x = np.array([[1.0, 2.0, 3.0]])
    w = np.array([[1.0, 0.0, -1.0], [2.0, 1.0, 0.0]])   # [out=2, in=3]
    # out_0 = 1 - 3 = -2 ; out_1 = 2 + 2 = 4
    np.testing.assert_array_equal(O.linear(x, w), [[-2.0, 4.0]])


def test_rope_closed_forms():
    # d = 2: the single pair rotates by angle p
    for p in [0, 1, 5, 1000]:
        y = O.rope_rotate(np.array([[[1.0, 0.0], [0.0, 1.0]]]), np.array([p]), 10000.0)
        np.testing.assert_allclose(y[0, 0], [math.cos(p), math.sin(p)], atol=1e-12)
        np.testing.assert_allclose(y[0, 1], [-math.sin(p), math.cos(p)], atol=1e-12)
    # d = 4, theta = 10000: pair 0 -> angle p, pair 1 (dims 1, 3) -> angle p / 100
    p = 7
    y = O.rope_rotate(np.array([[[0.0, 1.0, 0.0, 0.0]]]), np.array([p]), 10000.0)
    np.testing.assert_allclose(y[0, 0], [0, math.cos(p / 100), 0, math.sin(p / 100)], atol=1e-12)


def test_rope_invariants():
    rng = np.random.default_rng(1)
    d = 16
    q, k = rng.normal(size=(1, 1, d)), rng.normal(size=(1, 1, d))
    # position 0 is the identity
    np.testing.assert_array_equal(O.rope_rotate(q, np.array([0]), 1e4), q)
    # each rotated pair keeps its norm
    y = O.rope_rotate(q, np.array([123]), 1e4)
    h = d // 2
    np.testing.assert_allclose(y[..., :h] ** 2 + y[..., h:] ** 2, q[..., :h] ** 2 + q[..., h:] ** 2, rtol=1e-12)
    # scores depend only on the relative position
    def dot(pq, pk):
        return float(np.sum(O.rope_rotate(q, np.array([pq]), 1e4) * O.rope_rotate(k, np.array([pk]), 1e4)))
    assert dot(10, 3) == pytest.approx(dot(110, 103), rel=1e-10)


def test_silu_closed_form():
    np.testing.assert_allclose(O.silu(np.array([0.0, math.log(3.0)])), [0.0, 0.75 * math.log(3.0)], rtol=1e-15)
    assert O.silu(np.array([40.0]))[0] == pytest.approx(40.0, rel=1e-15)


# ---------------------------------------------------------------- attention

def _pool_from_logical(Ks, Vs, table, P, n_kv, d):
    """Scatter logical keys / values of each sequence into a pool, written out
    from the page layout definition one element at a time."""
    pool = np.full((P, 2, n_kv, 16 * d), np.nan)
    for b, (K, V) in enumerate(zip(Ks, Vs)):
        for g in range(n_kv):
            for t in range(K.shape[1]):
                page, slot = table[b][t // 16], t % 16
                for i in range(d):
                    pool[page, 0, g, slot * d + i] = K[g, t, i]
                    pool[page, 1, g, i * 16 + slot] = V[g, t, i]
    return pool


def test_page_gather_matches_logical_layout():
    rng = np.random.default_rng(2)
    n_kv, d, ctx = 2, 4, [5, 16, 33]
    Ks = [rng.normal(size=(n_kv, c, d)) for c in ctx]
    Vs = [rng.normal(size=(n_kv, c, d)) for c in ctx]
    P = 10
    table = O.kv_alloc(ctx, P, 3, 3)
    pool = _pool_from_logical(Ks, Vs, table, P, n_kv, d)
    for b, c in enumerate(ctx):
        K, V = O.page_kv(pool, table[b], c, n_kv, d)
        np.testing.assert_array_equal(K, Ks[b])
        np.testing.assert_array_equal(V, Vs[b])
        # a window [first, c) reads only its own pages and returns those positions
        for first in sorted({0, 1, 15, 16, 17, c - 1} & set(range(c))):
            sub = table[b].copy()
            sub[:first // 16] = -1          # pages before the window are never read
            K, V = O.page_kv(pool, sub, c, n_kv, d, first=first)
            np.testing.assert_array_equal(K, Ks[b][:, first:])
            np.testing.assert_array_equal(V, Vs[b][:, first:])


def test_attention_invariants():
    rng = np.random.default_rng(3)
    n_q, n_kv, d, n = 4, 2, 8, 37
    q = rng.normal(size=(n_q, d))
    K = rng.normal(size=(n_kv, n, d))
    V = rng.normal(size=(n_kv, n, d))
    # V == 1: rows of the softmax sum to one
    np.testing.assert_allclose(O.attention_row(q, K, np.ones_like(V), 0, n - 1), 1.0, rtol=1e-14)
    # a single key returns its value row (group of head h is h // 2)
    o = O.attention_row(q, K, V, n - 1, n - 1)
    for h in range(n_q):
        np.testing.assert_allclose(o[h], V[h // 2, n - 1], rtol=1e-15)
    # equal keys give the mean of the values in the window
    Ke = np.repeat(K[:, :1], n, axis=1)
    o = O.attention_row(q, Ke, V, 5, n - 1)
    for h in range(n_q):
        np.testing.assert_allclose(o[h], V[h // 2, 5:].mean(axis=0), rtol=1e-12)
    # two keys: weight of the first is a logistic function of the score gap
    o = O.attention_row(q, K, V, 0, 1)
    for h in range(n_q):
        g = h // 2
        s0, s1 = K[g, 0] @ q[h] / math.sqrt(d), K[g, 1] @ q[h] / math.sqrt(d)
        w0 = 1.0 / (1.0 + math.exp(s1 - s0))
        np.testing.assert_allclose(o[h], w0 * V[g, 0] + (1 - w0) * V[g, 1], rtol=1e-12)


def test_window_start_reading():
    assert O.window_start(10, 0) == 0
    assert O.window_start(10, 4) == 7       # keys 7, 8, 9, 10: the newest W including p
    assert O.window_start(2, 4) == 0
    assert O.window_start(3, 4) == 0 and O.window_start(4, 4) == 1


# ---------------------------------------------------------------- routing

def test_topk_matches_stable_argsort_and_ties():
    rng = np.random.default_rng(4)
    logits = rng.normal(size=(50, 16))
    logits[0, [3, 9, 12]] = 5.0              # exact three-way tie at the top
    ids, w = O.topk_route(logits, 4)
    for b in range(50):
        p = np.exp(logits[b] - logits[b].max())
        p /= p.sum()
        ref = np.argsort(-p, kind="stable")[:4]
        np.testing.assert_array_equal(ids[b], ref)
        np.testing.assert_allclose(w[b].sum(), 1.0, rtol=1e-14)
    assert ids[0, :3].tolist() == [3, 9, 12]
    # k = 1 gives weight one; k = E gives the full softmax
    _, w1 = O.topk_route(logits, 1)
    np.testing.assert_array_equal(w1, 1.0)
    idsE, wE = O.topk_route(logits, 16)
    for b in range(50):
        p = np.exp(logits[b] - logits[b].max())
        p /= p.sum()
        np.testing.assert_allclose(wE[b], p[idsE[b]], rtol=1e-13)
    # top-k on the logits followed by a softmax over the k gives the same weights
    for b in range(50):
        z = logits[b][ids[b]]
        np.testing.assert_allclose(w[b], np.exp(z - z.max()) / np.exp(z - z.max()).sum(), rtol=1e-13)


def test_route_weights_of_a_given_choice():
    rng = np.random.default_rng(14)
    logits = rng.normal(size=(30, 12))
    ids, w = O.topk_route(logits, 3)
    np.testing.assert_allclose(O.route_weights(logits, ids), w, rtol=1e-14)
    # any choice: exp(z_i) / sum over the chosen exp(z_j), summing to one
    other = np.stack([rng.permutation(12)[:3] for _ in range(30)])
    got = O.route_weights(logits, other)
    for b in range(30):
        e = np.array([math.exp(logits[b, i]) for i in other[b]])
        np.testing.assert_allclose(got[b], e / e.sum(), rtol=1e-13)
    np.testing.assert_allclose(got.sum(axis=1), 1.0, rtol=1e-14)


def test_permute_is_stable_counting_sort():
    rng = np.random.default_rng(5)
    B, E, k = 40, 8, 3
    ids = np.stack([rng.permutation(E)[:k] for _ in range(B)]).astype(np.int32)
    perm, off, slot_pos = O.moe_permute(ids, E)
    flat = ids.reshape(-1)
    # brute force: walk experts in order, pairs in (token, slot) order
    ref = [i for e in range(E) for i in range(B * k) if flat[i] == e]
    np.testing.assert_array_equal(perm, ref)
    for e in range(E):
        assert (flat[perm[off[e]:off[e + 1]]] == e).all()
    np.testing.assert_array_equal(perm[slot_pos], np.arange(B * k))   # unpermute is the inverse


# ---------------------------------------------------------------- whole layer, brute force

def _weights(cfg, rng):
    H, d = cfg.hidden, cfg.head_dim
    w = {"g_attn": 1 + 0.1 * rng.normal(size=H), "g_ffn": 1 + 0.1 * rng.normal(size=H),
         "w_qkv": 0.3 * rng.normal(size=((cfg.n_q + 2 * cfg.n_kv) * d, H)),
         "w_o": 0.3 * rng.normal(size=(H, cfg.n_q * d))}
    if cfg.n_experts:
        E, I = cfg.n_experts, cfg.moe_ffn
        w["w_router"] = rng.normal(size=(E, H))
        w["w_gate_up"] = 0.3 * rng.normal(size=(E, 2 * I, H))
        w["w_down"] = 0.3 * rng.normal(size=(E, H, I))
    else:
        w["w_gate_up"] = 0.3 * rng.normal(size=(2 * cfg.ffn, H))
        w["w_down"] = 0.3 * rng.normal(size=(H, cfg.ffn))
    return w


def _brute_layer(cfg, w, Ks, Vs, x, ctx):
    """Whole decode layer with scalar loops over logical (unpaged) keys and values."""
    H, nq, nkv, d = cfg.hidden, cfg.n_q, cfg.n_kv, cfg.head_dim
    out = []
    for b in range(len(x)):
        r = list(x[b])
        ms = sum(v * v for v in r) / H
        xn = [r[i] / math.sqrt(ms + cfg.rms_eps) * w["g_attn"][i] for i in range(H)]
        qkv = [sum(w["w_qkv"][j][i] * xn[i] for i in range(H)) for j in range((nq + 2 * nkv) * d)]
        p = int(ctx[b]) - 1
        heads = [qkv[h * d:(h + 1) * d] for h in range(nq + 2 * nkv)]
        for h in range(nq + nkv):                       # q heads, then k heads
            u = heads[h]
            rot = [0.0] * d
            for i in range(d // 2):
                a = p * cfg.rope_theta ** (-2.0 * i / d)
                rot[i] = u[i] * math.cos(a) - u[i + d // 2] * math.sin(a)
                rot[i + d // 2] = u[i + d // 2] * math.cos(a) + u[i] * math.sin(a)
            heads[h] = rot
        o = []
        lo = max(0, p - cfg.window + 1) if cfg.window else 0
        for h in range(nq):
            g = h // (nq // nkv)
            keys = [list(Ks[b][g][t]) for t in range(p)] + [heads[nq + g]]
            vals = [list(Vs[b][g][t]) for t in range(p)] + [heads[nq + nkv + g]]
            s = [sum(heads[h][i] * keys[t][i] for i in range(d)) / math.sqrt(d) for t in range(lo, p + 1)]
            m = max(s)
            e = [math.exp(v - m) for v in s]
            z = sum(e)
            o.extend(sum(e[j] / z * vals[lo + j][i] for j in range(len(e))) for i in range(d))
        hres = [r[i] + sum(w["w_o"][i][j] * o[j] for j in range(nq * d)) for i in range(H)]
        ms = sum(v * v for v in hres) / H
        hn = [hres[i] / math.sqrt(ms + cfg.rms_eps) * w["g_ffn"][i] for i in range(H)]

        def swiglu(wgu, wd, F):
            gu = [sum(wgu[j][i] * hn[i] for i in range(H)) for j in range(2 * F)]
            act = [gu[j] / (1 + math.exp(-gu[j])) * gu[F + j] for j in range(F)]
            return [sum(wd[i][j] * act[j] for j in range(F)) for i in range(H)]

        if cfg.n_experts:
            lg = [sum(w["w_router"][e][i] * hn[i] for i in range(H)) for e in range(cfg.n_experts)]
            m = max(lg)
            pr = [math.exp(v - m) for v in lg]
            chosen = sorted(range(cfg.n_experts), key=lambda e: (-pr[e], e))[:cfg.top_k]
            z = sum(pr[e] for e in chosen)
            y = [0.0] * H
            for e in chosen:
                ye = swiglu(w["w_gate_up"][e], w["w_down"][e], cfg.moe_ffn)
                y = [y[i] + pr[e] / z * ye[i] for i in range(H)]
        else:
            y = swiglu(w["w_gate_up"], w["w_down"], cfg.ffn)
        out.append([hres[i] + y[i] for i in range(H)])
    return np.array(out)


def _setup(cfgs, ctx, seed):
    rng = np.random.default_rng(seed)
    B = len(ctx)
    nkv, d = cfgs[0].n_kv, cfgs[0].head_dim
    need = sum(-(-c // 16) for c in ctx)
    P = need + 3
    table = O.kv_alloc(ctx, P, seed, max(-(-c // 16) for c in ctx))
    ws, pools, logical = [], [], []
    for cfg in cfgs:
        ws.append(_weights(cfg, rng))
        Ks = [rng.normal(size=(nkv, c, d)) for c in ctx]
        Vs = [rng.normal(size=(nkv, c, d)) for c in ctx]
        logical.append((Ks, Vs))
        pools.append(_pool_from_logical(Ks, Vs, table, P, nkv, d))
    x = rng.normal(size=(B, cfgs[0].hidden))
    return ws, pools, logical, table, x


MICRO = Cfg(hidden=8, n_q=4, n_kv=2, head_dim=4, ffn=6)
MICRO_MOE = Cfg(hidden=8, n_q=4, n_kv=2, head_dim=4, n_experts=5, top_k=2, moe_ffn=3)


@pytest.mark.parametrize("cfg", [MICRO, Cfg(**{**MICRO.__dict__, "window": 5}), MICRO_MOE])
def test_layer_matches_brute_force(cfg):
    ctx = [3, 19, 40]
    ws, pools, logical, table, x = _setup([cfg], ctx, 11)
    live = O.run_ops([cfg], ws, pools, table, ctx, {"resid": x.copy()}, 0, cfg.n_experts and 14 or 10)
    ref = _brute_layer(cfg, ws[0], logical[0][0], logical[0][1], x, ctx)
    np.testing.assert_allclose(live["resid"], ref, rtol=1e-11, atol=1e-11)


def test_kv_append_writes_the_rotated_new_token():
    cfg = MICRO
    ctx = [3, 19]
    ws, pools, logical, table, x = _setup([cfg], ctx, 12)
    live = O.run_ops([cfg], ws, pools, table, ctx, {"resid": x.copy()}, 0, 4)
    nq, nkv, d = cfg.n_q, cfg.n_kv, cfg.head_dim
    for b, c in enumerate(ctx):
        K, V = O.page_kv(pools[0], table[b], c, nkv, d)
        np.testing.assert_array_equal(K[:, c - 1], live["qkv"][b, nq * d:(nq + nkv) * d].reshape(nkv, d))
        np.testing.assert_array_equal(V[:, c - 1], live["qkv"][b, (nq + nkv) * d:].reshape(nkv, d))
        np.testing.assert_array_equal(K[:, :c - 1], logical[0][0][b][:, :c - 1])   # older slots untouched


def test_window_covering_context_equals_full():
    ctx = [3, 19, 40]
    full = Cfg(**{**MICRO.__dict__, "window": 0})
    wide = Cfg(**{**MICRO.__dict__, "window": 40})
    outs = []
    for cfg in (full, wide):
        ws, pools, _, table, x = _setup([cfg], ctx, 13)
        outs.append(O.run_ops([cfg], ws, pools, table, ctx, {"resid": x.copy()}, 0, 10)["resid"])
    np.testing.assert_array_equal(outs[0], outs[1])


def test_page_shuffle_invariance():
    cfg = MICRO
    ctx = [3, 19, 40]
    rng = np.random.default_rng(14)
    w = _weights(cfg, rng)
    Ks = [rng.normal(size=(2, c, 4)) for c in ctx]
    Vs = [rng.normal(size=(2, c, 4)) for c in ctx]
    x = rng.normal(size=(3, 8))
    outs = []
    for seed in (1, 2):
        P = 9
        table = O.kv_alloc(ctx, P, seed, 3)
        pool = _pool_from_logical(Ks, Vs, table, P, 2, 4)
        outs.append(O.run_ops([cfg], [w], [pool], table, ctx, {"resid": x.copy()}, 0, 10)["resid"])
    np.testing.assert_array_equal(outs[0], outs[1])


def test_moe_special_cases():
    rng = np.random.default_rng(15)
    H, I, E = 8, 3, 4
    # identical experts: the MoE layer equals the dense SwiGLU layer with those weights
    moe = Cfg(hidden=H, n_q=4, n_kv=2, head_dim=4, n_experts=E, top_k=2, moe_ffn=I)
    dense = Cfg(hidden=H, n_q=4, n_kv=2, head_dim=4, ffn=I)
    ctx = [3, 19]
    ws, pools, _, table, x = _setup([moe], ctx, 16)
    wm = ws[0]
    wm["w_gate_up"] = np.repeat(wm["w_gate_up"][:1], E, axis=0)
    wm["w_down"] = np.repeat(wm["w_down"][:1], E, axis=0)
    wd = {k: v for k, v in wm.items() if k != "w_router"}
    wd["w_gate_up"], wd["w_down"] = wm["w_gate_up"][0], wm["w_down"][0]
    a = O.run_ops([moe], [wm], [pools[0].copy()], table, ctx, {"resid": x.copy()}, 0, 14)["resid"]
    b = O.run_ops([dense], [wd], [pools[0].copy()], table, ctx, {"resid": x.copy()}, 0, 10)["resid"]
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12)
    # k = E: softmax-weighted sum over every expert
    allk = Cfg(**{**moe.__dict__, "top_k": E})
    ws, pools, _, table, x = _setup([allk], ctx, 17)
    w = ws[0]
    live = O.run_ops([allk], ws, pools, table, ctx, {"resid": x.copy()}, 0, 7)
    h, hn = live["resid"].copy(), live["hn"]
    live = O.run_ops([allk], ws, pools, table, ctx, live, 7, 14)
    lg = hn @ w["w_router"].T
    p = np.exp(lg - lg.max(1, keepdims=True))
    p /= p.sum(1, keepdims=True)
    y = np.zeros_like(h)
    for e in range(E):
        gu = hn @ w["w_gate_up"][e].T
        y += p[:, e:e + 1] * ((O.silu(gu[:, :I]) * gu[:, I:]) @ w["w_down"][e].T)
    np.testing.assert_allclose(live["resid"], h + y, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- partitions

def _cut_results(cfgs, ctx, seed, cuts):
    ws, pools, _, table, x = _setup(cfgs, ctx, seed)
    live = {"resid": x.copy()}
    bounds = [0] + list(cuts) + [sum(14 if c.n_experts else 10 for c in cfgs)]
    for a, b in zip(bounds[:-1], bounds[1:]):
        live = O.run_ops(cfgs, ws, pools, table, ctx, live, a, b)
    return live["resid"], pools


@pytest.mark.parametrize("cfg", [MICRO, MICRO_MOE])
def test_every_two_and_three_way_cut_composes_bit_exactly(cfg):
    ctx = [3, 19]
    n = 14 if cfg.n_experts else 10
    ref, ref_pools = _cut_results([cfg], ctx, 21, [])
    for c1 in range(1, n):
        out, pools = _cut_results([cfg], ctx, 21, [c1])
        np.testing.assert_array_equal(out, ref)
        np.testing.assert_array_equal(pools[0], ref_pools[0])
        for c2 in range(c1 + 1, n):
            out, _ = _cut_results([cfg], ctx, 21, [c1, c2])
            np.testing.assert_array_equal(out, ref)


def test_hybrid_block_random_cuts_compose():
    swa = Cfg(**{**MICRO.__dict__, "window": 7})
    cfgs = [swa, swa, swa, MICRO]
    ctx = [3, 19, 40]
    ref, _ = _cut_results(cfgs, ctx, 22, [])
    rng = np.random.default_rng(22)
    for _ in range(6):
        k = int(rng.integers(1, 6))
        cuts = sorted(rng.choice(np.arange(1, 40), size=k, replace=False).tolist())
        out, _ = _cut_results(cfgs, ctx, 22, cuts)
        np.testing.assert_array_equal(out, ref)


def test_afd_and_cad_templates_compose():
    cfg = MICRO
    ctx = [3, 19]
    ref, _ = _cut_results([cfg], ctx, 23, [])
    np.testing.assert_array_equal(_cut_results([cfg], ctx, 23, [6])[0], ref)      # attention | FFN
    np.testing.assert_array_equal(_cut_results([cfg], ctx, 23, [3, 5])[0], ref)   # core attention isolated
