"""Test plumbing: put a workload on the GPU through the C ABI, and hand the
same seeded inputs to the CPU oracle as float64 arrays."""
from __future__ import annotations

import numpy as np
import torch

import oracle as O
import workloads as W
from workloads import gen


def f64(t: torch.Tensor) -> np.ndarray:
    """float64 host copy (converted on the device, where it is fast)."""
    return t.detach().double().cpu().numpy()


def rel_err(gpu, ref) -> float:
    """max |gpu - ref| / max |ref| (normwise), inf if gpu is not finite."""
    g = np.asarray(gpu, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    if not np.isfinite(g).all():
        return float("inf")
    den = np.abs(r).max()
    return float(np.abs(g - r).max() / (den if den > 0 else 1.0))


def elem_err(gpu, ref) -> float:
    """max over elements of |gpu - ref| / (|ref| + 1e-3 max |ref|), inf if gpu is
    not finite: the element-wise figure reported beside the normwise one."""
    g = np.asarray(gpu, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    if not np.isfinite(g).all():
        return float("inf")
    den = np.abs(r).max()
    den = den if den > 0 else 1.0
    return float((np.abs(g - r) / (np.abs(r) + 1e-3 * den)).max())


TOL = 1e-2

# Lines printed at the end of the pytest session (tests/conftest.py): measured
# error figures and counts that a passing test would otherwise not show.
REPORT: list[str] = []


def report(line: str) -> None:
    REPORT.append(line)


def assert_close(name, gpu, ref, tol=TOL):
    e = rel_err(gpu, ref)
    assert e <= tol, f"{name}: max rel err {e:.3e} > {tol}"
    return e


def rowwise_errors(gpu, ref):
    """Per-row normwise errors and the element-wise figure of every row."""
    g = np.asarray(gpu, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    norm = np.array([rel_err(g[i], r[i]) for i in range(r.shape[0])])
    elem = np.array([elem_err(g[i], r[i]) for i in range(r.shape[0])])
    return norm, elem


def assert_rows_close(name, gpu, ref, tol=TOL):
    """Every row within `tol` normwise (max |gpu - ref| / max |ref| per row).
    Returns (worst normwise, worst element-wise)."""
    norm, elem = rowwise_errors(gpu, ref)
    bad = np.nonzero(~(norm <= tol))[0]
    assert bad.size == 0, f"{name}: {bad.size} rows above {tol}, worst {norm.max():.3e} (row {int(np.argmax(norm))})"
    return float(norm.max()), float(elem.max())


def routing_check(tag, ids, weights, logits, ref, k, min_fixed=0.9):
    """Top-k routing evidence. ids / weights / logits: the GPU's (int, fp32
    values as float64); ref: the oracle's live set of the same step.
      * ids equal the oracle's top-k of the GPU's own logits for every token
        (the same decision on the same fp32 numbers), weights within 1e-6;
      * against the oracle's own logits z, with d = GPU logits - z: the
        oracle's top-k set S cannot change under d when its k-th / (k+1)-th
        gap exceeds max(d outside S) - min(d inside S); such tokens must
        choose S, and at least `min_fixed` of all tokens must be such tokens.
        Where, in addition, every adjacent gap inside S exceeds the same
        bound taken over the ranks on either side, the ordered ids must match.
    Returns (expert ids to evaluate the oracle with: the oracle's own where the
    sets agree, the GPU's elsewhere; summary string)."""
    B = ids.shape[0]
    same_ids, same_w = O.topk_route(logits, k)
    np.testing.assert_array_equal(ids, same_ids, err_msg=f"{tag}: ids differ from the top-k of the GPU logits")
    assert np.abs(weights - same_w).max() <= 1e-6, f"{tag}: routing weights differ"
    z = ref["logits"]
    d = logits - z
    order = np.argsort(-z, axis=1, kind="stable")            # oracle ranking (ties to the lower index)
    zs = np.take_along_axis(z, order, axis=1)
    ds = np.take_along_axis(d, order, axis=1)
    gaps = zs[:, :-1] - zs[:, 1:]                            # gap between ranks r and r + 1
    # bound for the boundary between ranks r and r + 1: max d below it - min d above it
    lo_max = np.maximum.accumulate(ds[:, ::-1], axis=1)[:, ::-1][:, 1:]   # max d over ranks > r
    hi_min = np.minimum.accumulate(ds, axis=1)[:, :-1]                    # min d over ranks <= r
    bound = lo_max - hi_min
    set_fixed = gaps[:, k - 1] > bound[:, k - 1]
    order_fixed = set_fixed & np.all(gaps[:, :k - 1] > bound[:, :k - 1], axis=1)
    same_set = np.array([set(ids[b].tolist()) == set(ref["topk_ids"][b].tolist()) for b in range(B)])
    bad = np.nonzero(set_fixed & ~same_set)[0]
    assert bad.size == 0, f"{tag}: tokens clear of near-ties chose other experts: {bad[:10]}"
    np.testing.assert_array_equal(ids[order_fixed], ref["topk_ids"][order_fixed],
                                  err_msg=f"{tag}: ordered ids differ on tokens clear of near-ties")
    assert set_fixed.mean() >= min_fixed, f"{tag}: only {set_fixed.mean():.1%} of tokens clear of near-ties"
    forced = np.where(same_set[:, None], ref["topk_ids"], ids)
    summary = (f"max |dlogit| {np.abs(d).max():.2e}; {int((~set_fixed).sum())}/{B} near-tie tokens outside the "
               f"set check ({int((~same_set).sum())} chose another set), {int((~order_fixed).sum())} outside the "
               f"order check; ids = oracle top-k of the GPU logits for all {B}")
    return forced, summary


class Setup:
    """One workload instantiated on the device (and optionally mirrored for the oracle)."""

    def __init__(self, w: W.Workload, seed: int = 0, device="cuda", split_pages: int = 0,
                 gen_device: str | None = None, ctx=None, alloc_seed=None, nan_trap=False, tiled=False):
        from paper_2609_14237_amd import binding as B
        from paper_2609_14237_amd import runtime as R
        self.w = w
        self.seed = seed
        self.device = device
        gdev = gen_device or device
        self.ctx = np.asarray(gen.contexts(w, seed) if ctx is None else ctx, dtype=np.int32)
        self.pool_pages = gen.pool_pages_for(self.ctx)
        self.max_pages = max(w.max_pages, int(-(-int(self.ctx.max()) // 16)))
        self.page_table = np.zeros((w.batch, self.max_pages), dtype=np.int32)
        st = B.ods_kv_alloc(self.pool_pages, self.ctx, w.batch, seed if alloc_seed is None else alloc_seed,
                            self.max_pages, self.page_table)
        assert st == 0, B.ods_last_error()
        self.weights = [{k: v.to(device) for k, v in gen.layer_weights(cfg, seed, l, gdev, w.router_std).items()}
                        for l, cfg in enumerate(w.layers)]
        self.pools = [gen.kv_pool(cfg, self.pool_pages, seed, l, gdev).to(device) for l, cfg in enumerate(w.layers)]
        if nan_trap:
            for l, cfg in enumerate(w.layers):
                self._plant_nans(self.pools[l], cfg)
        self.x = gen.activations(w.batch, w.layers[0].hidden, seed, gdev).to(device)
        # the block may hold tiled copies of the projection weights; self.weights stays row-major
        self.block = R.DeviceBlock(w.layers, self.weights, self.pools, self.pool_pages, tiled=tiled)
        self.batch = R.DeviceBatch(torch.from_numpy(self.ctx).to(device),
                                   torch.from_numpy(self.page_table).to(device), split_pages)
        self.state = R.DeviceState(self.block, self.batch, device, fill=float("nan"))
        self.R = R

    def _plant_nans(self, pool, cfg):
        """NaN in every unused page and in every slot at or past each sequence's context."""
        used = np.zeros(self.pool_pages, dtype=bool)
        d = cfg.head_dim
        v = pool.view(self.pool_pages, 2, cfg.n_kv, 16 * d)
        for b, c in enumerate(self.ctx):
            n = -(-int(c) // 16)
            used[self.page_table[b, :n]] = True
            last = int(self.page_table[b, n - 1])
            for slot in range(int(c) - (n - 1) * 16, 16):
                v[last, 0, :, slot * d:(slot + 1) * d] = float("nan")
                v[last, 1, :, slot::16] = float("nan")
        unused = torch.from_numpy(np.nonzero(~used)[0]).to(pool.device)
        if unused.numel():
            v[unused] = float("nan")

    # ---------------------------------------------------------------- GPU side
    def reset_resid(self, x=None):
        self.state.view("resid", *self.x.shape).copy_(self.x if x is None else x)

    def run(self, a: int, b: int):
        self.R.run_partition(self.block, a, b, self.batch, self.state)

    def buf(self, name, *shape):
        return self.state.view(name, *shape)

    # ---------------------------------------------------------------- oracle side
    def oracle_weights(self):
        """float64 weights, converted once per setup (per-expert stacks lazily)."""
        if getattr(self, "_w64", None) is None:
            self._w64 = [{k: (LazyF64(v) if v.dim() == 3 else f64(v)) for k, v in w.items()} for w in self.weights]
        return self._w64

    def oracle_inputs_windowed(self, rows):
        """float64 inputs of the given rows, with one page table per layer: a
        sliding-window layer carries only the pages of each row's window (the
        oracle reads no others), a full-attention layer all of the row's pages."""
        rows = np.asarray(rows)
        tables, pools = [], []
        for l, cfg in enumerate(self.w.layers):
            table = np.full((len(rows), self.max_pages), -1, dtype=np.int32)
            pages, off = [], 0
            for i, b in enumerate(rows):
                c = int(self.ctx[b])
                n = -(-c // 16)
                p0 = max(0, c - cfg.window) // 16 if cfg.window > 0 else 0
                pages.append(self.page_table[b, p0:n])
                table[i, p0:n] = np.arange(off, off + n - p0)
                off += n - p0
            idx = torch.from_numpy(np.concatenate(pages).astype(np.int64)).to(self.device)
            pools.append(f64(self.pools[l].index_select(0, idx)))
            tables.append(table)
        return dict(weights=self.oracle_weights(), pools=pools, page_table=tables, ctx=self.ctx[rows].copy(),
                    x=f64(self.x[torch.from_numpy(rows).to(self.device)]))

    def row_chunks(self, rows, budget_bytes=3 << 30):
        """Split rows into consecutive chunks whose float64 pages (all layers,
        window pages only for sliding-window layers) stay within budget_bytes."""
        out, cur, used = [], [], 0
        for b in rows:
            c = int(self.ctx[b])
            nb = 0
            for cfg in self.w.layers:
                n = -(-c // 16) - (max(0, c - cfg.window) // 16 if cfg.window > 0 else 0)
                nb += n * 2 * cfg.n_kv * 16 * cfg.head_dim * 8
            if cur and used + nb > budget_bytes:
                out.append(cur)
                cur, used = [], 0
            cur.append(int(b))
            used += nb
        if cur:
            out.append(cur)
        return out

    def oracle_inputs(self, rows=None):
        """float64 copies of every input (optionally only the given rows and their pages).
        Per-expert weight stacks are converted lazily, one expert at a time."""
        rows = np.arange(self.w.batch) if rows is None else np.asarray(rows)
        weights = self.oracle_weights()
        n_pages = [-(-int(self.ctx[b]) // 16) for b in rows]
        pages = np.concatenate([self.page_table[b, :n] for b, n in zip(rows, n_pages)])
        sub_table = np.full((len(rows), self.max_pages), -1, dtype=np.int32)
        off = 0
        for i, n in enumerate(n_pages):
            sub_table[i, :n] = np.arange(off, off + n)
            off += n
        idx = torch.from_numpy(pages.astype(np.int64)).to(self.device)
        pools = [f64(p.index_select(0, idx)) for p in self.pools]
        return dict(weights=weights, pools=pools, page_table=sub_table, ctx=self.ctx[rows].copy(),
                    x=f64(self.x[torch.from_numpy(rows).to(self.device)]))


class LazyF64:
    """Indexable float64 view of a device tensor stack: [e] converts one slice."""

    def __init__(self, t):
        self.t = t
        self.shape = tuple(t.shape)
        self._cache = {}

    def __getitem__(self, e):
        e = int(e)
        if e not in self._cache:
            self._cache[e] = f64(self.t[e])
        return self._cache[e]


def oracle_run(inp, cfgs, a, b, live=None):
    live = {"resid": inp["x"].copy()} if live is None else live
    return O.run_ops(cfgs, inp["weights"], inp["pools"], inp["page_table"], inp["ctx"], live, a, b)
