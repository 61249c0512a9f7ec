"""Test plumbing: put a workload on the GPU through the C ABI, and hand the
same seeded inputs to the CPU oracle as float64 arrays."""
from __future__ import annotations

import numpy as np
import torch

import oracle as O
import workloads as W
from workloads import gen


def f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def rel_err(gpu, ref) -> float:
    """max |gpu - ref| / max |ref| (normwise), inf if gpu is not finite."""
    g = np.asarray(gpu, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    if not np.isfinite(g).all():
        return float("inf")
    den = np.abs(r).max()
    return float(np.abs(g - r).max() / (den if den > 0 else 1.0))


TOL = 1e-2


def assert_close(name, gpu, ref, tol=TOL):
    e = rel_err(gpu, ref)
    assert e <= tol, f"{name}: max rel err {e:.3e} > {tol}"
    return e


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
    def oracle_inputs(self, rows=None):
        """float64 copies of every input (optionally only the given rows and their pages).
        Per-expert weight stacks are converted lazily, one expert at a time."""
        rows = np.arange(self.w.batch) if rows is None else np.asarray(rows)
        weights = [{k: (LazyF64(v) if v.dim() == 3 else f64(v)) for k, v in w.items()} for w in self.weights]
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
