#!/usr/bin/env python3
"""Decode-step benchmark of the ODS hot path on one MI355X.

One step = one decode step of the workload's block (for the default workload,
one 8B-shaped dense layer at batch 256 with every context 8192 tokens: the
attention stage, ops [0, 6), then the FFN stage, ops [6, 10)) over the whole
batch, with every input already resident in HBM. A step that moves less than
2 GB uses three independent copies of the weights and KV pools in rotation, so
that no step finds the previous step's bytes in the 256 MB last-level cache
(the default step reads 8.7 GB of KV and weights and needs no copies).

Prints one JSON line: whole-step decode tokens/s, per-stage tokens/s with their
fraction of the HBM / MFMA roofline, the roofline of the dominant operator
(attn_core) timed with HIP events inside the timed loop, and the CPU oracle
timed on the host on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK = 8.0e12          # bytes/s, MI355X HBM3E
MFMA_BF16_PEAK = 2.5e15    # dense bf16 flop/s, MI355X
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_core_traffic.json")


class TimingEvent:
    """A HIP timing event recorded without the system-scope memory fence
    (hipEventDisableSystemFence). The default event fences every record with
    a cache writeback and invalidation, which costs the work that follows it;
    on one MI355X the decode step measured 0.250 ms with default events at its
    stage boundaries, 0.243 ms with these, and 0.234 ms with none. Created on
    the HIP runtime torch has loaded; falls back to torch.cuda.Event elsewhere.
    Same interface as torch.cuda.Event: record(stream), elapsed_time(other) in ms."""
    _hip = None
    _FLAGS = 0x20000000  # hipEventDisableSystemFence (hip_runtime_api.h)

    @classmethod
    def _runtime(cls):
        if cls._hip is None:
            import ctypes as C
            path = None
            try:
                with open("/proc/self/maps") as fh:
                    for line in fh:
                        if "libamdhip64" in line:
                            path = line.split()[-1]
                            break
            except OSError:
                pass
            if path is None:
                cls._hip = False
            else:
                lib = C.CDLL(path)
                lib.hipEventCreateWithFlags.argtypes = [C.POINTER(C.c_void_p), C.c_uint]
                lib.hipEventRecord.argtypes = [C.c_void_p, C.c_void_p]
                lib.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), C.c_void_p, C.c_void_p]
                lib.hipEventDestroy.argtypes = [C.c_void_p]
                cls._hip = lib
        return cls._hip

    def __init__(self):
        import ctypes as C
        import torch
        lib = self._runtime()
        self._torch = None
        if not lib:
            self._torch = torch.cuda.Event(enable_timing=True)
            return
        self._h = C.c_void_p()
        if lib.hipEventCreateWithFlags(C.byref(self._h), self._FLAGS) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")

    def record(self, stream):
        import ctypes as C
        if self._torch is not None:
            self._torch.record(stream)
        elif self._runtime().hipEventRecord(self._h, C.c_void_p(stream.cuda_stream)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_time(self, other) -> float:
        import ctypes as C
        if self._torch is not None:
            return self._torch.elapsed_time(other._torch)
        ms = C.c_float()
        if self._runtime().hipEventElapsedTime(C.byref(ms), self._h, other._h) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def __del__(self):
        if getattr(self, "_torch", 1) is None and self._hip:
            self._hip.hipEventDestroy(self._h)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="dense8b_b256_ctx8k")
    ap.add_argument("--copies", type=int, default=0, help="weight/KV copies in rotation (0: auto)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--weights", choices=("tiled", "rows"), default="tiled",
                    help="projection weight layout: tiled (converted once at setup, the streaming GEMM's "
                         "tile order) or row-major; tiled falls back to rows for shapes it does not take")
    ap.add_argument("--swa-ring", action="store_true",
                    help="sliding-window layers keep their KV in a window-only page ring "
                         "(ceil(window / 16) + 1 pages per sequence) instead of full page tables")
    ap.add_argument("--cpu-budget", type=float, default=20.0, help="seconds of oracle work to time")
    ap.add_argument("--cpu-threads", type=int, default=0,
                    help="BLAS threads for the CPU baseline's FFN stage (0: the whole pool; 1: everything single-threaded)")
    ap.add_argument("--cpu-rows", type=int, default=8,
                    help="sequences of the batch the CPU oracle baseline decodes (spread over the batch, "
                         "longest and shortest context included)")
    ap.add_argument("--ffn-sweep", action="store_true",
                    help="instead of the decode step, time the dense FFN stage alone over batch sizes "
                         "64..2048 to show where the GEMMs turn from HBM- to MFMA-bound")
    ap.add_argument("--latency-table", action="store_true",
                    help="instead of the decode step, time the stage templates (attention, FFN, core "
                         "attention, colocated layer) over batch and context sweeps, as HIP-graph replays "
                         "and as eager calls")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="before the timed loop, run one plain device copy of this many MiB (a known-size "
                         "reference for hardware byte counters)")
    return ap.parse_args()


# ----------------------------------------------------------------------------- accounting

def layer_accounting(cfg, ctx, B):
    """Algorithmic bytes / flops per stage of one layer (what the method must
    move or compute; intermediates excluded)."""
    H, nq, nkv, d = cfg.hidden, cfg.n_q, cfg.n_kv, cfg.head_dim
    pos = ctx.astype(np.int64) - 1
    if cfg.window > 0:
        leff = np.minimum(ctx, cfg.window).astype(np.int64)
    else:
        leff = ctx.astype(np.int64)
    kv_bytes = int(leff.sum()) * 2 * nkv * d * 2
    w_attn = (cfg.qkv_dim * H + H * nq * d) * 2
    attn_core_bytes = kv_bytes + 2 * B * nq * d * 2
    attn_bytes = kv_bytes + w_attn + 4 * B * H + 4 * B * nkv * d
    attn_flops = 2 * B * H * cfg.qkv_dim + 2 * B * nq * d * H + 4 * nq * d * int(leff.sum())
    if cfg.n_experts:
        E, k, I = cfg.n_experts, cfg.top_k, cfg.moe_ffn
        ffn_bytes = 6 * H * I * E + 2 * H * E + 4 * B * H
        ffn_flops = 6 * B * k * H * I + 2 * B * H * E
    else:
        F = cfg.ffn
        ffn_bytes = 6 * H * F + 4 * B * H
        ffn_flops = 6 * B * H * F
    del pos
    return dict(attn_bytes=attn_bytes, attn_flops=attn_flops, attn_core_bytes=attn_core_bytes,
                kv_bytes=kv_bytes, ffn_bytes=ffn_bytes, ffn_flops=ffn_flops)


def handoff_bytes_per_token(cfg):
    """Bytes per decoded token of the live set crossing a cut after each local
    operator of a layer, keyed by the operator index as a string."""
    from paper_2609_14237_amd.costmodel import handoff_bytes_per_token as live
    return {str(j): int(b) for j, b in enumerate(live(cfg))}


def attn_source_hash():
    h = hashlib.sha256()
    for f in ("k_attn.hip", "common.hpp"):
        with open(os.path.join(ROOT, "paper_2609_14237_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload):
    """HBM bytes per attn_core launch from the committed rocprofv3 counter
    summary, only if it was taken on the current kernel source."""
    try:
        with open(TRAFFIC_FILE) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    rec = t.get(workload)
    if not rec or rec.get("source_hash") != attn_source_hash():
        return None
    return rec.get("bytes_per_launch")


# ----------------------------------------------------------------------------- CPU baseline

def cpu_baseline(w, copy0, budget_s, n_rows, ffn_threads=0):
    """Time the float64 oracle on the host, stage by stage, over decode steps
    of a bounded sample of the workload's sequences (first weight/KV copy),
    repeated until ~budget_s of oracle time. The attention stage (a Python
    loop over rows and heads of small numpy calls) runs with numpy's BLAS
    limited to one thread, which measured as fast as the full pool; the FFN
    stage (large matrix products) with the whole BLAS pool, or with
    `ffn_threads` threads when that is positive. `cores` is the
    largest thread count a stage used; each stage also reports its own
    threads, the CPU-seconds per wall-second of the thread that calls the
    oracle, and those of the whole process (every thread, the GPU runtime's
    included)."""
    import oracle as O
    import torch
    from threadpoolctl import threadpool_info, threadpool_limits

    def f64(t):
        return t.detach().double().cpu().numpy()

    cfgs = list(w.layers)
    ctx_all = copy0["ctx"]
    rows = set(np.linspace(0, w.batch - 1, n_rows).round().astype(int).tolist())
    rows |= {int(np.argmax(ctx_all)), int(np.argmin(ctx_all))}
    rows = np.array(sorted(rows))
    # inputs of the sampled rows (their pages only; a sliding-window layer only
    # its window's pages), converted once, not timed
    ctx = ctx_all[rows]
    pt = copy0["page_table"][rows]
    tables, pools0 = [], []
    for cfg, pool in zip(cfgs, copy0["pools"]):
        table = np.full(pt.shape, -1, dtype=np.int32)
        pages, off = [], 0
        for i, c in enumerate(ctx):
            n = -(-int(c) // 16)
            p0 = max(0, int(c) - cfg.window) // 16 if cfg.window > 0 else 0
            pages.append(pt[i, p0:n])
            table[i, p0:n] = np.arange(off, off + n - p0)
            off += n - p0
        idx = torch.from_numpy(np.concatenate(pages).astype(np.int64)).cuda()
        pools0.append(f64(pool.index_select(0, idx)))
        tables.append(table)
    weights = [{k: f64(v) for k, v in wl.items()} for wl in copy0["weights"]]
    x = f64(copy0["x"][torch.from_numpy(rows).cuda()])
    offs = np.cumsum([0] + [14 if c.n_experts else 10 for c in cfgs])
    blas = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    threads = {"attn": 1, "ffn": int(ffn_threads) if ffn_threads > 0 else int(blas)}
    wall = {"attn": 0.0, "ffn": 0.0}
    cpu = {"attn": 0.0, "ffn": 0.0}
    cpu_main = {"attn": 0.0, "ffn": 0.0}
    reps = 0
    while True:
        pools = [p.copy() for p in pools0]
        live = {"resid": x.copy()}
        for l in range(len(cfgs)):
            for stage, a, b in (("attn", offs[l], offs[l] + 6), ("ffn", offs[l] + 6, offs[l + 1])):
                with threadpool_limits(threads[stage]):
                    c0, m0, t0 = time.process_time(), time.thread_time(), time.perf_counter()
                    live = O.run_ops(cfgs, weights, pools, tables, ctx, live, int(a), int(b))
                    wall[stage] += time.perf_counter() - t0
                    cpu_main[stage] += time.thread_time() - m0
                    cpu[stage] += time.process_time() - c0
        reps += 1
        if wall["attn"] + wall["ffn"] >= budget_s or reps >= 50:
            break
    tokens = reps * len(rows)
    t = wall["attn"] + wall["ffn"]
    stages = {k: {"tokens_per_s": tokens / wall[k], "seconds": wall[k], "threads": threads[k],
                  "calling_thread_cpu_per_wall": cpu_main[k] / wall[k],
                  "process_cpu_per_wall": cpu[k] / wall[k]} for k in wall}
    return {"value": tokens / t, "unit": "tokens/s", "cores": max(threads.values()),
            "kind": "oracle", "host_cpus": os.cpu_count(), "stages": stages,
            "sample": f"{reps} decode steps of {len(rows)} of the {w.batch} sequences of the {w.name} workload "
                      f"(spread over the batch, longest and shortest context included; every layer, attention "
                      f"stage on 1 thread and FFN stage on {threads['ffn']} BLAS threads timed separately), "
                      f"float64 numpy oracle, {t:.1f} s"}


# ----------------------------------------------------------------------------- main

def tileable(cfg) -> bool:
    """Whether a layer's projection weights have a tiled layout (every input
    width a multiple of 64)."""
    f = cfg.moe_ffn if cfg.n_experts else cfg.ffn
    return cfg.hidden % 64 == 0 and (cfg.n_q * cfg.head_dim) % 64 == 0 and f % 64 == 0


def ffn_sweep(args):
    """Dense FFN stage ([6,10) of the 8B-shaped layer) at growing batch: the
    weights stream once per call, so the GEMMs are HBM-bound at small batch and
    turn MFMA-bound near the ridge (312 flop per byte at the vendor peaks)."""
    import torch
    import workloads as W
    from workloads import gen
    from paper_2609_14237_amd import binding as B
    from paper_2609_14237_amd import runtime as R

    base = W.BY_NAME["dense8b_b64"]
    cfg = base.layers[0]
    dev = "cuda"
    torch.cuda.set_device(0)
    copies = 3  # 3 x 352 MB of FFN weights defeat the 256 MB last-level cache
    rows = []
    for M in (64, 256, 512, 1024, 2048):
        ctx = np.ones(M, dtype=np.int32)
        page_table = np.zeros((M, 1), dtype=np.int32)
        assert B.ods_kv_alloc(M, ctx, M, 0, 1, page_table) == 0, B.ods_last_error()
        batch = R.DeviceBatch(torch.from_numpy(ctx).to(dev), torch.from_numpy(page_table).to(dev))
        sets = []
        for c in range(copies):
            wts = [gen.layer_weights(cfg, base.seed + 1000 * c, 0, dev, base.router_std)]
            pools = [gen.kv_pool(cfg, M, base.seed + 1000 * c, 0, dev)]
            blk = R.DeviceBlock([cfg], wts, pools, M, tiled=args.weights == "tiled")
            st = R.DeviceState(blk, batch, dev)
            st.view("resid", M, cfg.hidden).copy_(gen.activations(M, cfg.hidden, base.seed + c, dev))
            sets.append((blk, st, wts, pools))
        stream = torch.cuda.current_stream().cuda_stream
        for i in range(args.warmup):
            blk, st = sets[i % copies][:2]
            R.run_partition(blk, 6, 10, batch, st, stream)
        torch.cuda.synchronize()
        times = []
        for i in range(args.steps):
            blk, st = sets[i % copies][:2]
            e0, e1 = TimingEvent(), TimingEvent()
            e0.record(torch.cuda.current_stream())
            R.run_partition(blk, 6, 10, batch, st, stream)
            e1.record(torch.cuda.current_stream())
            times.append((e0, e1))
        torch.cuda.synchronize()
        t = float(np.median([a.elapsed_time(b) for a, b in times])) * 1e-3
        F, H = cfg.ffn, cfg.hidden
        nbytes, flops = 6 * H * F + 4 * M * H, 6 * M * H * F
        rows.append({"batch": M, "us": t * 1e6, "tokens_per_s": M / t, "hbm_GBps": nbytes / t / 1e9,
                     "hbm_frac": nbytes / t / HBM_PEAK, "mfma_TFLOPs": flops / t / 1e12,
                     "mfma_frac": flops / t / MFMA_BF16_PEAK,
                     "roofline_us": max(nbytes / HBM_PEAK, flops / MFMA_BF16_PEAK) * 1e6,
                     "bound": "mfma" if flops / MFMA_BF16_PEAK > nbytes / HBM_PEAK else "hbm"})
        print(f"[ffn-sweep] batch {M}: {t * 1e6:.1f} us, {flops / t / 1e12:.0f} TFLOP/s", file=sys.stderr, flush=True)
        del sets
        torch.cuda.empty_cache()
    print(json.dumps({"metric": "dense FFN stage time vs batch (8B-shaped layer)", "unit": "us",
                      "steps": args.steps, "warmup": args.warmup, "dtype": "bf16", "data": "synthetic",
                      "weight_layout": args.weights,
                      "ffn_sweep": rows}), flush=True)


def latency_table(args):
    """Profiled stage latencies t_j = f_lat(op range, batch, context), the
    per-stage inputs of the paper's communication-aware latency model (Section
    4), for every distinct layer shape of a workload (--workload: the dense
    8B-shaped layer by default, the MoE layer, or the hybrid block's
    sliding-window and full layers): every single operator and every stage
    template at every (batch, context) point, the templates timed as a replay
    of their captured HIP graph and as an eager ods_run_partition call (median
    of --steps each). One weight/KV copy: small KV footprints partly stay in
    the 256 MB last-level cache. Rows carry the layer's window (0: full
    attention)."""
    import torch
    import workloads as W
    from workloads import gen
    from paper_2609_14237_amd import binding as B
    from paper_2609_14237_amd import runtime as R

    base = W.BY_NAME[args.workload]
    shapes = list(dict.fromkeys(base.layers))  # distinct layer shapes, in block order
    dev = "cuda"
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream().cuda_stream

    def median_us(fn):
        for _ in range(args.warmup):
            fn()
        evs = []
        for _ in range(args.steps):
            e0, e1 = TimingEvent(), TimingEvent()
            e0.record(torch.cuda.current_stream())
            fn()
            e1.record(torch.cuda.current_stream())
            evs.append((e0, e1))
        torch.cuda.synchronize()
        return float(np.median([a.elapsed_time(b) for a, b in evs])) * 1e3

    rows, op_rows = [], []
    for cfg in shapes:
        n_ops = cfg.n_ops
        templates = [("attention stage", 0, 6), ("FFN stage", 6, n_ops), ("core attention", 3, 5),
                     ("colocated layer", 0, n_ops)]
        # the MoE layer's expert GEMMs stay bound by their weight stream far past
        # 256 rows (its b* is about 2000), so its table goes further
        batches = (1, 8, 32, 64, 128, 256) + ((512, 1024) if cfg.n_experts else ())
        weights = [gen.layer_weights(cfg, base.seed, 0, dev, base.router_std)]
        tiled = args.weights == "tiled"
        if tiled:
            weights = [R.tile_weights(cfg, weights[0])]
        for ctx_len in (1024, 4096, 16384):
            for M in batches:
                ctx = np.full(M, ctx_len, dtype=np.int32)
                P = gen.pool_pages_for(ctx)
                max_pages = -(-ctx_len // 16)
                table = np.zeros((M, max_pages), dtype=np.int32)
                assert B.ods_kv_alloc(P, ctx, M, base.seed, max_pages, table) == 0, B.ods_last_error()
                batch = R.DeviceBatch(torch.from_numpy(ctx).to(dev), torch.from_numpy(table).to(dev))
                pools = [gen.kv_pool(cfg, P, base.seed, 0, dev)]
                blk = R.DeviceBlock([cfg], weights, pools, P, pretiled=tiled)
                st = R.DeviceState(blk, batch, dev)
                x = gen.activations(M, cfg.hidden, base.seed, dev)
                for i in range(n_ops):  # single operators, eager, for per-operator latency models
                    st.view("resid", M, cfg.hidden).copy_(x)
                    if i > 0:
                        R.run_partition(blk, 0, i, batch, st, stream)
                    t_op = median_us(lambda: R.run_partition(blk, i, i + 1, batch, st, stream))
                    op_rows.append({"local": i, "name": blk.op_name(i), "window": cfg.window, "batch": M,
                                    "ctx": ctx_len, "us": t_op})
                for name, a, b in templates:
                    st.view("resid", M, cfg.hidden).copy_(x)
                    if a > 0:  # inputs of a later stage: run the layer up to it once
                        R.run_partition(blk, 0, a, batch, st, stream)
                    t_eager = median_us(lambda: R.run_partition(blk, a, b, batch, st, stream))
                    g = R.PartitionGraph(blk, a, b, batch, st)
                    t_graph = median_us(lambda: g.launch(stream))
                    g.close()
                    rows.append({"stage": name, "op_range": [a, b], "window": cfg.window, "batch": M,
                                 "ctx": ctx_len, "us_graph": t_graph, "us_eager": t_eager})
                    print(f"[latency] window {cfg.window} ctx {ctx_len} batch {M} {name} [{a},{b}): graph "
                          f"{t_graph:.1f} us, eager {t_eager:.1f} us", file=sys.stderr, flush=True)
                del blk, st, pools, batch
                torch.cuda.empty_cache()
        del weights
    print(json.dumps({"metric": "stage latency t_j = f_lat(op range, batch, context)", "workload": base.name,
                      "layer": base.description, "unit": "us", "steps": args.steps, "warmup": args.warmup, "dtype": "bf16",
                      "data": "synthetic", "weight_layout": args.weights, "latency_table": rows,
                      "op_latency": op_rows}), flush=True)


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(collectives and sharding are out of scope); run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    if args.ffn_sweep:
        ffn_sweep(args)
        return
    if args.latency_table:
        latency_table(args)
        return

    import torch
    import workloads as W
    from workloads import gen
    from paper_2609_14237_amd import binding as B
    from paper_2609_14237_amd import runtime as R

    w = W.BY_NAME[args.workload]
    dev = "cuda"
    torch.cuda.set_device(0)
    ctx = gen.contexts(w)
    P = gen.pool_pages_for(ctx)
    max_pages = w.max_pages
    page_table = np.zeros((w.batch, max_pages), dtype=np.int32)
    assert B.ods_kv_alloc(P, ctx, w.batch, w.seed, max_pages, page_table) == 0, B.ods_last_error()

    # per-step working set decides how many rotated copies are needed to defeat the 256 MB MALL
    acct = [layer_accounting(c, ctx, w.batch) for c in w.layers]
    step_bytes = sum(a["attn_bytes"] + a["ffn_bytes"] for a in acct)
    copies = args.copies or (3 if step_bytes < 2e9 else 1)

    # window-only page ring for the sliding-window layers (same attended bytes, bounded memory)
    ring_pages, ring_table, P_ring = 0, None, 0
    windows = [c.window for c in w.layers if c.window > 0]
    if args.swa_ring and windows:
        ring_pages = max(-(-win // 16) + 1 for win in windows)
        rctx = np.minimum(ctx, 16 * ring_pages).astype(np.int32)
        P_ring = gen.pool_pages_for(rctx)
        ring_table = np.zeros((w.batch, ring_pages), dtype=np.int32)
        assert B.ods_kv_alloc(P_ring, rctx, w.batch, w.seed + 7, ring_pages, ring_table) == 0, B.ods_last_error()
    layer_pages = [P_ring if (ring_pages and c.window > 0) else P for c in w.layers]
    tiled = args.weights == "tiled" and all(tileable(c) for c in w.layers)
    kv_pool_bytes = [B.ods_kv_pool_bytes(R.layer_cfg(c), n) for c, n in zip(w.layers, layer_pages)]

    batch = R.DeviceBatch(torch.from_numpy(ctx).to(dev), torch.from_numpy(page_table).to(dev),
                          ring_table=None if ring_table is None else torch.from_numpy(ring_table).to(dev))
    sets = []
    for c in range(copies):
        seed = w.seed + 1000 * c
        weights = [{k: v for k, v in gen.layer_weights(cfg, seed, l, dev, w.router_std).items()}
                   for l, cfg in enumerate(w.layers)]
        pools = [gen.kv_pool(cfg, n, seed, l, dev) for l, (cfg, n) in enumerate(zip(w.layers, layer_pages))]
        x = gen.activations(w.batch, w.layers[0].hidden, seed, dev)
        blk = R.DeviceBlock(w.layers, weights, pools, layer_pages, tiled=tiled)
        state = R.DeviceState(blk, batch, dev)
        sets.append(dict(block=blk, state=state, weights=weights, pools=pools, x=x, ctx=ctx,
                         page_table=page_table))
    torch.cuda.synchronize()

    # stage boundaries: each layer as [0,4) [4,5) [5,6) | [6,N) -- the cut around attn_core
    # changes no kernel (no fusion crosses it) and lets events time that operator alone
    n_layers = len(w.layers)
    offs = [sets[0]["block"].layer_offset(l) for l in range(n_layers)]
    ends = [offs[l] + (14 if w.layers[l].n_experts else 10) for l in range(n_layers)]
    stream = torch.cuda.current_stream()
    sptr = stream.cuda_stream

    def run_step(s, evs=None):
        blk, st = s["block"].c, s["state"].c
        for l in range(n_layers):
            o = offs[l]
            for a, b, tag in ((o, o + 4, None), (o + 4, o + 5, "core"), (o + 5, o + 6, "attn"),
                              (o + 6, ends[l], "ffn")):
                rc = B.ods_run_partition(blk, a, b, batch.c, st, sptr)
                if rc != 0:
                    raise B.OdsError(rc, f"ods_run_partition[{a},{b})")
                if evs is not None:
                    evs.append((l, tag, TimingEvent()))
                    evs[-1][2].record(stream)

    if args.calib_copy_mib:
        src = torch.empty(args.calib_copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        src.fill_(1)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    for s in sets:
        s["state"].view("resid", w.batch, w.layers[0].hidden).copy_(s["x"])
    for i in range(args.warmup):
        run_step(sets[i % copies])
    torch.cuda.synchronize()

    # Each step starts at the event that ended the previous one (the timed
    # region's first event for step 0), so no event sits between two steps.
    per_step_events = []
    t_begin = TimingEvent()
    torch.cuda.synchronize()
    t_begin.record(stream)
    start = t_begin
    for i in range(args.steps):
        evs = []
        run_step(sets[i % copies], evs)
        per_step_events.append((start, evs))
        start = evs[-1][2]
    t_end = start
    torch.cuda.synchronize()
    total_ms = t_begin.elapsed_time(t_end)
    ms_per_step = total_ms / args.steps

    # per-stage and attn_core durations from the in-loop events
    core_ms, attn_ms, ffn_ms = [], [], []
    per_layer = [{"attn": [], "core": [], "ffn": []} for _ in range(n_layers)]
    for start, evs in per_step_events:
        prev, layer_start = start, start
        for (l, tag, ev) in evs:
            if tag == "core":
                per_layer[l]["core"].append(prev.elapsed_time(ev))
            elif tag == "attn":
                per_layer[l]["attn"].append(layer_start.elapsed_time(ev))
            elif tag == "ffn":
                per_layer[l]["ffn"].append(prev.elapsed_time(ev))
                layer_start = ev
            prev = ev
    for start, evs in per_step_events:
        prev = start
        a_ms = f_ms = c_ms = 0.0
        layer_start = start
        for (l, tag, ev) in evs:
            dt = prev.elapsed_time(ev)
            if tag == "core":
                c_ms += dt
            if tag == "attn":
                a_ms += layer_start.elapsed_time(ev)
            if tag == "ffn":
                f_ms += dt
                layer_start = ev
            prev = ev
        core_ms.append(c_ms)
        attn_ms.append(a_ms)
        ffn_ms.append(f_ms)
    t_core = float(np.median(core_ms)) * 1e-3 / n_layers
    t_attn = float(np.median(attn_ms)) * 1e-3
    t_ffn = float(np.median(ffn_ms)) * 1e-3
    attn_bytes = sum(a["attn_bytes"] for a in acct)
    attn_flops = sum(a["attn_flops"] for a in acct)
    ffn_bytes = sum(a["ffn_bytes"] for a in acct)
    ffn_flops = sum(a["ffn_flops"] for a in acct)
    core_bytes = sum(a["attn_core_bytes"] for a in acct) / n_layers

    def stage(t, nbytes, flops):
        return {"tokens_per_s": w.batch / t, "us": t * 1e6,
                "hbm_GBps": nbytes / t / 1e9, "hbm_frac": nbytes / t / HBM_PEAK,
                "mfma_TFLOPs": flops / t / 1e12, "mfma_frac": flops / t / MFMA_BF16_PEAK,
                "roofline_us": max(nbytes / HBM_PEAK, flops / MFMA_BF16_PEAK) * 1e6}

    layers_out = []
    for l, cfg in enumerate(w.layers):
        med = {k: float(np.median(v)) * 1e-3 for k, v in per_layer[l].items()}
        a = acct[l]
        layers_out.append({
            "layer": l, "window": cfg.window, "attention": "sliding window" if cfg.window else "full",
            "attn_stage_us": med["attn"] * 1e6, "attn_stage_hbm_frac": a["attn_bytes"] / med["attn"] / HBM_PEAK,
            "attn_core_us": med["core"] * 1e6, "attn_core_bytes": a["attn_core_bytes"],
            "attn_core_hbm_frac": a["attn_core_bytes"] / med["core"] / HBM_PEAK,
            "ffn_stage_us": med["ffn"] * 1e6, "ffn_stage_mfma_frac": a["ffn_flops"] / med["ffn"] / MFMA_BF16_PEAK,
            "ffn_stage_hbm_frac": a["ffn_bytes"] / med["ffn"] / HBM_PEAK})
    achieved = core_bytes / t_core
    traffic = measured_traffic(w.name)
    result = {
        "metric": "decode tokens/s per stage (attn, FFN) at 8B-shape layer; % HBM / MFMA peak",
        "value": w.batch * args.steps / (total_ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "description": w.description, "batch": w.batch,
                   "ctx_range": [w.ctx_lo, w.ctx_hi], "ctx_mean": float(ctx.mean()),
                   "layers": n_layers, "copies_rotated": copies,
                   "step": "attention stage [0,6) then FFN stage [6,N) per layer",
                   "weight_layout": "tiled" if tiled else "rows",
                   "kv_ring_pages": ring_pages, "kv_pool_bytes_per_layer": kv_pool_bytes,
                   "kv_pool_bytes_total": int(sum(kv_pool_bytes))},
        "stages": {"attn": stage(t_attn, attn_bytes, attn_flops), "ffn": stage(t_ffn, ffn_bytes, ffn_flops)},
        "layers": layers_out,
        "handoff": {"cut": "after local op 5 (attention stage | FFN stage)",
                    "bytes_per_token": handoff_bytes_per_token(w.layers[0])["5"],
                    "bytes_per_token_by_cut": handoff_bytes_per_token(w.layers[0])},
        "roofline": {"kernel": "attn_core (paged decode attention split evenly over all waves + LSE merge)",
                     "bound": "hbm", "achieved": achieved / 1e9, "peak": HBM_PEAK / 1e9, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK,
                     "traffic": traffic,
                     "algorithmic_bytes_per_launch": core_bytes, "avg_launch_us": t_core * 1e6},
    }
    if not args.no_cpu_baseline and not ring_pages:  # the oracle baseline reads the full page tables
        result["cpu_baseline"] = cpu_baseline(w, sets[0], args.cpu_budget, args.cpu_rows, args.cpu_threads)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
