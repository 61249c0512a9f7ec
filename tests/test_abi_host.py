"""Host-side checks of the C ABI that need no GPU: the library loads and exports
every symbol the header declares, the page allocator agrees bit-for-bit with
the oracle's independent implementation, buffer sizing, and every argument
error path (all of which return before anything is enqueued)."""
import ctypes as C
import os
import re
from dataclasses import replace

import numpy as np
import pytest

import oracle as O
import workloads as W
from workloads import gen

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

B = pytest.importorskip("paper_2609_14237_amd.binding")
from paper_2609_14237_amd import runtime as R  # noqa: E402


def header_functions():
    text = open(os.path.join(ROOT, "include", "ods.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ods_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = header_functions()
    assert len(names) >= 10
    lib = C.CDLL(B.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(B.SIGNATURES)


@pytest.mark.parametrize("w", W.ALL + W.SHARES, ids=lambda w: w.name)
def test_kv_alloc_matches_oracle_bit_exactly(w):
    ctx = gen.contexts(w)
    P = gen.pool_pages_for(ctx)
    table = np.zeros((w.batch, w.max_pages), dtype=np.int32)
    assert B.ods_kv_alloc(P, ctx, w.batch, w.seed, w.max_pages, table) == B.ODS_OK
    np.testing.assert_array_equal(table, O.kv_alloc(ctx, P, w.seed, w.max_pages))


def test_kv_alloc_small_vector_and_errors():
    ctx = np.array([20, 16, 1, 33], dtype=np.int32)
    t = np.zeros((4, 3), dtype=np.int32)
    assert B.ods_kv_alloc(10, ctx, 4, 0, 3, t) == B.ODS_OK
    np.testing.assert_array_equal(t, O.kv_alloc(ctx, 10, 0, 3))
    assert B.ods_kv_alloc(5, ctx, 4, 0, 3, t) == B.ODS_ENOMEM
    assert B.ods_kv_alloc(10, ctx, 4, 0, 2, t) == B.ODS_ERANGE
    bad = np.array([20, 0], dtype=np.int32)
    assert B.ods_kv_alloc(10, bad, 2, 0, 3, t) == B.ODS_EINVAL
    assert B.lib.ods_kv_alloc(10, None, 4, 0, 3, t.ctypes.data_as(C.POINTER(C.c_int32))) == B.ODS_EINVAL
    assert "pool" in B.ods_last_error() or "null" in B.ods_last_error()


FAKE = 0x10000  # an aligned, never-dereferenced address: every call below fails validation first


def fake_block(cfgs):
    ws = [{k: FAKE_T for k in ("g_attn", "w_qkv", "w_o", "g_ffn", "w_gate_up", "w_down", "w_router")}
          for _ in cfgs]
    return R.DeviceBlock(cfgs, ws, [FAKE_T] * len(cfgs), 100)


class _FakeTensor:
    def data_ptr(self):
        return FAKE


FAKE_T = _FakeTensor()


def fake_state(**override):
    s = B.ods_state()
    for name in B.BUFFERS:
        setattr(s, name, FAKE)
    s.ws = FAKE
    s.ws_bytes = 1 << 40
    for k, v in override.items():
        setattr(s, k, v)
    return s


def fake_batch(batch=4, max_pages=8):
    return B.ods_batch(batch, max_pages, FAKE, FAKE, 0)


def test_block_ops_and_names():
    blk = fake_block(W.HYBRID_4L.layers)
    assert blk.num_ops() == 40
    assert blk.op_name(4) == "attn_core" and blk.op_name(39) == "down_residual"
    assert blk.op_name(40) is None
    moe = fake_block(W.MOE_B512.layers)
    assert moe.num_ops() == 14
    assert [moe.op_name(i) for i in range(7, 14)] == ["router", "topk_softmax", "moe_permute", "expert_gate_up",
                                                      "silu_mul", "expert_down", "moe_combine_residual"]


@pytest.mark.parametrize("rng", [(-1, 3), (0, 0), (5, 4), (0, 11), (10, 11)])
def test_range_errors(rng):
    blk = fake_block(W.TINY.layers)
    st = B.ods_run_partition(blk.c, rng[0], rng[1], fake_batch(), fake_state(), 0)
    assert st == B.ODS_ERANGE


@pytest.mark.parametrize("buf,op", [("xn", (0, 1)), ("qkv", (1, 2)), ("o", (4, 5)), ("resid", (5, 6)),
                                    ("hn", (6, 7)), ("act", (7, 9)), ("gu", (7, 8)), ("ws", (4, 5))])
def test_null_live_buffer_is_rejected(buf, op):
    blk = fake_block(W.TINY.layers)
    st = B.ods_run_partition(blk.c, op[0], op[1], fake_batch(), fake_state(**{buf: None}), 0)
    assert st == B.ODS_EINVAL
    assert buf in B.ods_last_error()


def test_misaligned_pointer_is_rejected():
    blk = fake_block(W.TINY.layers)
    st = B.ods_run_partition(blk.c, 0, 1, fake_batch(), fake_state(xn=FAKE + 2), 0)
    assert st == B.ODS_EINVAL and "aligned" in B.ods_last_error()


def test_unsupported_shapes():
    for cfg in (replace(W.TINY.layers[0], head_dim=96), replace(W.TINY.layers[0], n_q=5),
                replace(W.TINY.layers[0], n_q=64, n_kv=2), replace(W.TINY.layers[0], ffn=690),
                replace(W.MOE_B512.layers[0], top_k=65, n_experts=128)):
        blk = fake_block([cfg])
        assert B.ods_run_partition(blk.c, 0, 1, fake_batch(), fake_state(), 0) == B.ODS_EUNSUPPORTED


def test_attention_batch_limit():
    blk = fake_block(W.TINY.layers)
    assert B.ods_run_partition(blk.c, 4, 5, fake_batch(4097), fake_state(), 0) == B.ODS_EUNSUPPORTED
    assert "4096" in B.ods_last_error()
    # the limit is attn_core's: the other operators take larger batches
    assert B.ods_run_partition(blk.c, 4, 5, fake_batch(4096), fake_state(ws_bytes=0), 0) == B.ODS_ENOMEM


def test_empty_batch_passes_validation_and_enqueues_nothing():
    """batch = 0 returns ODS_OK once the block and range are valid, before any
    device call, and reads no batch or state pointer (null ones included). The
    pointers here are fake, so the case runs only where no GPU is visible;
    tests/test_gpu_edges.py runs it on real buffers."""
    import torch
    if torch.cuda.is_available():
        pytest.skip("fake device pointers: covered on real buffers by the GPU test")
    for wl in (W.TINY, W.MOE_B512, W.HYBRID_4L):
        blk = fake_block(wl.layers)
        assert B.ods_run_partition(blk.c, 0, blk.num_ops(), fake_batch(0), fake_state(), 0) == B.ODS_OK
        assert B.ods_attn_stage(blk.c, 0, fake_batch(0), fake_state(), 0) == B.ODS_OK
        assert B.ods_ffn_stage(blk.c, 0, fake_batch(0), fake_state(), 0) == B.ODS_OK
    blk = fake_block(W.TINY.layers)
    nulls = {name: None for name in B.BUFFERS}
    assert B.ods_run_partition(blk.c, 0, 10, B.ods_batch(0, 0, None, None, 0), fake_state(ws=None, **nulls),
                               0) == B.ODS_OK
    # the block and the range are still checked
    assert B.ods_run_partition(blk.c, 0, 11, fake_batch(0), fake_state(), 0) == B.ODS_ERANGE


def test_workspace_too_small():
    blk = fake_block(W.DENSE_8B_B64.layers)
    batch = fake_batch(64, 256)
    need = B.ods_workspace_bytes(blk.c, batch)
    assert need > 0
    st = B.ods_run_partition(blk.c, 4, 5, batch, fake_state(ws_bytes=need - 1), 0)
    assert st == B.ODS_ENOMEM


def test_buffer_sizes():
    blk = fake_block(W.MOE_B512.layers)
    n = 512
    assert B.ods_live_bytes(blk.c, n, B.BUFFERS.index("resid")) == n * 4096 * 2
    assert B.ods_live_bytes(blk.c, n, B.BUFFERS.index("qkv")) == n * (32 + 8) * 128 * 2
    assert B.ods_live_bytes(blk.c, n, B.BUFFERS.index("xp")) == n * 8 * 4096 * 2
    assert B.ods_live_bytes(blk.c, n, B.BUFFERS.index("expert_off")) == 65 * 4
    assert B.ods_live_bytes(blk.c, n, B.BUFFERS.index("gu")) == 0
    cfg = R.layer_cfg(W.DENSE_8B_B64.layers[0])
    assert B.ods_kv_pool_bytes(cfg, 10) == 10 * 2 * 8 * 16 * 128 * 2


def test_bench_handoff_bytes_match_the_live_set_table():
    """Live-set bytes per token at each cut of the dense 8B-shaped layer: the
    residual stream (8 KiB) plus what later operators of the layer still read."""
    import bench
    t = bench.handoff_bytes_per_token(W.BY_NAME["dense8b_b64"].layers[0])
    KiB = 1024
    assert [t[str(j)] for j in range(10)] == [16 * KiB, 20 * KiB, 20 * KiB, 16 * KiB, 16 * KiB, 8 * KiB,
                                              16 * KiB, 64 * KiB, 36 * KiB, 8 * KiB]
    m = bench.handoff_bytes_per_token(W.BY_NAME["moe64x8_b512"].layers[0])
    assert len(m) == 14 and m["5"] == m["13"] == 8 * KiB
    assert m["9"] == 8 * KiB + 8 * 8 * KiB + 64  # xp rows of the k = 8 slots, routing weights and slots


def test_graph_entry_points_reject_null_handles():
    blk = fake_block(W.TINY.layers)
    batch, state = fake_batch(), fake_state()
    assert B.lib.ods_partition_graph(C.byref(blk.c), 0, 1, C.byref(batch), C.byref(state), None) == B.ODS_EINVAL
    assert B.ods_graph_launch(None, 0) == B.ODS_EINVAL
    assert B.ods_graph_destroy(None) == B.ODS_OK


def test_ring_pages_validation():
    """A window-only ring must hold the window's pages plus the next one."""
    from dataclasses import replace as _r
    cfg = _r(W.TINY.layers[0], window=64)  # needs ceil(64 / 16) + 1 = 5 ring pages
    blk = fake_block([cfg])
    for ring in (4, -1):
        batch = B.ods_batch(4, 8, FAKE, FAKE, 0, ring, FAKE)
        assert B.ods_run_partition(blk.c, 4, 5, batch, fake_state(), 0) == B.ODS_EINVAL, ring
        assert "ring" in B.ods_last_error()
    # a ring with a null table is rejected by name for the KV operators of a window layer
    batch = B.ods_batch(4, 8, FAKE, FAKE, 0, 5, None)
    assert B.ods_run_partition(blk.c, 3, 4, batch, fake_state(), 0) == B.ODS_EINVAL
    assert "ring_table" in B.ods_last_error()
    # full-attention layers ignore the ring (no validation against it)
    full = fake_block([W.TINY.layers[0]])
    batch = B.ods_batch(4, 8, FAKE, FAKE, 0, 1, None)
    assert B.ods_workspace_bytes(full.c, batch) > 0


def test_tiled_weight_sizes_and_errors():
    """16 KB per (slab, N tile, 64-wide K step); N tiles of 128 rows, or 64 gate
    plus 64 up rows for a gated weight, with the last tile zero-padded."""
    KB16 = 16 * 1024
    assert B.ods_tiled_weight_bytes(4096, 4096, 0, 1) == 32 * 64 * KB16
    assert B.ods_tiled_weight_bytes(14336, 4096, 1, 1) == 224 * 64 * KB16
    assert B.ods_tiled_weight_bytes(1536, 4096, 1, 64) == 64 * 24 * 64 * KB16
    assert B.ods_tiled_weight_bytes(130, 128, 0, 3) == 3 * 2 * 2 * KB16
    assert B.ods_tiled_weight_bytes(65, 64, 1, 1) == 2 * 1 * KB16
    far = FAKE + (1 << 32)
    for args in [(0, 64, 0, 1), (64, 96, 0, 1), (64, 0, 0, 1), (64, 64, 2, 1), (64, 64, 0, 0)]:
        assert B.ods_tiled_weight_bytes(*args) == 0, args
        assert B.ods_tile_weight(FAKE, far, *args, 0) == B.ODS_EINVAL, args
    assert B.ods_tile_weight(None, far, 64, 64, 0, 1, 0) == B.ODS_EINVAL
    assert B.ods_tile_weight(FAKE + 2, far, 64, 64, 0, 1, 0) == B.ODS_EINVAL
    assert "aligned" in B.ods_last_error()
    assert B.ods_tile_weight(FAKE, FAKE + 4096, 64, 64, 0, 1, 0) == B.ODS_EINVAL  # dst overlaps src
    assert "overlap" in B.ods_last_error()


def test_tiled_layout_validation():
    """Tiled weights need every projection's input width to be a multiple of 64;
    an unknown layout value is rejected."""
    tiny = fake_block(W.TINY.layers)  # ffn 688 = 10.75 x 64
    tiny._layers[0].weight_layout = B.ODS_WEIGHTS_TILED
    assert B.ods_run_partition(tiny.c, 0, 1, fake_batch(), fake_state(), 0) == B.ODS_EUNSUPPORTED
    assert "multiples of 64" in B.ods_last_error()
    assert B.ods_workspace_bytes(tiny.c, fake_batch()) == 0
    odd = fake_block([replace(W.TINY.layers[0], ffn=704)])
    odd._layers[0].weight_layout = 7
    assert B.ods_run_partition(odd.c, 0, 1, fake_batch(), fake_state(), 0) == B.ODS_EINVAL
    assert "weight_layout" in B.ods_last_error()
    moe = fake_block([replace(W.MOE_B512.layers[0], moe_ffn=1544)])
    moe._layers[0].weight_layout = B.ODS_WEIGHTS_TILED
    assert B.ods_run_partition(moe.c, 0, 1, fake_batch(), fake_state(), 0) == B.ODS_EUNSUPPORTED
    ok = fake_block(W.DENSE_8B_B64.layers)
    ok._layers[0].weight_layout = B.ODS_WEIGHTS_TILED
    assert B.ods_workspace_bytes(ok.c, fake_batch(64, 256)) > 0


def test_bench_refuses_more_than_one_gpu():
    """The benchmark measures one GPU; --gpus N > 1 exits with a message before
    touching a device."""
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)


def test_scratch_entry_point_validates_before_touching_the_device():
    """ods_run_partition_scratch rejects what ods_run_partition rejects, and a
    range whose workspace exceeds the library's scratch, before any device call."""
    blk = fake_block(W.TINY.layers)
    assert B.ods_run_partition_scratch(blk.c, 0, 0, fake_batch(), fake_state(), 0) == B.ODS_ERANGE
    assert B.lib.ods_run_partition_scratch(C.byref(blk.c), 0, 4, None, C.byref(fake_state()), 0) == B.ODS_EINVAL
    # the 8B-shaped layer at batch 4096 needs more than the 64 MiB the library holds
    big = fake_block(W.DENSE_8B_B256.layers)
    batch = fake_batch(4096, 512)
    assert B.ods_workspace_bytes(big.c, batch) > B.SCRATCH_BYTES
    assert B.ods_run_partition_scratch(big.c, 0, 10, batch, fake_state(ws=None, ws_bytes=0), 0) == B.ODS_ENOMEM
    assert "scratch" in B.ods_last_error()
    # every evaluated block fits
    for w in W.ALL + W.SHARES:
        blk = fake_block(w.layers)
        assert 0 < B.ods_workspace_bytes(blk.c, fake_batch(w.batch, w.max_pages)) <= B.SCRATCH_BYTES, w.name


def test_kv_alloc_worked_example_in_the_library():
    """The library's allocator reproduces the specification's worked example
    (tests/golden/kv_alloc_worked_example.txt), independently of the oracle."""
    rows = [l.split() for l in open(os.path.join(ROOT, "tests", "golden", "kv_alloc_worked_example.txt"))
            if l.strip() and not l.startswith("#")]
    ex = {}
    pages = []
    for key, *vals in rows:
        if key == "pages":
            pages.append([int(v) for v in vals])
        else:
            ex[key] = [int(v, 0) for v in vals]
    ctx = np.array(ex["contexts"], dtype=np.int32)
    table = np.zeros((len(ctx), 3), dtype=np.int32)
    assert B.ods_kv_alloc(ex["pool_pages"][0], ctx, len(ctx), ex["seed"][0], 3, table) == B.ODS_OK
    for b, want in enumerate(pages):
        assert table[b, :len(want)].tolist() == want
        assert (table[b, len(want):] == -1).all()
