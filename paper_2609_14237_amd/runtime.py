"""PyTorch-side marshalling around the C ABI: packs device tensors into the
ods_* structs and allocates the live buffers and workspace the library sizes.
No operator of the decode step is computed here."""
from __future__ import annotations

import ctypes as C

import torch

from . import binding as _b
from .binding import ods_batch, ods_block, ods_layer, ods_layer_cfg, ods_state


def layer_cfg(cfg) -> ods_layer_cfg:
    """ods_layer_cfg from any object with the layer-shape attributes."""
    return ods_layer_cfg(cfg.hidden, cfg.n_q, cfg.n_kv, cfg.head_dim, cfg.ffn, cfg.n_experts, cfg.top_k,
                         cfg.moe_ffn, cfg.window, cfg.rope_theta, cfg.rms_eps)


def _ptr(t):
    if t is None:
        return None
    return t.data_ptr()


def _tile_shapes(cfg):
    """(out, in, gated, groups) of each projection weight, as ods_tile_weight takes them."""
    qkv = (cfg.n_q + 2 * cfg.n_kv) * cfg.head_dim
    H, E = cfg.hidden, cfg.n_experts
    shapes = {"w_qkv": (qkv, H, 0, 1), "w_o": (H, cfg.n_q * cfg.head_dim, 0, 1)}
    if E:
        shapes.update(w_gate_up=(cfg.moe_ffn, H, 1, E), w_down=(H, cfg.moe_ffn, 0, E))
    else:
        shapes.update(w_gate_up=(cfg.ffn, H, 1, 1), w_down=(H, cfg.ffn, 0, 1))
    return shapes


def tile_weights(cfg, w: dict, stream=None) -> dict:
    """Tiled copies (ODS_WEIGHTS_TILED) of a layer's projection weights, converted
    by ods_tile_weight on the device; the other entries of w are passed through."""
    stream = stream if stream is not None else torch.cuda.current_stream()
    out = dict(w)
    for name, (o, i, gated, groups) in _tile_shapes(cfg).items():
        src = w[name]
        n = _b.ods_tiled_weight_bytes(o, i, gated, groups)
        if n == 0:
            raise ValueError(f"{name}: no tiled layout for out={o}, in={i} (in must be a multiple of 64)")
        dst = torch.empty(n // 2, dtype=torch.bfloat16, device=src.device)
        _b._check(_b.ods_tile_weight(src.data_ptr(), dst.data_ptr(), o, i, gated, groups, stream.cuda_stream),
                  f"ods_tile_weight({name})")
        out[name] = dst
    return out


class DeviceBlock:
    """ods_block over per-layer weight dicts and KV pools (tensors stay referenced).
    pool_pages is one count for every layer or a list with one per layer. With
    tiled=True the projection weights are converted once into the tiled layout
    (ODS_WEIGHTS_TILED) the weight-streaming GEMM reads fastest, and the block
    references those copies; pretiled=True takes weights tile_weights() already
    converted."""

    def __init__(self, cfgs, weights, pools, pool_pages, tiled: bool = False, pretiled: bool = False):
        self.cfgs = list(cfgs)
        self.tiled = tiled or pretiled
        self.weights = [tile_weights(c, w) if tiled and not pretiled else w for c, w in zip(self.cfgs, weights)]
        self.pools = list(pools)
        n = len(self.cfgs)
        pages = list(pool_pages) if isinstance(pool_pages, (list, tuple)) else [pool_pages] * n
        self._layers = (ods_layer * n)()
        for i, (cfg, w, pool) in enumerate(zip(self.cfgs, self.weights, self.pools)):
            L = self._layers[i]
            L.cfg = layer_cfg(cfg)
            for name in ("g_attn", "w_qkv", "w_o", "g_ffn", "w_gate_up", "w_down", "w_router"):
                setattr(L, name, _ptr(w.get(name)))
            L.kv_pool = _ptr(pool)
            L.pool_pages = pages[i] if pool is not None else 0
            L.weight_layout = _b.ODS_WEIGHTS_TILED if self.tiled else _b.ODS_WEIGHTS_ROWS
        self.c = ods_block(n, C.cast(self._layers, C.POINTER(ods_layer)))

    def num_ops(self) -> int:
        return _b.ods_block_num_ops(self.c)

    def op_name(self, op: int):
        return _b.ods_op_name(self.c, op)

    def layer_offset(self, layer: int) -> int:
        return sum(14 if c.n_experts else 10 for c in self.cfgs[:layer])


class DeviceBatch:
    """ods_batch over device int32 ctx_lens [B] and page_table [B, max_pages], and
    optionally a window-only page ring [B, ring_pages] for sliding-window layers."""

    def __init__(self, ctx_lens: torch.Tensor, page_table: torch.Tensor, split_pages: int = 0,
                 ring_table: torch.Tensor | None = None):
        assert ctx_lens.dtype == torch.int32 and page_table.dtype == torch.int32
        self.ctx_lens = ctx_lens.contiguous()
        self.page_table = page_table.contiguous()
        self.ring_table = None if ring_table is None else ring_table.contiguous()
        B, max_pages = self.page_table.shape
        ring_pages = 0
        if self.ring_table is not None:
            assert self.ring_table.dtype == torch.int32 and self.ring_table.shape[0] == B
            ring_pages = self.ring_table.shape[1]
        self.c = ods_batch(B, max_pages, _ptr(self.ctx_lens), _ptr(self.page_table), split_pages, ring_pages,
                           _ptr(self.ring_table))

    @property
    def batch(self) -> int:
        return self.c.batch


_BUF_DTYPE = {"logits": torch.float32, "topk_w": torch.float32, "topk_ids": torch.int32,
              "perm": torch.int32, "slot_pos": torch.int32, "expert_off": torch.int32}


class DeviceState:
    """Live buffers sized by ods_live_bytes and a workspace of ods_workspace_bytes."""

    def __init__(self, block: DeviceBlock, batch: DeviceBatch, device="cuda", fill=None):
        self.buffers = {}
        for i, name in enumerate(_b.BUFFERS):
            nbytes = _b.ods_live_bytes(block.c, batch.batch, i)
            if nbytes == 0:
                continue
            dt = _BUF_DTYPE.get(name, torch.bfloat16)
            n = nbytes // torch.tensor([], dtype=dt).element_size()
            t = torch.empty(n, dtype=dt, device=device)
            if fill is not None:
                t.fill_(fill if dt != torch.int32 else -7)
            self.buffers[name] = t
        self.ws_bytes = _b.ods_workspace_bytes(block.c, batch.c)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        self.c = ods_state()
        for name, t in self.buffers.items():
            setattr(self.c, name, t.data_ptr())
        self.c.ws = self.ws.data_ptr()
        self.c.ws_bytes = self.ws_bytes

    def view(self, name: str, *shape):
        t = self.buffers[name]
        n = 1
        for s in shape:
            n *= s
        return t[:n].view(*shape)


def current_stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def run_partition(block: DeviceBlock, op_begin: int, op_end: int, batch: DeviceBatch, state: DeviceState,
                  stream: int | None = None) -> None:
    st = _b.ods_run_partition(block.c, op_begin, op_end, batch.c, state.c,
                              current_stream() if stream is None else stream)
    _b._check(st, f"ods_run_partition[{op_begin},{op_end})")


def run_partition_scratch(block: DeviceBlock, op_begin: int, op_end: int, batch: DeviceBatch, state: DeviceState,
                          stream: int | None = None) -> None:
    """ods_run_partition_scratch: the same range on the library's own workspace (state.ws is not used)."""
    st = _b.ods_run_partition_scratch(block.c, op_begin, op_end, batch.c, state.c,
                                      current_stream() if stream is None else stream)
    _b._check(st, f"ods_run_partition_scratch[{op_begin},{op_end})")


def attn_stage(block, layer, batch, state, stream=None) -> None:
    st = _b.ods_attn_stage(block.c, layer, batch.c, state.c, current_stream() if stream is None else stream)
    _b._check(st, f"ods_attn_stage({layer})")


def ffn_stage(block, layer, batch, state, stream=None) -> None:
    st = _b.ods_ffn_stage(block.c, layer, batch.c, state.c, current_stream() if stream is None else stream)
    _b._check(st, f"ods_ffn_stage({layer})")


class PartitionGraph:
    """Operators [op_begin, op_end) captured once as a HIP graph; launch()
    replays them on a stream with the buffers bound at capture. Rewrite the
    device contents (resid, ctx_lens, page_table) between launches; keep the
    block, batch and state objects (and their buffers) alive while the graph is."""

    def __init__(self, block: DeviceBlock, op_begin: int, op_end: int, batch: DeviceBatch, state: DeviceState):
        st, h = _b.ods_partition_graph(block.c, op_begin, op_end, batch.c, state.c)
        _b._check(st, f"ods_partition_graph[{op_begin},{op_end})")
        self.handle = h
        self._keep = (block, batch, state)

    def launch(self, stream: int | None = None) -> None:
        _b._check(_b.ods_graph_launch(self.handle, current_stream() if stream is None else stream), "ods_graph_launch")

    def close(self) -> None:
        if self.handle:
            _b.ods_graph_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
