"""ctypes binding of libods.so: the C ABI declared in include/ods.h, same names.

Argument marshalling only. Every operator of the decode path runs in the HIP
library; PyTorch is used here for device memory and streams. Importing this
module fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libods.so")

ODS_OK, ODS_EINVAL, ODS_ERANGE, ODS_ENOMEM, ODS_EUNSUPPORTED, ODS_EHIP = 0, -1, -2, -3, -4, -5
STATUS_NAMES = {0: "ODS_OK", -1: "ODS_EINVAL", -2: "ODS_ERANGE", -3: "ODS_ENOMEM",
                -4: "ODS_EUNSUPPORTED", -5: "ODS_EHIP"}
PAGE_TOKENS = 16
SCRATCH_BYTES = 64 << 20  # ODS_SCRATCH_BYTES
ODS_WEIGHTS_ROWS, ODS_WEIGHTS_TILED = 0, 1

BUFFERS = ("resid", "xn", "qkv", "o", "hn", "gu", "act", "logits", "topk_w", "topk_ids", "perm",
           "slot_pos", "expert_off", "xp", "gu_p", "act_p", "yp")


class ods_layer_cfg(C.Structure):
    _fields_ = [("hidden", C.c_int32), ("n_q", C.c_int32), ("n_kv", C.c_int32), ("head_dim", C.c_int32),
                ("ffn", C.c_int32), ("n_experts", C.c_int32), ("top_k", C.c_int32), ("moe_ffn", C.c_int32),
                ("window", C.c_int32), ("rope_theta", C.c_float), ("rms_eps", C.c_float)]


class ods_layer(C.Structure):
    _fields_ = [("cfg", ods_layer_cfg),
                ("g_attn", C.c_void_p), ("w_qkv", C.c_void_p), ("w_o", C.c_void_p), ("g_ffn", C.c_void_p),
                ("w_gate_up", C.c_void_p), ("w_down", C.c_void_p), ("w_router", C.c_void_p),
                ("kv_pool", C.c_void_p), ("pool_pages", C.c_int64), ("weight_layout", C.c_int32)]


class ods_block(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("layers", C.POINTER(ods_layer))]


class ods_batch(C.Structure):
    _fields_ = [("batch", C.c_int32), ("max_pages", C.c_int32), ("ctx_lens", C.c_void_p),
                ("page_table", C.c_void_p), ("split_pages", C.c_int32), ("ring_pages", C.c_int32),
                ("ring_table", C.c_void_p)]


class ods_state(C.Structure):
    _fields_ = [("resid", C.c_void_p), ("xn", C.c_void_p), ("qkv", C.c_void_p), ("o", C.c_void_p),
                ("hn", C.c_void_p), ("gu", C.c_void_p), ("act", C.c_void_p),
                ("logits", C.c_void_p), ("topk_w", C.c_void_p),
                ("topk_ids", C.c_void_p), ("perm", C.c_void_p), ("slot_pos", C.c_void_p),
                ("expert_off", C.c_void_p),
                ("xp", C.c_void_p), ("gu_p", C.c_void_p), ("act_p", C.c_void_p), ("yp", C.c_void_p),
                ("ws", C.c_void_p), ("ws_bytes", C.c_size_t)]


# Every symbol include/ods.h declares, with its ctypes signature.
SIGNATURES = {
    "ods_kv_alloc": (C.c_int, [C.c_int64, C.POINTER(C.c_int32), C.c_int32, C.c_uint64, C.c_int32,
                               C.POINTER(C.c_int32)]),
    "ods_kv_pool_bytes": (C.c_size_t, [C.POINTER(ods_layer_cfg), C.c_int64]),
    "ods_live_bytes": (C.c_size_t, [C.POINTER(ods_block), C.c_int32, C.c_int]),
    "ods_workspace_bytes": (C.c_size_t, [C.POINTER(ods_block), C.POINTER(ods_batch)]),
    "ods_block_num_ops": (C.c_int32, [C.POINTER(ods_block)]),
    "ods_op_name": (C.c_char_p, [C.POINTER(ods_block), C.c_int32]),
    "ods_run_partition": (C.c_int, [C.POINTER(ods_block), C.c_int32, C.c_int32, C.POINTER(ods_batch),
                                    C.POINTER(ods_state), C.c_void_p]),
    "ods_run_partition_scratch": (C.c_int, [C.POINTER(ods_block), C.c_int32, C.c_int32, C.POINTER(ods_batch),
                                            C.POINTER(ods_state), C.c_void_p]),
    "ods_attn_stage": (C.c_int, [C.POINTER(ods_block), C.c_int32, C.POINTER(ods_batch),
                                 C.POINTER(ods_state), C.c_void_p]),
    "ods_ffn_stage": (C.c_int, [C.POINTER(ods_block), C.c_int32, C.POINTER(ods_batch),
                                C.POINTER(ods_state), C.c_void_p]),
    "ods_partition_graph": (C.c_int, [C.POINTER(ods_block), C.c_int32, C.c_int32, C.POINTER(ods_batch),
                                      C.POINTER(ods_state), C.POINTER(C.c_void_p)]),
    "ods_graph_launch": (C.c_int, [C.c_void_p, C.c_void_p]),
    "ods_graph_destroy": (C.c_int, [C.c_void_p]),
    "ods_last_error": (C.c_char_p, []),
    "ods_tiled_weight_bytes": (C.c_size_t, [C.c_int32, C.c_int32, C.c_int32, C.c_int32]),
    "ods_tile_weight": (C.c_int, [C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                  C.c_void_p]),
}


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build the HIP library first "
                          "(python -m paper_2609_14237_amd.build)")
    lib = C.CDLL(LIB_PATH)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()


class OdsError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = lib.ods_last_error().decode()
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)}: {msg}")


def _check(status: int, where: str) -> int:
    if status != ODS_OK:
        raise OdsError(status, where)
    return status


# ---------------------------------------------------------------- C entry points

def ods_kv_alloc(pool_pages: int, ctx_lens_host, batch: int, seed: int, max_pages: int, page_table_host) -> int:
    """ctx_lens_host: int32 numpy [batch]; page_table_host: int32 numpy [batch, max_pages] (written)."""
    return lib.ods_kv_alloc(pool_pages, ctx_lens_host.ctypes.data_as(C.POINTER(C.c_int32)), batch, seed,
                            max_pages, page_table_host.ctypes.data_as(C.POINTER(C.c_int32)))


def ods_kv_pool_bytes(cfg: ods_layer_cfg, pool_pages: int) -> int:
    return lib.ods_kv_pool_bytes(C.byref(cfg), pool_pages)


def ods_live_bytes(blk: ods_block, batch: int, which: int) -> int:
    return lib.ods_live_bytes(C.byref(blk), batch, which)


def ods_workspace_bytes(blk: ods_block, batch: ods_batch) -> int:
    return lib.ods_workspace_bytes(C.byref(blk), C.byref(batch))


def ods_block_num_ops(blk: ods_block) -> int:
    return lib.ods_block_num_ops(C.byref(blk))


def ods_op_name(blk: ods_block, op: int):
    r = lib.ods_op_name(C.byref(blk), op)
    return None if r is None else r.decode()


def ods_run_partition(blk: ods_block, op_begin: int, op_end: int, batch: ods_batch, state: ods_state,
                      stream: int) -> int:
    return lib.ods_run_partition(C.byref(blk), op_begin, op_end, C.byref(batch), C.byref(state), stream)


def ods_run_partition_scratch(blk: ods_block, op_begin: int, op_end: int, batch: ods_batch, state: ods_state,
                              stream: int) -> int:
    return lib.ods_run_partition_scratch(C.byref(blk), op_begin, op_end, C.byref(batch), C.byref(state), stream)


def ods_attn_stage(blk: ods_block, layer: int, batch: ods_batch, state: ods_state, stream: int) -> int:
    return lib.ods_attn_stage(C.byref(blk), layer, C.byref(batch), C.byref(state), stream)


def ods_ffn_stage(blk: ods_block, layer: int, batch: ods_batch, state: ods_state, stream: int) -> int:
    return lib.ods_ffn_stage(C.byref(blk), layer, C.byref(batch), C.byref(state), stream)


def ods_last_error() -> str:
    return lib.ods_last_error().decode()


def ods_partition_graph(blk: ods_block, op_begin: int, op_end: int, batch: ods_batch, state: ods_state):
    """(status, exec handle or None)."""
    h = C.c_void_p()
    st = lib.ods_partition_graph(C.byref(blk), op_begin, op_end, C.byref(batch), C.byref(state), C.byref(h))
    return st, h.value


def ods_graph_launch(exec_handle: int, stream: int) -> int:
    return lib.ods_graph_launch(exec_handle, stream)


def ods_graph_destroy(exec_handle) -> int:
    return lib.ods_graph_destroy(exec_handle)


def ods_tiled_weight_bytes(out: int, in_: int, gated: int, groups: int) -> int:
    return lib.ods_tiled_weight_bytes(out, in_, gated, groups)


def ods_tile_weight(src: int, dst: int, out: int, in_: int, gated: int, groups: int, stream: int) -> int:
    return lib.ods_tile_weight(src, dst, out, in_, gated, groups, stream)
