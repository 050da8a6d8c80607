"""ctypes binding of libbsr.so: the C ABI of include/bsr.h, same names.

Argument marshalling only.  Device memory and streams are passed as integer
addresses / handles (for example ``tensor.data_ptr()`` and
``torch.cuda.Stream().cuda_stream``); every step of the restore path runs in
the library.  Importing this module fails loudly when the library has not
been built: there is no fallback implementation.
"""

from __future__ import annotations

import ctypes as ct
import os
from typing import List, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbsr.so")

BSR_ABI_VERSION = 4
BSR_MAX_GROUPS = 8
BSR_MAX_INSTALL_BATCH = 32
BSR_MAX_BOUND_REQUESTS = 16
BSR_STATIC_SCRATCH_BYTES = 2 << 20
BSR_NO_CHUNK = 0xFFFFFFFF

BSR_OK = 0
BSR_E_ARG, BSR_E_STATE, BSR_E_MISSING, BSR_E_CORRUPT, BSR_E_TIMEOUT = -1, -2, -3, -4, -5
BSR_E_TRANSFER, BSR_E_NOMEM, BSR_E_STAGING, BSR_E_BUSY, BSR_E_DEVICE, BSR_E_NOTFOUND = -6, -7, -8, -9, -10, -11

BSR_FAIL_NONE, BSR_FAIL_MISSING, BSR_FAIL_CORRUPT = 0, 1, 2
BSR_FAIL_TIMEOUT, BSR_FAIL_TRANSFER, BSR_FAIL_ABORT, BSR_FAIL_BLOCK_TABLE = 3, 4, 5, 6

BSR_KIND_CONTIG, BSR_KIND_PLANAR = 0, 1
BSR_FLAG_TIME_INSTALL, BSR_FLAG_TRUSTED_TABLES, BSR_FLAG_SDMA_COPIES, BSR_FLAG_TWO_STREAMS = 1, 2, 4, 8
BSR_FLAG_TIME_STAGE = 16
BSR_INJECT_NONE, BSR_INJECT_DELAY_MS, BSR_INJECT_TRANSFER_ERROR, BSR_INJECT_LAUNCH_ERROR = 0, 1, 2, 3
BSR_TIER_PINNED, BSR_TIER_FILE, BSR_TIER_NONE = 0, 1, 255
BSR_FILE_DIRECT = 1

_STRUCT_IDS = {"layout": 1, "config": 2, "group_dst": 3, "dev_status": 4, "stats": 5, "admission": 6}


class bsr_group_desc(ct.Structure):
    _fields_ = [("block_tokens", ct.c_uint32), ("n_tensors", ct.c_uint32),
                ("record_bytes", ct.c_uint32), ("kind", ct.c_uint32), ("split_bytes", ct.c_uint32)]


class bsr_layout(ct.Structure):
    _fields_ = [("chunk_tokens", ct.c_uint32), ("n_groups", ct.c_uint32),
                ("groups", bsr_group_desc * BSR_MAX_GROUPS)]


class bsr_config(ct.Structure):
    _fields_ = [("window_chunks", ct.c_uint32), ("install_batch", ct.c_uint32),
                ("hip_device", ct.c_int32), ("flags", ct.c_uint32),
                ("window_timeout_ms", ct.c_uint32), ("max_bound_requests", ct.c_uint32),
                ("staging_budget_bytes", ct.c_uint64)]


class bsr_group_dst(ct.Structure):
    _fields_ = [("block_table", ct.c_void_p), ("tensor_bases", ct.c_void_p), ("valid", ct.c_void_p),
                ("n_blocks", ct.c_uint32), ("pool_blocks", ct.c_uint32)]


class bsr_dev_status(ct.Structure):
    _fields_ = [("fail", ct.c_uint32), ("first_failed_chunk", ct.c_uint32),
                ("q", ct.c_uint32 * BSR_MAX_GROUPS), ("exposed_tokens", ct.c_uint64),
                ("fallback", ct.c_uint32), ("phase", ct.c_uint32), ("reserved", ct.c_uint32 * 2)]


class bsr_stats(ct.Structure):
    _fields_ = [("request_id", ct.c_uint64), ("n_hit_chunks", ct.c_uint32),
                ("window_chunks", ct.c_uint32), ("install_batch", ct.c_uint32),
                ("n_windows", ct.c_uint32), ("n_chunks_enqueued", ct.c_uint32),
                ("n_install_launches", ct.c_uint32), ("slot_bytes", ct.c_uint64),
                ("staging_required_bytes", ct.c_uint64), ("peak_live_staging_bytes", ct.c_uint64),
                ("aux_device_bytes", ct.c_uint64), ("h2d_bytes", ct.c_uint64),
                ("installed_bytes", ct.c_uint64), ("exposed_tokens", ct.c_uint64),
                ("fallback", ct.c_int32), ("fail_reason", ct.c_int32),
                ("first_failed_chunk", ct.c_uint32), ("q_mask", ct.c_uint32),
                ("probe_ns", ct.c_uint64), ("enqueue_ns", ct.c_uint64), ("commit_wait_ns", ct.c_uint64),
                ("install_ms_total", ct.c_double), ("install_ms_max", ct.c_double),
                ("host_bounce_bytes", ct.c_uint64), ("file_tier_chunks", ct.c_uint32),
                ("n_stage_launches", ct.c_uint32), ("stage_bytes", ct.c_uint64),
                ("stage_ms_total", ct.c_double)]


class bsr_admission(ct.Structure):
    _fields_ = [("staging_budget_bytes", ct.c_uint64), ("max_bound_requests", ct.c_uint32),
                ("n_bound", ct.c_uint32), ("bound_staging_bytes", ct.c_uint64),
                ("peak_bound_staging_bytes", ct.c_uint64), ("peak_n_bound", ct.c_uint32),
                ("n_refused", ct.c_uint32), ("aux_device_bytes", ct.c_uint64)]


class BsrError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"bsr error {code}: {msg}")
        self.code = code


def _load() -> ct.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2608_17826_amd.build`")
    lib = ct.CDLL(LIB_PATH)
    P, U32, U64, I32, VP = ct.POINTER, ct.c_uint32, ct.c_uint64, ct.c_int32, ct.c_void_p
    sig = {
        "bsr_abi_version": (I32, []),
        "bsr_set_timing": (ct.c_int, [VP, U32]),
        "bsr_struct_size": (U64, [I32]),
        "bsr_last_error": (ct.c_char_p, []),
        "bsr_slot_bytes": (U64, [P(bsr_layout)]),
        "bsr_staging_bytes": (U64, [P(bsr_layout), U32]),
        "bsr_plan_staging_bytes": (U64, [VP, U32]),
        "bsr_chunk_keys": (ct.c_int, [U64, VP, U64, U32, VP]),
        "bsr_ctx_create": (ct.c_int, [P(bsr_layout), P(bsr_config), P(VP)]),
        "bsr_ctx_create_static": (ct.c_int, [P(bsr_layout), P(bsr_config), P(VP)]),
        "bsr_ctx_destroy": (ct.c_int, [VP]),
        "bsr_store_reserve": (ct.c_int, [VP, U64]),
        "bsr_store_adopt": (ct.c_int, [VP, VP, U64]),
        "bsr_store_put_chunk": (ct.c_int, [VP, U64, P(VP)]),
        "bsr_store_put_chunks": (ct.c_int, [VP, U32, VP, P(VP)]),
        "bsr_store_remove": (ct.c_int, [VP, U64, I32]),
        "bsr_store_payload": (ct.c_int, [VP, U64, U32, P(VP), P(U64), P(U64)]),
        "bsr_store_count": (ct.c_int, [VP, P(U64), P(U64)]),
        "bsr_probe": (ct.c_int, [VP, U64, U64, VP, U64, P(U32), VP, VP]),
        "bsr_request_bind": (ct.c_int, [VP, U64, U32, P(bsr_group_dst), VP, U64, VP, VP, VP]),
        "bsr_restore_window": (ct.c_int, [VP, U64, U32, U32]),
        "bsr_next_window": (ct.c_int, [VP, U64, P(U32), P(U32)]),
        "bsr_mark_group_invalid": (ct.c_int, [VP, U64, U32]),
        "bsr_commit": (ct.c_int, [VP, U64, P(U64), P(I32)]),
        "bsr_invalidate": (ct.c_int, [VP, U64, I32]),
        "bsr_request_running": (ct.c_int, [VP, U64]),
        "bsr_request_end": (ct.c_int, [VP, U64]),
        "bsr_stats_get": (ct.c_int, [VP, P(bsr_stats)]),
        "bsr_request_stats": (ct.c_int, [VP, U64, P(bsr_stats)]),
        "bsr_admission_get": (ct.c_int, [VP, P(bsr_admission)]),
        "bsr_debug_inject": (ct.c_int, [VP, I32, U32, U32]),
        "bsr_measure_h2d": (ct.c_int, [VP, U64, U32, U32, P(ct.c_double)]),
        "bsr_measure_stage": (ct.c_int, [VP, U64, U32, P(ct.c_double)]),
        "bsr_measure_scatter": (ct.c_int, [VP, U32, U64, U32, U64, U32, P(ct.c_double)]),
        "bsr_file_tier_open": (ct.c_int, [VP, ct.c_char_p, U32, U32, U32]),
        "bsr_file_tier_put_chunk": (ct.c_int, [VP, U64, P(VP)]),
        "bsr_file_tier_remove": (ct.c_int, [VP, U64, I32]),
        "bsr_file_tier_count": (ct.c_int, [VP, P(U64)]),
        "bsr_tier_set_available": (ct.c_int, [VP, I32, I32]),
        "bsr_plan_tiers": (ct.c_int, [VP, U64, VP, U32]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype, f.argtypes = res, args
    if lib.bsr_abi_version() != BSR_ABI_VERSION:
        raise ImportError(f"libbsr.so ABI {lib.bsr_abi_version()} != binding ABI {BSR_ABI_VERSION}; rebuild")
    for name, cls in (("layout", bsr_layout), ("config", bsr_config), ("group_dst", bsr_group_dst),
                      ("dev_status", bsr_dev_status), ("stats", bsr_stats), ("admission", bsr_admission)):
        n = lib.bsr_struct_size(_STRUCT_IDS[name])
        if n != ct.sizeof(cls):
            raise ImportError(f"struct {name}: library size {n} != binding size {ct.sizeof(cls)}")
    return lib


_lib = _load()
EXPORTED = [n for n in dir(_lib) if n.startswith("bsr_")]


def _check(rc: int) -> None:
    if rc != BSR_OK:
        raise BsrError(rc, bsr_last_error())


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


# ---- library / layout -------------------------------------------------------
def bsr_abi_version() -> int:
    return _lib.bsr_abi_version()


def bsr_set_timing(ctx: "Ctx", flags: int) -> None:
    _check(_lib.bsr_set_timing(ctx, flags))


def bsr_last_error() -> str:
    return _lib.bsr_last_error().decode()


def make_layout(chunk_tokens: int, groups: Sequence[Tuple[int, int, int, int, int]]) -> bsr_layout:
    """groups: (block_tokens, n_tensors, record_bytes, kind, split_bytes) per group."""
    L = bsr_layout()
    L.chunk_tokens = chunk_tokens
    L.n_groups = len(groups)
    for g, (bt, nt, rb, kind, split) in enumerate(groups):
        L.groups[g] = bsr_group_desc(bt, nt, rb, kind, split)
    return L


def bsr_slot_bytes(layout: bsr_layout) -> int:
    n = _lib.bsr_slot_bytes(ct.byref(layout))
    if n == 0:
        raise BsrError(BSR_E_ARG, bsr_last_error())
    return n


def bsr_staging_bytes(layout: bsr_layout, window_chunks: int) -> int:
    n = _lib.bsr_staging_bytes(ct.byref(layout), window_chunks)
    if n == 0:
        raise BsrError(BSR_E_ARG, bsr_last_error())
    return n


def bsr_plan_staging_bytes(ctx: "Ctx", n_hit_chunks: int) -> int:
    n = _lib.bsr_plan_staging_bytes(ctx, n_hit_chunks)
    if n == 0:
        raise BsrError(BSR_E_ARG, bsr_last_error())
    return n


def bsr_chunk_keys(salt: int, tokens: np.ndarray, chunk_tokens: int) -> np.ndarray:
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    keys = np.zeros(max(1, len(tokens) // chunk_tokens), dtype=np.uint64)
    _check(_lib.bsr_chunk_keys(salt, _ptr(tokens), len(tokens), chunk_tokens, _ptr(keys)))
    return keys[:len(tokens) // chunk_tokens]


# ---- context ------------------------------------------------------------------
class Ctx:
    """A bsr_ctx* with the layout, window and admission budget it was created with."""

    def __init__(self, handle: int, layout: bsr_layout, window_chunks: int, staging_budget_bytes: int = 0):
        self.handle, self.layout, self.window_chunks = handle, layout, window_chunks
        self.staging_budget_bytes = staging_budget_bytes

    @property
    def _as_parameter_(self):  # lets ctypes pass a Ctx where bsr_ctx* is expected
        return ct.c_void_p(self.handle)


def bsr_ctx_create(layout: bsr_layout, window_chunks: int, hip_device: int = 0,
                   install_batch: int = 0, flags: int = 0, window_timeout_ms: int = 0,
                   staging_budget_bytes: int = 0, max_bound_requests: int = 0) -> Ctx:
    cfg = bsr_config(window_chunks, install_batch, hip_device, flags, window_timeout_ms,
                     max_bound_requests, staging_budget_bytes)
    out = ct.c_void_p()
    _check(_lib.bsr_ctx_create(ct.byref(layout), ct.byref(cfg), ct.byref(out)))
    return Ctx(out.value, layout, window_chunks, staging_budget_bytes)


def bsr_ctx_create_static(layout: bsr_layout, window_chunks: int, hip_device: int = 0,
                          install_batch: int = 0, flags: int = 0, window_timeout_ms: int = 0) -> Ctx:
    """A context whose device scratch is the library's static per-GPU array
    (no device or pinned allocation); one session slot."""
    cfg = bsr_config(window_chunks, install_batch, hip_device, flags, window_timeout_ms, 0, 0)
    out = ct.c_void_p()
    _check(_lib.bsr_ctx_create_static(ct.byref(layout), ct.byref(cfg), ct.byref(out)))
    return Ctx(out.value, layout, window_chunks, 0)


def bsr_ctx_destroy(ctx: Ctx) -> None:
    if ctx.handle:
        _check(_lib.bsr_ctx_destroy(ctx))
        ctx.handle = 0


# ---- store --------------------------------------------------------------------
def bsr_store_reserve(ctx: Ctx, nbytes: int) -> None:
    _check(_lib.bsr_store_reserve(ctx, nbytes))


def bsr_store_adopt(ctx: Ctx, arena_addr: int, nbytes: int) -> None:
    _check(_lib.bsr_store_adopt(ctx, arena_addr, nbytes))


def bsr_store_put_chunk(ctx: Ctx, key: int, payloads: Sequence[np.ndarray]) -> None:
    arrs = [np.ascontiguousarray(p, dtype=np.uint8) for p in payloads]
    ptrs = (ct.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs])
    _check(_lib.bsr_store_put_chunk(ctx, int(key), ptrs))


def bsr_store_put_chunks(ctx: Ctx, keys: Sequence[int], payloads: Sequence[Sequence[np.ndarray]]) -> None:
    """payloads[i][g]: chunk i's payload of group g."""
    n = len(keys)
    karr = np.ascontiguousarray(np.asarray([int(k) for k in keys], dtype=np.uint64))
    arrs = [np.ascontiguousarray(p, dtype=np.uint8) for per in payloads for p in per]
    ptrs = (ct.c_void_p * max(1, len(arrs)))(*[a.ctypes.data for a in arrs])
    _check(_lib.bsr_store_put_chunks(ctx, n, _ptr(karr), ptrs))


def bsr_store_remove(ctx: Ctx, key: int, group: int = -1) -> None:
    _check(_lib.bsr_store_remove(ctx, int(key), group))


def bsr_store_payload(ctx: Ctx, key: int, group: int) -> Tuple[int, int, int]:
    p, n, t = ct.c_void_p(), ct.c_uint64(), ct.c_uint64()
    _check(_lib.bsr_store_payload(ctx, int(key), group, ct.byref(p), ct.byref(n), ct.byref(t)))
    return p.value, n.value, t.value


def bsr_store_count(ctx: int) -> Tuple[int, int]:
    a, b = ct.c_uint64(), ct.c_uint64()
    _check(_lib.bsr_store_count(ctx, ct.byref(a), ct.byref(b)))
    return a.value, b.value


# ---- hot path -------------------------------------------------------------------
def bsr_probe(ctx: Ctx, request_id: int, salt: int, tokens: np.ndarray):
    """-> (n_hit_chunks, hit bitmap as uint8 0/1 per chunk, keys uint64)"""
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    n_chunks = len(tokens) // ctx.layout.chunk_tokens
    bits = np.zeros(max(1, (n_chunks + 7) // 8), dtype=np.uint8)
    keys = np.zeros(max(1, n_chunks), dtype=np.uint64)
    n = ct.c_uint32()
    _check(_lib.bsr_probe(ctx, request_id, salt, _ptr(tokens), len(tokens), ct.byref(n),
                          _ptr(bits), _ptr(keys)))
    bitmap = np.unpackbits(bits, bitorder="little")[:n_chunks]
    return n.value, bitmap, keys[:n_chunks]


def group_dst(block_table_ptr: int, tensor_bases_ptr: int, valid_ptr: int, n_blocks: int,
              pool_blocks: int) -> bsr_group_dst:
    return bsr_group_dst(block_table_ptr, tensor_bases_ptr, valid_ptr, n_blocks, pool_blocks)


def bsr_request_bind(ctx: Ctx, request_id: int, n_hit_chunks: int, dsts: Sequence[bsr_group_dst],
                     staging_ptr: int, staging_bytes: int, status_ptr: int, copy_stream: int,
                     compute_stream: int) -> None:
    arr = (bsr_group_dst * len(dsts))(*dsts)
    _check(_lib.bsr_request_bind(ctx, request_id, n_hit_chunks, arr, staging_ptr, staging_bytes,
                                 status_ptr, copy_stream, compute_stream))


def bsr_restore_window(ctx: Ctx, request_id: int, first_chunk: int, n_chunks: int) -> None:
    _check(_lib.bsr_restore_window(ctx, request_id, first_chunk, n_chunks))


def bsr_next_window(ctx: Ctx, request_id: int) -> Tuple[int, int]:
    """(first_chunk, n_chunks) of the plan's next window; n_chunks = 0 when done."""
    f, n = ct.c_uint32(), ct.c_uint32()
    _check(_lib.bsr_next_window(ctx, request_id, ct.byref(f), ct.byref(n)))
    return f.value, n.value


def bsr_mark_group_invalid(ctx: Ctx, request_id: int, group: int) -> None:
    _check(_lib.bsr_mark_group_invalid(ctx, request_id, group))


def bsr_commit(ctx: Ctx, request_id: int) -> Tuple[int, int]:
    e, f = ct.c_uint64(), ct.c_int32()
    _check(_lib.bsr_commit(ctx, request_id, ct.byref(e), ct.byref(f)))
    return e.value, f.value


def bsr_invalidate(ctx: Ctx, request_id: int, reason: int = BSR_FAIL_ABORT) -> None:
    _check(_lib.bsr_invalidate(ctx, request_id, reason))


def bsr_request_running(ctx: Ctx, request_id: int) -> None:
    _check(_lib.bsr_request_running(ctx, request_id))


def bsr_request_end(ctx: Ctx, request_id: int) -> None:
    _check(_lib.bsr_request_end(ctx, request_id))


def bsr_stats_get(ctx: int) -> dict:
    s = bsr_stats()
    _check(_lib.bsr_stats_get(ctx, ct.byref(s)))
    return {name: getattr(s, name) for name, _ in bsr_stats._fields_}


def bsr_request_stats(ctx: Ctx, request_id: int) -> dict:
    s = bsr_stats()
    _check(_lib.bsr_request_stats(ctx, request_id, ct.byref(s)))
    return {name: getattr(s, name) for name, _ in bsr_stats._fields_}


def bsr_admission_get(ctx: Ctx) -> dict:
    a = bsr_admission()
    _check(_lib.bsr_admission_get(ctx, ct.byref(a)))
    return {name: getattr(a, name) for name, _ in bsr_admission._fields_}


def bsr_debug_inject(ctx: Ctx, kind: int, chunk: int = 0, param: int = 0) -> None:
    _check(_lib.bsr_debug_inject(ctx, kind, chunk, param))


def bsr_measure_h2d(ctx: Ctx, nbytes: int, n_streams: int = 1, reps: int = 10) -> float:
    g = ct.c_double()
    _check(_lib.bsr_measure_h2d(ctx, nbytes, n_streams, reps, ct.byref(g)))
    return g.value


BSR_SCATTER_WARM_SOURCE = 1


def bsr_measure_scatter(ctx: Ctx, block_bytes: int, data_bytes: int, reps: int = 5, seed: int = 1,
                        flags: int = 0) -> float:
    g = ct.c_double()
    _check(_lib.bsr_measure_scatter(ctx, block_bytes, data_bytes, reps, seed, flags, ct.byref(g)))
    return g.value


def bsr_measure_stage(ctx: Ctx, nbytes: int, reps: int = 10) -> float:
    g = ct.c_double()
    _check(_lib.bsr_measure_stage(ctx, nbytes, reps, ct.byref(g)))
    return g.value


# ---- file-backed lower tier ------------------------------------------------------
def bsr_file_tier_open(ctx: Ctx, directory: str, load_concurrency: int = 1, readahead_chunks: int = 0,
                       flags: int = 0) -> None:
    _check(_lib.bsr_file_tier_open(ctx, directory.encode(), load_concurrency, readahead_chunks, flags))


def bsr_file_tier_put_chunk(ctx: Ctx, key: int, payloads: Sequence[np.ndarray]) -> None:
    arrs = [np.ascontiguousarray(p, dtype=np.uint8) for p in payloads]
    ptrs = (ct.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs])
    _check(_lib.bsr_file_tier_put_chunk(ctx, int(key), ptrs))


def bsr_file_tier_remove(ctx: Ctx, key: int, group: int = -1) -> None:
    _check(_lib.bsr_file_tier_remove(ctx, int(key), group))


def bsr_file_tier_count(ctx: Ctx) -> int:
    n = ct.c_uint64()
    _check(_lib.bsr_file_tier_count(ctx, ct.byref(n)))
    return n.value


def bsr_tier_set_available(ctx: Ctx, tier: int, available: bool) -> None:
    _check(_lib.bsr_tier_set_available(ctx, tier, int(bool(available))))


def bsr_plan_tiers(ctx: Ctx, request_id: int, n_chunks: int) -> np.ndarray:
    out = np.zeros(max(1, n_chunks), dtype=np.uint8)
    _check(_lib.bsr_plan_tiers(ctx, request_id, _ptr(out), n_chunks))
    return out[:n_chunks]
