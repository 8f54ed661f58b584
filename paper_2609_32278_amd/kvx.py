"""Thin ctypes binding of libkvx (include/kvx.h): argument marshalling only.

Every function keeps the C ABI's name.  Device buffers are torch CUDA tensors
(PyTorch provides device memory and streams only; every step of the
computation runs in libkvx's HIP kernels).  The library must have been built
(``__graft_entry__.build()`` or ``python paper_2609_32278_amd/build.py``);
loading raises ``KvxNotBuilt`` otherwise -- there is no fallback.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkvx.so")

KVX_OK, KVX_EINVAL, KVX_ENOMEM, KVX_ERANGE, KVX_EUNSUPPORTED, KVX_EHIP = range(6)
KVX_KV_BF16, KVX_KV_FP8_E4M3 = 0, 1
STATUS_NAMES = {0: "KVX_OK", 1: "KVX_EINVAL", 2: "KVX_ENOMEM", 3: "KVX_ERANGE",
                4: "KVX_EUNSUPPORTED", 5: "KVX_EHIP"}

KVX_EVICT_LRU, KVX_EVICT_RR = 0, 1
KVX_ROPE_HALF, KVX_ROPE_INTERLEAVED = 0, 1
NOALLOC_PLAN_BYTES, NOALLOC_PARTS_BYTES = 8 << 20, 56 << 20  # KVX_NOALLOC_* in include/kvx.h

# Every symbol include/kvx.h and include/kvx_cache.h declare.
EXPORTS = ["kv_pool_create", "kv_pool_destroy", "kv_pool_layout", "kv_pool_write_pages",
           "kv_pool_read_pages", "kv_pool_record_bytes", "kv_pool_spill", "kv_pool_reload", "store_kv", "store_kv_rope", "extend_attention", "extend_attention_noalloc", "extend_attention_plan",
           "kv_pool_set_split_keys", "kv_pool_set_scaled_q", "kvx_last_error",
           "kvx_cache_create", "kvx_cache_create_tiered", "kvx_cache_set_recency_tiers", "kvx_cache_destroy", "kvx_cache_begin_turn",
           "kvx_cache_begin_turn_tiered", "kvx_cache_end_turn", "kvx_cache_complete", "kvx_cache_agent",
           "kvx_cache_agent_host", "kvx_cache_join", "kvx_cache_group", "kvx_cache_stats",
           "kvx_radix_create", "kvx_radix_destroy", "kvx_radix_begin", "kvx_radix_end", "kvx_radix_complete",
           "kvx_radix_match", "kvx_radix_stats"]


class KvxNotBuilt(ImportError):
    pass


class KvxError(RuntimeError):
    def __init__(self, status: int, func: str, message: str):
        super().__init__(f"{func}: {STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class kvx_batch(ctypes.Structure):
    _fields_ = [("num_reqs", ctypes.c_int32), ("prefix_lens", ctypes.c_void_p),
                ("extend_lens", ctypes.c_void_p), ("page_indptr", ctypes.c_void_p),
                ("page_ids", ctypes.c_void_p)]


class kvx_pool_layout(ctypes.Structure):
    _fields_ = [("k_base", ctypes.c_void_p), ("v_base", ctypes.c_void_p), ("num_pages", ctypes.c_int64),
                ("page_size", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("kv_dtype", ctypes.c_int32), ("elem_bytes", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("k_stride_page", ctypes.c_int64), ("k_stride_head", ctypes.c_int64),
                ("k_stride_slot", ctypes.c_int64), ("k_stride_dim", ctypes.c_int64),
                ("v_stride_page", ctypes.c_int64), ("v_stride_head", ctypes.c_int64),
                ("v_stride_slot", ctypes.c_int64), ("v_stride_dim", ctypes.c_int64),
                ("k_scale", ctypes.c_void_p), ("v_scale", ctypes.c_void_p)]


class kvx_rope(ctypes.Structure):
    _fields_ = [("theta", ctypes.c_double), ("inv_freq", ctypes.c_void_p), ("rotary_dim", ctypes.c_int32),
                ("style", ctypes.c_int32), ("q_norm", ctypes.c_void_p), ("k_norm", ctypes.c_void_p),
                ("norm_eps", ctypes.c_float)]


class kvx_work_item(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("req", "kv_head", "tok_begin", "tok_count", "key_begin", "key_end", "part", "xcd")]


WORK_ITEM_DTYPE = np.dtype([(n, np.int32) for n, _ in kvx_work_item._fields_])


class kvx_radix_counters(ctypes.Structure):
    _fields_ = [("num_pages", ctypes.c_int64), ("free_pages", ctypes.c_int64), ("cached_pages", ctypes.c_int64),
                ("temp_pages", ctypes.c_int64), ("nodes", ctypes.c_int64), ("leaves", ctypes.c_int64),
                ("evicted_pages", ctypes.c_int64), ("evictions", ctypes.c_int64), ("active", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class kvx_cache_stats_t(ctypes.Structure):
    _fields_ = [("num_pages", ctypes.c_int64), ("free_pages", ctypes.c_int64), ("cached_pages", ctypes.c_int64),
                ("turn_pages", ctypes.c_int64), ("evicted_pages", ctypes.c_int64), ("evictions", ctypes.c_int64),
                ("agents", ctypes.c_int32), ("active_agents", ctypes.c_int32), ("host_pages", ctypes.c_int64),
                ("host_used", ctypes.c_int64), ("spilled_pages", ctypes.c_int64), ("reloaded_pages", ctypes.c_int64),
                ("host_dropped_pages", ctypes.c_int64), ("group_pages", ctypes.c_int64)]


class kvx_cache_moves(ctypes.Structure):
    _fields_ = [("spill_pages", ctypes.POINTER(ctypes.c_int32)), ("spill_slots", ctypes.POINTER(ctypes.c_int32)),
                ("reload_pages", ctypes.POINTER(ctypes.c_int32)), ("reload_slots", ctypes.POINTER(ctypes.c_int32)),
                ("n_spill", ctypes.c_int64), ("n_reload", ctypes.c_int64)]

_lib = None


def lib():
    """The loaded libkvx (raises KvxNotBuilt if the shared library is missing)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise KvxNotBuilt(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
        sig = {
            "kv_pool_create": [i64, i32, i32, i32, i32, P, P, ctypes.POINTER(P)],
            "kv_pool_destroy": [P],
            "kv_pool_layout": [P, ctypes.POINTER(kvx_pool_layout)],
            "kv_pool_write_pages": [P, P, i64, P, P, P],
            "kv_pool_read_pages": [P, P, i64, P, P, P],
            "kv_pool_record_bytes": [P, ctypes.POINTER(i64)],
            "kv_pool_spill": [P, P, P, i64, P, i64, P],
            "kv_pool_reload": [P, P, P, i64, P, i64, P],
            "store_kv": [P, ctypes.POINTER(kvx_batch), P, P, P],
            "store_kv_rope": [P, ctypes.POINTER(kvx_batch), ctypes.POINTER(kvx_rope), P, i32, P, P, P, P],
            "extend_attention": [P, ctypes.POINTER(kvx_batch), P, i32, f32, P, P, P],
            "extend_attention_noalloc": [P, ctypes.POINTER(kvx_batch), P, i32, f32, P, P, P],
            "extend_attention_plan": [ctypes.POINTER(kvx_batch), i32, i32, i32, i32, P, i64, ctypes.POINTER(i64)],
            "kv_pool_set_split_keys": [P, i32],
            "kv_pool_set_scaled_q": [P, i32],
            "kvx_cache_create": [i64, i32, i32, i32, ctypes.POINTER(P)],
            "kvx_cache_create_tiered": [i64, i64, i32, i32, i32, ctypes.POINTER(P)],
            "kvx_cache_set_recency_tiers": [P, i64],
            "kvx_cache_begin_turn_tiered": [P, i64, i32, ctypes.POINTER(i32), P, i64, ctypes.POINTER(kvx_cache_moves)],
            "kvx_cache_agent_host": [P, i64, ctypes.POINTER(i32), P, i64],
            "kvx_cache_join": [P, i64, i64, i32],
            "kvx_cache_group": [P, i64, ctypes.POINTER(i32), P, i64],
            "kvx_cache_destroy": [P],
            "kvx_cache_begin_turn": [P, i64, i32, ctypes.POINTER(i32), P, i64],
            "kvx_cache_end_turn": [P, i64],
            "kvx_cache_complete": [P, i64],
            "kvx_cache_agent": [P, i64, ctypes.POINTER(i32), P, i64],
            "kvx_cache_stats": [P, ctypes.POINTER(kvx_cache_stats_t)],
            "kvx_radix_create": [i64, i32, i32, i32, ctypes.POINTER(P)],
            "kvx_radix_destroy": [P],
            "kvx_radix_begin": [P, i64, P, i32, ctypes.POINTER(i32), P, i64],
            "kvx_radix_end": [P, i64],
            "kvx_radix_complete": [P, i64],
            "kvx_radix_match": [P, P, i32, ctypes.POINTER(i32), P, i64],
            "kvx_radix_stats": [P, ctypes.POINTER(kvx_radix_counters)],
        }
        for name, args in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = ctypes.c_int
        L.kvx_last_error.argtypes = []
        L.kvx_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def kvx_last_error() -> str:
    return lib().kvx_last_error().decode()


def _check(status: int, func: str):
    if status != KVX_OK:
        raise KvxError(status, func, kvx_last_error())


def _stream(stream):
    if stream is None:
        import torch
        if torch.cuda.is_available() and torch.cuda.is_initialized():
            return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        return None
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def _need(t, nbytes: int, name: str) -> None:
    """Reject a tensor smaller than the call reads or writes (raw int addresses are
    the caller's responsibility): the kernels index it by the sizes alone."""
    if t is None or isinstance(t, int):
        return
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{name}: {have} bytes, the call needs {nbytes}")


def _dptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError("expected a device (CUDA/HIP) tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return t.data_ptr()


# ----------------------------------------------------------------------- batch

class Batch:
    """Host lengths and page_indptr plus the device page table, as a kvx_batch."""

    def __init__(self, prefix_lens, extend_lens, page_indptr, page_ids_dev):
        self.prefix_lens = np.ascontiguousarray(prefix_lens, dtype=np.int32)
        self.extend_lens = np.ascontiguousarray(extend_lens, dtype=np.int32)
        self.page_indptr = np.ascontiguousarray(page_indptr, dtype=np.int32)
        self.page_ids = page_ids_dev  # device int32 tensor (or an int address)
        if len(self.page_indptr) != len(self.prefix_lens) + 1 or len(self.extend_lens) != len(self.prefix_lens):
            raise ValueError("prefix_lens and extend_lens need one entry per request, page_indptr one more")
        if len(self.page_indptr):
            _need(page_ids_dev, 4 * int(self.page_indptr[-1]), "page_ids")
        if page_ids_dev is not None and not isinstance(page_ids_dev, int) and page_ids_dev.element_size() != 4:
            raise ValueError(f"page_ids must hold 4-byte (int32) page ids, got {page_ids_dev.dtype}")
        self.c = kvx_batch(len(self.prefix_lens), self.prefix_lens.ctypes.data,
                           self.extend_lens.ctypes.data, self.page_indptr.ctypes.data,
                           _dptr(page_ids_dev) if page_ids_dev is not None else None)

    @property
    def total_extend(self) -> int:
        return int(self.extend_lens.astype(np.int64).sum())


# ------------------------------------------------------------------------ pool

def kv_pool_create(num_pages: int, page_size: int, num_kv_heads: int, head_dim: int,
                   kv_dtype: int = KVX_KV_BF16, k_scale=None, v_scale=None) -> ctypes.c_void_p:
    ks = None if k_scale is None else np.ascontiguousarray(k_scale, dtype=np.float32)
    vs = None if v_scale is None else np.ascontiguousarray(v_scale, dtype=np.float32)
    out = ctypes.c_void_p()
    _check(lib().kv_pool_create(int(num_pages), int(page_size), int(num_kv_heads), int(head_dim), int(kv_dtype),
                                None if ks is None else ks.ctypes.data, None if vs is None else vs.ctypes.data,
                                ctypes.byref(out)), "kv_pool_create")
    return out


def kv_pool_destroy(pool) -> None:
    _check(lib().kv_pool_destroy(pool), "kv_pool_destroy")


def kv_pool_layout(pool) -> dict:
    lay = kvx_pool_layout()
    _check(lib().kv_pool_layout(pool, ctypes.byref(lay)), "kv_pool_layout")
    return {name: getattr(lay, name) for name, _ in kvx_pool_layout._fields_}


def _geometry(pool) -> tuple:
    """(num_kv_heads, head_dim, elem_bytes) of a pool."""
    lay = kvx_pool_layout()
    _check(lib().kv_pool_layout(pool, ctypes.byref(lay)), "kv_pool_layout")
    return lay.num_kv_heads, lay.head_dim, lay.elem_bytes


def _page_buffers(pool, n, k, v) -> None:
    hkv, d, eb = _geometry(pool)
    _need(k, n * hkv * 16 * d * eb, "K buffer")
    _need(v, n * hkv * 16 * d * eb, "V buffer")


def kv_pool_write_pages(pool, page_ids, k_src, v_src, stream=None) -> None:
    ids = np.ascontiguousarray(page_ids, dtype=np.int32)
    _page_buffers(pool, ids.size, k_src, v_src)
    _check(lib().kv_pool_write_pages(pool, ids.ctypes.data, ids.size, _dptr(k_src), _dptr(v_src), _stream(stream)),
           "kv_pool_write_pages")


def kv_pool_read_pages(pool, page_ids, k_dst, v_dst, stream=None) -> None:
    ids = np.ascontiguousarray(page_ids, dtype=np.int32)
    _page_buffers(pool, ids.size, k_dst, v_dst)
    _check(lib().kv_pool_read_pages(pool, ids.ctypes.data, ids.size, _dptr(k_dst), _dptr(v_dst), _stream(stream)),
           "kv_pool_read_pages")


# ----------------------------------------------------------------- hot path

def kv_pool_record_bytes(pool) -> int:
    b = ctypes.c_int64()
    _check(lib().kv_pool_record_bytes(pool, ctypes.byref(b)), "kv_pool_record_bytes")
    return b.value


def _host_ptr(t) -> int:
    """Address of a pinned host tensor (or a raw int address)."""
    if isinstance(t, int):
        return t
    if t.is_cuda or not t.is_contiguous():
        raise ValueError("expected a contiguous host tensor")
    return t.data_ptr()


def _move(fn, pool, page_ids, slots, host, host_slots, stream):
    ids = np.ascontiguousarray(page_ids, dtype=np.int32)
    sl = np.ascontiguousarray(slots, dtype=np.int32)
    if ids.shape != sl.shape:
        raise ValueError("page_ids and slots differ in length")
    if not isinstance(host, int):
        _need(host, int(host_slots) * kv_pool_record_bytes(pool), "host")
    _check(getattr(lib(), fn)(pool, ids.ctypes.data, sl.ctypes.data, ids.size, _host_ptr(host), int(host_slots),
                              _stream(stream)), fn)


def kv_pool_spill(pool, page_ids, slots, host, host_slots: int, stream=None) -> None:
    _move("kv_pool_spill", pool, page_ids, slots, host, host_slots, stream)


def kv_pool_reload(pool, page_ids, slots, host, host_slots: int, stream=None) -> None:
    _move("kv_pool_reload", pool, page_ids, slots, host, host_slots, stream)


def _suffix_buffers(pool, batch: Batch, num_q_heads: int, **bufs) -> None:
    """Row buffers of a call: K_ext/V_ext [T, Hkv, d], Q/O [T, Hq, d] bf16, LSE [T, Hq] fp32."""
    hkv, d, _ = _geometry(pool)
    t = batch.total_extend
    rows = {"k_ext": t * hkv, "v_ext": t * hkv, "q": t * num_q_heads, "q_out": t * num_q_heads,
            "out": t * num_q_heads}
    for name, buf in bufs.items():
        if buf is not None and not isinstance(buf, int) and buf.element_size() != (4 if name == "lse" else 2):
            raise ValueError(f"{name}: {buf.dtype} elements; expected {'float32' if name == 'lse' else 'bf16'}")
        if name == "lse":
            _need(buf, 4 * t * num_q_heads, name)
        elif name in ("q_norm", "k_norm"):
            _need(buf, 2 * d, name)
        else:
            _need(buf, 2 * d * rows[name], name)


def store_kv(pool, batch: Batch, k_ext, v_ext, stream=None) -> None:
    _suffix_buffers(pool, batch, 0, k_ext=k_ext, v_ext=v_ext)
    _check(lib().store_kv(pool, ctypes.byref(batch.c), _dptr(k_ext), _dptr(v_ext), _stream(stream)), "store_kv")


def store_kv_rope(pool, batch: Batch, k_ext, v_ext, *, theta: float = 10000.0, rotary_dim: int, style: int = 0,
                  q=None, num_q_heads: int = 0, q_out=None, q_norm=None, k_norm=None, norm_eps: float = 1e-6,
                  inv_freq=None, stream=None) -> None:
    """store_kv with RMS norm (optional) and rotary embedding of Q and K fused in."""
    freqs = None if inv_freq is None else np.ascontiguousarray(inv_freq, dtype=np.float64)
    if freqs is not None and freqs.size < int(rotary_dim) // 2:
        raise ValueError(f"inv_freq: {freqs.size} entries, rotary_dim {rotary_dim} needs {int(rotary_dim) // 2}")
    _suffix_buffers(pool, batch, int(num_q_heads), k_ext=k_ext, v_ext=v_ext, q_norm=q_norm, k_norm=k_norm,
                    **({"q": q, "q_out": q_out} if num_q_heads else {}))
    r = kvx_rope(float(theta), None if freqs is None else freqs.ctypes.data, int(rotary_dim), int(style),
                 _dptr(q_norm), _dptr(k_norm), float(norm_eps))
    _check(lib().store_kv_rope(pool, ctypes.byref(batch.c), ctypes.byref(r), _dptr(q), int(num_q_heads),
                               _dptr(q_out), _dptr(k_ext), _dptr(v_ext), _stream(stream)), "store_kv_rope")


def extend_attention(pool, batch: Batch, q, num_q_heads: int, sm_scale: float, out, lse=None, stream=None) -> None:
    _suffix_buffers(pool, batch, int(num_q_heads), q=q, out=out, lse=lse)
    _check(lib().extend_attention(pool, ctypes.byref(batch.c), _dptr(q), int(num_q_heads), float(sm_scale),
                                  _dptr(out), _dptr(lse), _stream(stream)), "extend_attention")


def extend_attention_noalloc(pool, batch: Batch, q, num_q_heads: int, sm_scale: float, out, lse=None,
                             stream=None) -> None:
    """extend_attention without device allocation: plan and split parts go into the
    library's fixed per-GPU scratch (NOALLOC_PLAN_BYTES + NOALLOC_PARTS_BYTES)."""
    _suffix_buffers(pool, batch, int(num_q_heads), q=q, out=out, lse=lse)
    _check(lib().extend_attention_noalloc(pool, ctypes.byref(batch.c), _dptr(q), int(num_q_heads), float(sm_scale),
                                          _dptr(out), _dptr(lse), _stream(stream)), "extend_attention_noalloc")


def extend_attention_plan(batch: Batch, num_q_heads: int, num_kv_heads: int, head_dim: int,
                          split_keys: int = 0) -> np.ndarray:
    count = ctypes.c_int64()
    _check(lib().extend_attention_plan(ctypes.byref(batch.c), num_q_heads, num_kv_heads, head_dim, int(split_keys),
                                       None, 0, ctypes.byref(count)), "extend_attention_plan")
    items = np.zeros(count.value, dtype=WORK_ITEM_DTYPE)
    _check(lib().extend_attention_plan(ctypes.byref(batch.c), num_q_heads, num_kv_heads, head_dim, int(split_keys),
                                       items.ctypes.data, count.value, ctypes.byref(count)),
           "extend_attention_plan")
    return items


def kv_pool_set_split_keys(pool, keys: int) -> None:
    _check(lib().kv_pool_set_split_keys(pool, int(keys)), "kv_pool_set_split_keys")


def kv_pool_set_scaled_q(pool, enable: bool) -> None:
    _check(lib().kv_pool_set_scaled_q(pool, 1 if enable else 0), "kv_pool_set_scaled_q")


# ------------------------------------------------------------------ prefix cache (include/kvx_cache.h)

def kvx_cache_create(num_pages: int, page_size: int = 16, chunk_tokens: int = 1024, policy: int = KVX_EVICT_RR):
    out = ctypes.c_void_p()
    _check(lib().kvx_cache_create(int(num_pages), page_size, chunk_tokens, policy, ctypes.byref(out)),
           "kvx_cache_create")
    return out


def kvx_cache_create_tiered(num_pages: int, host_pages: int, page_size: int = 16, chunk_tokens: int = 1024,
                            policy: int = KVX_EVICT_RR):
    out = ctypes.c_void_p()
    _check(lib().kvx_cache_create_tiered(int(num_pages), int(host_pages), page_size, chunk_tokens, policy,
                                         ctypes.byref(out)), "kvx_cache_create_tiered")
    return out


def kvx_cache_set_recency_tiers(cache, tier_width: int) -> None:
    _check(lib().kvx_cache_set_recency_tiers(cache, int(tier_width)), "kvx_cache_set_recency_tiers")


def kvx_cache_destroy(cache) -> None:
    _check(lib().kvx_cache_destroy(cache), "kvx_cache_destroy")


def kvx_cache_begin_turn(cache, agent: int, prompt_len: int):
    """Returns (prefix_len, page_ids int32 array of ceil(prompt_len / 16) entries)."""
    ids = np.zeros(max(1, -(-int(prompt_len) // 16)), np.int32)
    prefix = ctypes.c_int32()
    _check(lib().kvx_cache_begin_turn(cache, int(agent), int(prompt_len), ctypes.byref(prefix), ids.ctypes.data,
                                      ids.size), "kvx_cache_begin_turn")
    return prefix.value, ids


def _moves(m: kvx_cache_moves) -> dict:
    def arr(ptr, n):
        out = np.empty(n, np.int32)
        if n:
            ctypes.memmove(out.ctypes.data, ptr, 4 * n)
        return out
    return {"spill_pages": arr(m.spill_pages, m.n_spill), "spill_slots": arr(m.spill_slots, m.n_spill),
            "reload_pages": arr(m.reload_pages, m.n_reload), "reload_slots": arr(m.reload_slots, m.n_reload)}


class KvxNoMemory(KvxError):
    """ENOMEM from a tiered turn start; ``moves`` holds the spills that must still run."""

    def __init__(self, err: KvxError, moves: dict):
        super().__init__(err.status, "kvx_cache_begin_turn_tiered", str(err))
        self.moves = moves


def kvx_cache_begin_turn_tiered(cache, agent: int, prompt_len: int):
    """Returns (prefix_len, page_ids, moves dict of int32 arrays spill_pages / spill_slots /
    reload_pages / reload_slots).  On ENOMEM raises KvxNoMemory carrying the spills."""
    ids = np.zeros(max(1, -(-int(prompt_len) // 16)), np.int32)
    prefix = ctypes.c_int32()
    m = kvx_cache_moves()
    st = lib().kvx_cache_begin_turn_tiered(cache, int(agent), int(prompt_len), ctypes.byref(prefix),
                                           ids.ctypes.data, ids.size, ctypes.byref(m))
    if st == KVX_ENOMEM:
        raise KvxNoMemory(KvxError(st, "kvx_cache_begin_turn_tiered", kvx_last_error()), _moves(m))
    _check(st, "kvx_cache_begin_turn_tiered")
    return prefix.value, ids, _moves(m)


def kvx_cache_end_turn(cache, agent: int) -> None:
    _check(lib().kvx_cache_end_turn(cache, int(agent)), "kvx_cache_end_turn")


def kvx_cache_complete(cache, agent: int) -> None:
    _check(lib().kvx_cache_complete(cache, int(agent)), "kvx_cache_complete")


def kvx_cache_agent(cache, agent: int):
    """Returns (cached_tokens, page_ids of the cached history)."""
    tok = ctypes.c_int32()
    _check(lib().kvx_cache_agent(cache, int(agent), ctypes.byref(tok), None, 0), "kvx_cache_agent")
    ids = np.zeros(tok.value // 16, np.int32)
    _check(lib().kvx_cache_agent(cache, int(agent), ctypes.byref(tok), ids.ctypes.data, ids.size), "kvx_cache_agent")
    return tok.value, ids


def kvx_cache_agent_host(cache, agent: int):
    """Returns (host_tokens, host records of the agent in logical order)."""
    tok = ctypes.c_int32()
    _check(lib().kvx_cache_agent_host(cache, int(agent), ctypes.byref(tok), None, 0), "kvx_cache_agent_host")
    ids = np.zeros(tok.value // 16, np.int32)
    _check(lib().kvx_cache_agent_host(cache, int(agent), ctypes.byref(tok), ids.ctypes.data, ids.size),
           "kvx_cache_agent_host")
    return tok.value, ids


def kvx_cache_join(cache, agent: int, group: int, shared_tokens: int) -> None:
    _check(lib().kvx_cache_join(cache, int(agent), int(group), int(shared_tokens)), "kvx_cache_join")


def kvx_cache_group(cache, group: int):
    """Returns (shared_tokens present, page ids of the group node)."""
    tok = ctypes.c_int32()
    _check(lib().kvx_cache_group(cache, int(group), ctypes.byref(tok), None, 0), "kvx_cache_group")
    ids = np.zeros(tok.value // 16, np.int32)
    _check(lib().kvx_cache_group(cache, int(group), ctypes.byref(tok), ids.ctypes.data, ids.size), "kvx_cache_group")
    return tok.value, ids


def kvx_cache_stats(cache) -> dict:
    st = kvx_cache_stats_t()
    _check(lib().kvx_cache_stats(cache, ctypes.byref(st)), "kvx_cache_stats")
    return {n: getattr(st, n) for n, _ in st._fields_}


# ------------------------------------------------------------------ token-content radix tree (include/kvx_radix.h)

def _tokens(tokens) -> np.ndarray:
    t = np.ascontiguousarray(np.asarray(tokens, dtype=np.int32))
    if t.ndim != 1:
        raise ValueError("tokens must be one-dimensional")
    return t


def kvx_radix_create(num_pages: int, page_size: int = 16, chunk_tokens: int = 1024, policy: int = KVX_EVICT_RR):
    out = ctypes.c_void_p()
    _check(lib().kvx_radix_create(int(num_pages), int(page_size), int(chunk_tokens), int(policy), ctypes.byref(out)),
           "kvx_radix_create")
    return out


def kvx_radix_destroy(tree) -> None:
    _check(lib().kvx_radix_destroy(tree), "kvx_radix_destroy")


def kvx_radix_begin(tree, agent: int, tokens, page_size: int = 16):
    """Start a request of `agent` over `tokens`; returns (prefix_len, page table)."""
    t = _tokens(tokens)
    n = len(t)
    table = np.zeros(max(1, (n + page_size - 1) // page_size), dtype=np.int32)
    prefix = ctypes.c_int32()
    _check(lib().kvx_radix_begin(tree, int(agent), t.ctypes.data, n, ctypes.byref(prefix), table.ctypes.data,
                                 len(table)), "kvx_radix_begin")
    return prefix.value, table


def kvx_radix_end(tree, agent: int) -> None:
    _check(lib().kvx_radix_end(tree, int(agent)), "kvx_radix_end")


def kvx_radix_complete(tree, agent: int) -> None:
    _check(lib().kvx_radix_complete(tree, int(agent)), "kvx_radix_complete")


def kvx_radix_match(tree, tokens, page_size: int = 16):
    """Longest cached whole-page prefix of `tokens`: (matched tokens, its pages)."""
    t = _tokens(tokens)
    m = ctypes.c_int32()
    pages = np.zeros(max(1, len(t) // page_size), dtype=np.int32)
    _check(lib().kvx_radix_match(tree, t.ctypes.data, len(t), ctypes.byref(m), pages.ctypes.data, len(pages)),
           "kvx_radix_match")
    return m.value, pages[: m.value // page_size].copy()


def kvx_radix_stats(tree) -> dict:
    st = kvx_radix_counters()
    _check(lib().kvx_radix_stats(tree, ctypes.byref(st)), "kvx_radix_stats")
    return {n: getattr(st, n) for n, _ in st._fields_ if n != "reserved"}
