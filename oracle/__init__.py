"""CPU oracle of prefix-extend attention -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It wraps ``oracle.c`` (plain fp64 C with
OpenMP, built by gcc into its own shared library) with ctypes and numpy; it
shares no code with the HIP library and never imports it.

Every function follows the definition of attention over the logical token
sequence of a request (the cached prefix then the uncached suffix, Section 1
and Section 2 of the paper); see ``oracle.c`` for the readings it takes where
the paper is silent.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

KV_BF16 = 0
KV_FP8_E4M3 = 1

MUTANTS = {
    "none": 0,
    "exclusive_diagonal": 1,
    "top_left_causal": 2,
    "kv_head_modulo": 3,
    "drop_partial_page": 4,
    "ignore_prefix": 5,
    "reversed_pages": 6,
    "scale_one_over_d": 7,
}


def build(force: bool = True) -> str:
    """Compile oracle.c with gcc (fp64, OpenMP, no fast-math, no FMA contraction)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + f".tmp{os.getpid()}"
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
               "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32, i64, dbl = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        lib.oracle_store_kv.restype = ctypes.c_int
        lib.oracle_store_kv.argtypes = [i32, P, P, P, P, P, i32, i64, i32, i32, i32, P, P, P, P, P, P]
        lib.oracle_extend_attention.restype = ctypes.c_int
        lib.oracle_extend_attention.argtypes = [i32, P, P, P, P, i32, i64, i32, i32, i32, i32, P, P,
                                                P, P, i64, P, P, P, dbl, P, P, i32, i32]
        lib.oracle_store_kv_f64.restype = ctypes.c_int
        lib.oracle_store_kv_f64.argtypes = [i32, P, P, P, P, P, i32, i64, i32, i32, i32, P, P, P, P, P, P]
        lib.oracle_bf16_round_array.restype = None
        lib.oracle_bf16_round_array.argtypes = [P, i64, P]
        lib.oracle_e4m3_encode_array.restype = None
        lib.oracle_e4m3_encode_array.argtypes = [P, i64, P]
        lib.oracle_e4m3_decode_array.restype = None
        lib.oracle_e4m3_decode_array.argtypes = [P, i64, P]
        lib.oracle_max_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(np.asarray(a), dtype=dtype)


def bf16_bits(t) -> np.ndarray:
    """uint16 bit patterns of a torch bf16 tensor (or pass a uint16 array through)."""
    if isinstance(t, np.ndarray):
        return _c(t, np.uint16)
    import torch
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def max_threads() -> int:
    return int(_load().oracle_max_threads())


# --------------------------------------------------------------------------- codec

def e4m3_encode(x: np.ndarray) -> np.ndarray:
    """OCP E4M3 codes of fp32 values: round to nearest, ties to even, saturating at +-448."""
    x = _c(x, np.float32)
    out = np.empty(x.shape, dtype=np.uint8)
    _load().oracle_e4m3_encode_array(_ptr(x), x.size, _ptr(out))
    return out


def bf16_round(x: np.ndarray) -> np.ndarray:
    """bf16 bit patterns nearest to float64 values (ties to even), rounded once."""
    x = _c(x, np.float64)
    out = np.empty(x.shape, dtype=np.uint16)
    _load().oracle_bf16_round_array(_ptr(x), x.size, _ptr(out))
    return out


def bf16_value(bits) -> np.ndarray:
    """float64 values of bf16 bit patterns (uint16 array or torch bf16)."""
    b = bf16_bits(bits)
    with np.errstate(invalid="ignore"):  # signalling-NaN patterns stay NaN
        return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def e4m3_decode(codes: np.ndarray) -> np.ndarray:
    codes = _c(codes, np.uint8)
    out = np.empty(codes.shape, dtype=np.float64)
    _load().oracle_e4m3_decode_array(_ptr(codes), codes.size, _ptr(out))
    return out


# --------------------------------------------------------------------------- pool

class OraclePool:
    """A host KV pool in the oracle's own layout [page][kv_head][slot][head_dim]."""

    def __init__(self, num_pages, num_kv_heads, head_dim, kv_dtype=KV_BF16, page_size=16,
                 k_scale=None, v_scale=None, fill=None):
        self.num_pages = int(num_pages)
        self.num_kv_heads = int(num_kv_heads)
        self.head_dim = int(head_dim)
        self.page_size = int(page_size)
        self.kv_dtype = int(kv_dtype)
        dt = np.uint16 if kv_dtype == KV_BF16 else np.uint8
        shape = (self.num_pages, self.num_kv_heads, self.page_size, self.head_dim)
        self.k = np.zeros(shape, dtype=dt)
        self.v = np.zeros(shape, dtype=dt)
        if fill is not None:
            self.k[...] = fill
            self.v[...] = fill
        self.k_scale = None if k_scale is None else _c(k_scale, np.float32)
        self.v_scale = None if v_scale is None else _c(v_scale, np.float32)
        if kv_dtype == KV_FP8_E4M3 and (self.k_scale is None or self.v_scale is None):
            raise ValueError("an fp8 pool needs k_scale and v_scale")


def _indptr64(a):
    return _c(a, np.int64)


def store_kv(pool: OraclePool, prefix_lens, extend_lens, page_indptr, page_ids, k_ext, v_ext):
    """Write the suffix rows k_ext/v_ext ([T, Hkv, d], bf16 bits or torch bf16) into the pool."""
    p = _c(prefix_lens, np.int32)
    e = _c(extend_lens, np.int32)
    qo = np.zeros(len(e) + 1, dtype=np.int64)
    np.cumsum(e, out=qo[1:])
    kb = bf16_bits(k_ext).reshape(-1)
    vb = bf16_bits(v_ext).reshape(-1)
    if kb.size != int(qo[-1]) * pool.num_kv_heads * pool.head_dim or vb.size != kb.size:
        raise ValueError("k_ext / v_ext size does not match sum(extend_lens) * Hkv * d")
    pi = _indptr64(page_indptr)
    ids = _c(page_ids, np.int32)
    rc = _load().oracle_store_kv(len(p), _ptr(p), _ptr(e), _ptr(qo), _ptr(pi), _ptr(ids),
                                 pool.page_size, pool.num_pages, pool.num_kv_heads, pool.head_dim,
                                 pool.kv_dtype, _ptr(pool.k_scale), _ptr(pool.v_scale),
                                 _ptr(kb), _ptr(vb), _ptr(pool.k), _ptr(pool.v))
    if rc != 0:
        raise ValueError(f"oracle_store_kv failed ({rc}): page id outside the pool")


def store_kv_values(pool: OraclePool, prefix_lens, extend_lens, page_indptr, page_ids, k_vals, v_ext):
    """store_kv with K given as exact float64 values [T, Hkv, d]: a bf16 pool holds
    their nearest bf16, an fp8 pool encode(float32(x) * float32(1/scale))."""
    p = _c(prefix_lens, np.int32)
    e = _c(extend_lens, np.int32)
    qo = np.zeros(len(e) + 1, dtype=np.int64)
    np.cumsum(e, out=qo[1:])
    kd = _c(k_vals, np.float64).reshape(-1)
    vb = bf16_bits(v_ext).reshape(-1)
    if kd.size != int(qo[-1]) * pool.num_kv_heads * pool.head_dim or vb.size != kd.size:
        raise ValueError("k_vals / v_ext size does not match sum(extend_lens) * Hkv * d")
    pi = _indptr64(page_indptr)
    ids = _c(page_ids, np.int32)
    rc = _load().oracle_store_kv_f64(len(p), _ptr(p), _ptr(e), _ptr(qo), _ptr(pi), _ptr(ids),
                                     pool.page_size, pool.num_pages, pool.num_kv_heads, pool.head_dim,
                                     pool.kv_dtype, _ptr(pool.k_scale), _ptr(pool.v_scale),
                                     _ptr(kd), _ptr(vb), _ptr(pool.k), _ptr(pool.v))
    if rc != 0:
        raise ValueError(f"oracle_store_kv_f64 failed ({rc}): page id outside the pool")


LOG2E_F32 = np.float32(1.4426950408889634)


def scaled_queries(q_rows, sm_scale) -> np.ndarray:
    """bf16 bits of the queries of the scaled-Q mode: each query times
    c = float32(float32(sm_scale) * float32(log2 e)) as a float32 product, rounded
    to bf16 (nearest, ties to even).  Attention of these queries with softmax scale
    ln 2 is the mode's result: exp2(bf16(q c) . k) = exp(ln 2 * bf16(q c) . k)."""
    c = np.float32(np.float32(sm_scale) * LOG2E_F32)
    q = bf16_value(q_rows).astype(np.float32)
    y = (q * c).astype(np.float32)  # one float32 product per element
    return bf16_round(y.astype(np.float64))


def extend_attention(pool: OraclePool, prefix_lens, extend_lens, page_indptr, page_ids, q_rows,
                     row_req, row_pos, num_q_heads, sm_scale, mutant="none", num_threads=0,
                     want_lse=False, scaled_q=False):
    """Attention outputs (float64 [n, Hq, d]) of the listed suffix rows.

    q_rows: bf16 [n, Hq, d] (torch bf16 or uint16 bits) -- the queries of those rows.
    row_req / row_pos: request index and suffix position of each row.
    scaled_q: the scaled-Q mode's definition instead (the queries of
    ``scaled_queries`` with softmax scale ln 2); the LSE is then in natural units of
    those scores.
    """
    if scaled_q:
        q_rows = scaled_queries(q_rows, sm_scale)
        sm_scale = float(np.log(2.0))
    p = _c(prefix_lens, np.int32)
    e = _c(extend_lens, np.int32)
    pi = _indptr64(page_indptr)
    ids = _c(page_ids, np.int32)
    rr = _c(row_req, np.int32)
    rp = _c(row_pos, np.int32)
    n = rr.size
    qb = bf16_bits(q_rows).reshape(-1)
    if qb.size != n * num_q_heads * pool.head_dim:
        raise ValueError("q_rows size does not match the row list")
    out = np.zeros((n, num_q_heads, pool.head_dim), dtype=np.float64)
    lse = np.zeros((n, num_q_heads), dtype=np.float64) if want_lse else None
    mut = MUTANTS[mutant] if isinstance(mutant, str) else int(mutant)
    rc = _load().oracle_extend_attention(
        len(p), _ptr(p), _ptr(e), _ptr(pi), _ptr(ids), pool.page_size, pool.num_pages,
        int(num_q_heads), pool.num_kv_heads, pool.head_dim, pool.kv_dtype, _ptr(pool.k), _ptr(pool.v),
        _ptr(pool.k_scale), _ptr(pool.v_scale), n, _ptr(rr), _ptr(rp), _ptr(qb), float(sm_scale),
        _ptr(out), _ptr(lse), mut, int(num_threads))
    if rc != 0:
        raise ValueError(f"oracle_extend_attention failed ({rc})")
    return (out, lse) if want_lse else out


def all_rows(extend_lens):
    """(row_req, row_pos) listing every suffix row in qo order."""
    e = np.asarray(extend_lens, dtype=np.int64)
    rr = np.repeat(np.arange(len(e), dtype=np.int32), e)
    rp = np.concatenate([np.arange(x, dtype=np.int32) for x in e]) if len(e) else np.zeros(0, np.int32)
    return rr, rp.astype(np.int32)
