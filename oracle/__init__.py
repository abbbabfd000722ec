"""CPU oracle for the layerwise prefix-KV path -- TEST INFRASTRUCTURE.

Only the tests, the smoke check and the benchmark's CPU-baseline leg import
this package.  The product library never does, and this package imports
nothing from the product.

The arithmetic lives in ``oracle.c`` (plain C, float64 attention, byte-level
scatter/gather); this module only loads it and marshals numpy arrays.  See
``oracle.c`` for what each function follows in the paper.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c with gcc into liboracle.so next to it."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC",
                               "-pthread", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        P, I64, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        lib.oco_assemble_layer.argtypes = [P, I64, I64, I32, P]
        lib.oco_assemble_layer.restype = None
        lib.oco_logical_kv.argtypes = [P, I64, I32, I32, I32, I32, P, P]
        lib.oco_logical_kv.restype = None
        lib.oco_ingest_layer.argtypes = [P, I64, I32, I32, I32, I32, P, I64, P, I64, I32]
        lib.oco_ingest_layer.restype = ctypes.c_int
        lib.oco_ingest_layer_mt.argtypes = [P, I64, I32, I32, I32, I32, P, I64, P, I64, I32, I32]
        lib.oco_ingest_layer_mt.restype = ctypes.c_int
        lib.oco_gather_layer.argtypes = [P, I64, I32, P, I64, I64, I32, I32, I32, I32, P]
        lib.oco_gather_layer.restype = ctypes.c_int
        lib.oco_append_suffix.argtypes = [P, P, I64, I32, I32, I32, P, I64, I64, P, I64, I32]
        lib.oco_append_suffix.restype = ctypes.c_int
        lib.oco_gather_chunks.argtypes = [P, I64, I32, P, I64, I64, I64, I32, I32, I32, I32, P]
        lib.oco_gather_chunks.restype = ctypes.c_int
        lib.oco_attention.argtypes = [P, P, P, P, P, I64, I64, I32, I32, I32, P, I64, P, I32]
        lib.oco_attention.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def _u16(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        raise TypeError("bfloat16 arrays travel as uint16 bit patterns")
    return a


def _chunk_ptrs(chunks: Sequence[np.ndarray]):
    arr = (ctypes.c_void_p * len(chunks))()
    for j, c in enumerate(chunks):
        if not c.flags["C_CONTIGUOUS"]:
            raise ValueError("chunk objects must be contiguous")
        arr[j] = c.ctypes.data
    return arr


def assemble_layer(chunks: Sequence[np.ndarray], slice_bytes: int, layer: int) -> np.ndarray:
    """Staging payload of one layer: the layer slice of every chunk object, in prefix order."""
    lib = _load()
    out = np.empty(len(chunks) * slice_bytes, dtype=np.uint8)
    lib.oco_assemble_layer(_chunk_ptrs(chunks), len(chunks), slice_bytes, layer, _ptr(out))
    return out


def logical_kv(chunks: Sequence[np.ndarray], G: int, n_kv: int, d: int, layer: int):
    """Logical prefix K, V [T][n_kv][d] (uint16 bf16 bits) decoded from chunk objects."""
    lib = _load()
    chunks = [_u16(c.reshape(-1)) for c in chunks]
    T = len(chunks) * G
    k = np.empty((T, n_kv, d), dtype=np.uint16)
    v = np.empty((T, n_kv, d), dtype=np.uint16)
    lib.oco_logical_kv(_chunk_ptrs(chunks), len(chunks), G, n_kv, d, layer, _ptr(k), _ptr(v))
    return k, v


def pool_shape(L: int, P: int, n_kv: int, Ps: int, d: int):
    return (L, 2, P, n_kv, Ps * d)


def ingest_layer(staging: np.ndarray, n_chunks: int, G: int, n_kv: int, d: int, Ps: int,
                 table: np.ndarray, pool: np.ndarray, layer: int, threads: int = 1) -> None:
    """Scatter a staging payload into ``pool`` (uint16, shape pool_shape) in
    place; with threads > 1 the chunks are divided over that many threads
    (same result for a table of distinct page ids)."""
    lib = _load()
    staging = _u16(staging.view(np.uint16) if staging.dtype == np.uint8 else staging)
    table = np.ascontiguousarray(table, dtype=np.int32)
    if not pool.flags["C_CONTIGUOUS"] or pool.dtype != np.uint16:
        raise ValueError("pool must be contiguous uint16")
    P = pool.shape[2]
    if staging.size != n_chunks * 2 * G * n_kv * d:
        raise ValueError("staging size does not match n_chunks * S")
    if threads > 1:
        rc = lib.oco_ingest_layer_mt(_ptr(staging), n_chunks, G, n_kv, d, Ps, _ptr(table), table.size,
                                     _ptr(pool), P, layer, threads)
    else:
        rc = lib.oco_ingest_layer(_ptr(staging), n_chunks, G, n_kv, d, Ps, _ptr(table), table.size,
                                  _ptr(pool), P, layer)
    if rc == -2:
        raise RuntimeError("could not start the ingest threads")
    if rc != 0:
        raise ValueError("block table entry out of range or too short")


def gather_layer(pool: np.ndarray, layer: int, table: np.ndarray, n_chunks: int, G: int,
                 n_kv: int, d: int, Ps: int) -> np.ndarray:
    lib = _load()
    table = np.ascontiguousarray(table, dtype=np.int32)
    out = np.empty(n_chunks * 2 * G * n_kv * d, dtype=np.uint16)
    rc = lib.oco_gather_layer(_ptr(pool), pool.shape[2], layer, _ptr(table), table.size, n_chunks,
                              G, n_kv, d, Ps, _ptr(out))
    if rc != 0:
        raise ValueError("block table entry out of range or too short")
    return out


def append_suffix(k_new: np.ndarray, v_new: np.ndarray, token0: int, table: np.ndarray, pool: np.ndarray,
                  layer: int, Ps: int) -> None:
    """Write one layer's suffix K/V ([T_s][n_kv][d] each) into ``pool`` at
    logical positions token0 .. token0+T_s-1, in place."""
    lib = _load()
    k_new, v_new = _u16(k_new), _u16(v_new)
    if k_new.shape != v_new.shape or k_new.ndim != 3:
        raise ValueError("k_new and v_new must both be [T_s][n_kv][d]")
    Ts, n_kv, d = k_new.shape
    table = np.ascontiguousarray(table, dtype=np.int32)
    if not pool.flags["C_CONTIGUOUS"] or pool.dtype != np.uint16:
        raise ValueError("pool must be contiguous uint16")
    rc = lib.oco_append_suffix(_ptr(k_new), _ptr(v_new), Ts, n_kv, d, Ps, _ptr(table), table.size, token0,
                               _ptr(pool), pool.shape[2], layer)
    if rc != 0:
        raise ValueError("block table entry out of range or too short")


def gather_chunks(pool: np.ndarray, table: np.ndarray, first_chunk: int, n_chunks: int, G: int, n_kv: int,
                  d: int, Ps: int) -> np.ndarray:
    """Chunk objects first_chunk .. first_chunk+n_chunks-1 rebuilt from the pool,
    all layers: uint16 [n_chunks][L*2*G*n_kv*d]."""
    lib = _load()
    table = np.ascontiguousarray(table, dtype=np.int32)
    L = pool.shape[0]
    out = np.empty((n_chunks, L * 2 * G * n_kv * d), dtype=np.uint16)
    rc = lib.oco_gather_chunks(_ptr(pool), pool.shape[2], L, _ptr(table), table.size, first_chunk, n_chunks,
                               G, n_kv, d, Ps, _ptr(out))
    if rc != 0:
        raise ValueError("block table entry out of range or too short")
    return out


def attention(q: np.ndarray, k_prefix: np.ndarray, v_prefix: np.ndarray, k_new: np.ndarray,
              v_new: np.ndarray, rows: Optional[Sequence[int]] = None, threads: Optional[int] = None
              ) -> np.ndarray:
    """float64 suffix-prefill attention.

    q [Ts][nq][d], k_prefix/v_prefix [Tp][nkv][d], k_new/v_new [Ts][nkv][d]
    (uint16 bf16 bits).  Returns [len(rows)][nq][d] float64 (all Ts rows when
    ``rows`` is None).
    """
    lib = _load()
    q, k_prefix, v_prefix, k_new, v_new = map(_u16, (q, k_prefix, v_prefix, k_new, v_new))
    Ts, nq, d = q.shape
    nkv = k_new.shape[1]
    Tp = k_prefix.shape[0] if k_prefix.size else 0
    if k_prefix.size and (k_prefix.shape[1:] != (nkv, d) or v_prefix.shape != k_prefix.shape):
        raise ValueError("prefix K/V must be [Tp][nkv][d]")
    if k_new.shape != (Ts, nkv, d) or v_new.shape != (Ts, nkv, d):
        raise ValueError("k_new/v_new must be [Ts][nkv][d]")
    if rows is None:
        rows_arr = np.arange(Ts, dtype=np.int64)
    else:
        rows_arr = np.ascontiguousarray(rows, dtype=np.int64)
    out = np.empty((rows_arr.size, nq, d), dtype=np.float64)
    if threads is None:
        threads = len(os.sched_getaffinity(0))
    # empty prefix arrays still need a valid pointer
    kp = k_prefix if k_prefix.size else np.zeros(1, np.uint16)
    vp = v_prefix if v_prefix.size else np.zeros(1, np.uint16)
    rc = lib.oco_attention(_ptr(q), _ptr(kp), _ptr(vp), _ptr(k_new), _ptr(v_new), Tp, Ts, nq, nkv,
                           d, _ptr(rows_arr), rows_arr.size, _ptr(out), threads)
    if rc != 0:
        raise ValueError(f"oracle attention failed ({rc})")
    return out
